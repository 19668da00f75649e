"""MI355X (gfx950) decode path of IndexTTS-2's Text-to-Semantic GPT.

Submodules:
  ftts      -- Python binding of libftts.so (the C ABI in include/ftts.h);
               imported on first use so that the seeded input generator can be
               used without loading the GPU library.
  workload  -- seeded synthetic inputs (weights, prefixes, lengths, uniforms).
  build     -- compiles libftts.so with hipcc for gfx950.
"""
__all__ = ["ftts", "workload", "build"]
