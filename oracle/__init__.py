"""Plain, slow CPU oracle of the GPT decode path (TEST INFRASTRUCTURE ONLY).

Only the test-suite, the smoke check and the benchmark's CPU-baseline leg may
import this package.  The product path (the HIP library and its Python binding)
never imports, calls or links anything here, and this package imports nothing
from the product path: inputs arrive as plain numpy arrays.

Contents
--------
gpt     -- the exact GPT-2 style decoder forward (Sec. II-A names GPT-2 as the
           Text-to-Semantic model class): LayerNorm, causal multi-head
           attention, GELU MLP, final LayerNorm and LM head; incremental
           (KV-cache) prefill/decode and the full causal forward.
quant   -- weight-only quantisation of the GPT linears to W8A16 / W4A16
           (Table I caption, Sec. III-B) and exact dequantisation.
sample  -- greedy and temperature / top-k / top-p sampling of the next token.

All arithmetic runs in the dtype the caller picks (fp64 for self-checks, fp32
for parity); readings of points the paper leaves open are listed in each module.
"""
from . import gpt, quant, sample  # noqa: F401
