"""Python binding of libftts (the C ABI in include/ftts.h).

Argument marshalling only: every step of the decode path runs in the HIP
kernels of libftts.so.  torch tensors provide device memory and the stream;
their data pointers are handed to the C entry points, which carry the same
names here.  If the library is missing the binding raises instead of falling
back to anything else.
"""
from __future__ import annotations

import ctypes
import os
import re

import numpy as np
import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libftts.so")
HEADER_PATH = os.path.join(os.path.dirname(_PKG), "include", "ftts.h")

F32, BF16, W8A16, W4A16 = 0, 1, 2, 3
WDTYPE_NAMES = {F32: "f32", BF16: "bf16", W8A16: "w8a16", W4A16: "w4a16"}
MAX_TOP_K = 64
MAX_BATCH = 64
PAGE = 64

_c = ctypes
i32, f32, vp = _c.c_int32, _c.c_float, _c.c_void_p


class FTTSError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"ftts error {code}: {msg}")
        self.code = code


class Config(_c.Structure):
    _fields_ = [("n_layer", i32), ("d_model", i32), ("n_head", i32), ("d_head", i32), ("d_ff", i32),
                ("vocab", i32), ("n_pos", i32), ("page_size", i32), ("wdtype", i32), ("group_size", i32),
                ("ln_eps", f32)]


class Linear(_c.Structure):
    _fields_ = [("w", vp), ("scale", vp), ("zero", vp), ("bias", vp)]


class Layer(_c.Structure):
    _fields_ = [("ln1_g", vp), ("ln1_b", vp), ("qkv", Linear), ("out", Linear), ("ln2_g", vp), ("ln2_b", vp),
                ("fc1", Linear), ("fc2", Linear)]


class Weights(_c.Structure):
    _fields_ = [("cfg", Config), ("tok_emb", vp), ("pos_emb", vp), ("layers", _c.POINTER(Layer)),
                ("lnf_g", vp), ("lnf_b", vp), ("head", Linear)]


class DitConfig(_c.Structure):
    _fields_ = [("n_layer", i32), ("d_model", i32), ("n_head", i32), ("d_head", i32), ("d_ff", i32),
                ("n_mel", i32), ("d_cond", i32), ("t_dim", i32), ("ln_eps", f32)]


class DitWeights(_c.Structure):
    _fields_ = [("cfg", DitConfig), ("in_", Linear), ("t1", Linear), ("t2", Linear), ("layers", _c.POINTER(Layer)),
                ("lnf_g", vp), ("lnf_b", vp), ("mel", Linear)]


class KvPool(_c.Structure):
    _fields_ = [("base", vp), ("n_pages", i32)]


class PageTable(_c.Structure):
    _fields_ = [("block_table", vp), ("seq_lens", vp), ("max_pages", i32)]


class Sampling(_c.Structure):
    _fields_ = [("temperature", f32), ("top_k", i32), ("top_p", f32)]


_lib = None


def lib():
    """The loaded libftts.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise FTTSError(-7, f"{LIB_PATH} is missing; build it with `python -m paper_2607_21042_amd.build`")
        L = _c.CDLL(LIB_PATH)
        P = _c.POINTER
        L.ftts_last_error.restype = _c.c_char_p
        L.ftts_version.restype = _c.c_char_p
        L.ftts_workspace_bytes.restype = _c.c_size_t
        L.ftts_workspace_bytes.argtypes = [P(Config), i32, i32]
        L.ftts_quantize_weights.restype = _c.c_int
        L.ftts_quantize_weights.argtypes = [i32, vp, _c.c_int64, _c.c_int64, i32, vp, vp, vp, vp]
        L.ftts_prefill.restype = _c.c_int
        L.ftts_prefill.argtypes = [P(Weights), vp, P(i32), i32, P(PageTable), P(KvPool), vp, vp, _c.c_size_t, vp]
        L.ftts_decode_step.restype = _c.c_int
        L.ftts_decode_step.argtypes = [P(Weights), vp, vp, P(PageTable), P(KvPool), vp, vp, vp, P(Sampling), i32,
                                       vp, _c.c_size_t, vp]
        L.ftts_prefill_ids.restype = _c.c_int
        L.ftts_prefill_ids.argtypes = [P(Weights), vp, P(i32), vp, P(i32), i32, i32, i32, P(PageTable), P(KvPool),
                                       vp, vp, _c.c_size_t, vp]
        L.ftts_decode_step_static.restype = _c.c_int
        L.ftts_decode_step_static.argtypes = [P(Weights), vp, vp, P(PageTable), P(KvPool), vp, vp, vp, P(Sampling),
                                              i32, vp]
        L.ftts_decode_step_hidden.restype = _c.c_int
        L.ftts_decode_step_hidden.argtypes = [P(Weights), vp, vp, P(PageTable), P(KvPool), vp, vp, vp, vp,
                                              P(Sampling), i32, vp, _c.c_size_t, vp]
        L.ftts_set_decode_path.restype = _c.c_int
        L.ftts_set_decode_path.argtypes = [i32]
        L.ftts_check_workspace.restype = _c.c_int
        L.ftts_check_workspace.argtypes = [vp, _c.c_size_t, vp]
        L.ftts_decode_path.restype = _c.c_int
        L.ftts_decode_path.argtypes = [P(Weights), i32]
        L.ftts_advance.restype = _c.c_int
        L.ftts_advance.argtypes = [vp, vp, vp, vp, vp, i32, i32, vp, vp, i32, i32, vp]
        L.ftts_sample.restype = _c.c_int
        L.ftts_sample.argtypes = [vp, i32, i32, P(Sampling), vp, vp, vp]
        L.ftts_dit_workspace_bytes.restype = _c.c_size_t
        L.ftts_dit_workspace_bytes.argtypes = [P(DitConfig), i32]
        L.ftts_dit_step.restype = _c.c_int
        L.ftts_dit_step.argtypes = [P(DitWeights), vp, vp, P(i32), i32, f32, f32, f32, vp, vp, vp, _c.c_size_t,
                                    vp]
        _lib = L
    return _lib


def header_functions():
    """Names of the functions declared in include/ftts.h."""
    with open(HEADER_PATH) as f:
        text = f.read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\**\s+\**(ftts_\w+)\s*\(", text, flags=re.M)))


def _check(rc: int):
    if rc != 0:
        raise FTTSError(rc, lib().ftts_last_error().decode())


def _ptr(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if not t.is_cuda:
        raise FTTSError(-1, "tensor must live on the GPU")
    if not t.is_contiguous():
        raise FTTSError(-1, "tensor must be contiguous")
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def version() -> str:
    return lib().ftts_version().decode()


def workspace_bytes(cfg: Config, max_batch: int, max_rows: int = 0) -> int:
    n = lib().ftts_workspace_bytes(_c.byref(cfg), max_batch, max_rows)
    if n == 0:
        raise FTTSError(-1, lib().ftts_last_error().decode())
    return n


def quantize_weights(wdtype: int, w, codes, scales, zeros=None, group_size: int = 128, stream=None):
    """ftts_quantize_weights on fp32 w [N][K] (device tensors)."""
    N, K = w.shape
    if w.dtype != torch.float32:
        raise FTTSError(-3, "w must be fp32")
    _check(lib().ftts_quantize_weights(wdtype, _ptr(w), N, K, group_size, _ptr(codes), _ptr(scales), _ptr(zeros),
                                       _stream(stream)))


def sample(logits, sampling: Sampling, uniforms, sampled_out, stream=None):
    """ftts_sample: logits [B][V] fp32 -> sampled_out [B] int32."""
    B, V = logits.shape
    _check(lib().ftts_sample(_ptr(logits), B, V, _c.byref(sampling), _ptr(uniforms), _ptr(sampled_out),
                             _stream(stream)))


def prefill(model, prefix_emb, lens, page_table, kv, last_logits, ws, stream=None):
    """ftts_prefill; `lens` is a host sequence of prefix lengths."""
    B = len(lens)
    lens_arr = (i32 * B)(*[int(x) for x in lens])
    _check(lib().ftts_prefill(_c.byref(model.c), _ptr(prefix_emb), lens_arr, B, _c.byref(page_table.c),
                              _c.byref(kv.c), _ptr(last_logits), _ptr(ws), ws.numel() * ws.element_size(),
                              _stream(stream)))


def prefill_ids(model, cond_emb, cond_lens, text_ids, text_lens, text_vocab, text_pos0, page_table, kv, last_logits,
                ws, stream=None):
    """ftts_prefill_ids; `cond_lens` and `text_lens` are host sequences."""
    B = len(cond_lens)
    cl = (i32 * B)(*[int(x) for x in cond_lens])
    tl = (i32 * B)(*[int(x) for x in text_lens])
    _check(lib().ftts_prefill_ids(_c.byref(model.c), _ptr(cond_emb), cl, _ptr(text_ids), tl, int(text_vocab),
                                  int(text_pos0), B, _c.byref(page_table.c), _c.byref(kv.c), _ptr(last_logits),
                                  _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))


def decode_step(model, tokens, positions, page_table, kv, logits_out, sampled_out, uniforms, sampling: Sampling,
                ws, stream=None, hidden_out=None):
    """ftts_decode_step for B = tokens.numel() sequences; with hidden_out ([B][d_model]
    fp32) it is ftts_decode_step_hidden."""
    B = tokens.numel()
    if hidden_out is None:
        _check(lib().ftts_decode_step(_c.byref(model.c), _ptr(tokens), _ptr(positions), _c.byref(page_table.c),
                                      _c.byref(kv.c), _ptr(logits_out), _ptr(sampled_out), _ptr(uniforms),
                                      _c.byref(sampling), B, _ptr(ws), ws.numel() * ws.element_size(),
                                      _stream(stream)))
    else:
        _check(lib().ftts_decode_step_hidden(_c.byref(model.c), _ptr(tokens), _ptr(positions),
                                             _c.byref(page_table.c), _c.byref(kv.c), _ptr(logits_out),
                                             _ptr(hidden_out), _ptr(sampled_out), _ptr(uniforms),
                                             _c.byref(sampling), B, _ptr(ws), ws.numel() * ws.element_size(),
                                             _stream(stream)))


def decode_step_static(model, tokens, positions, page_table, kv, logits_out, sampled_out, uniforms,
                       sampling: Sampling, stream=None):
    """ftts_decode_step_static: ftts_decode_step with the library's static scratch
    instead of a workspace (for callers that cannot allocate)."""
    _check(lib().ftts_decode_step_static(_c.byref(model.c), _ptr(tokens), _ptr(positions), _c.byref(page_table.c),
                                         _c.byref(kv.c), _ptr(logits_out), _ptr(sampled_out), _ptr(uniforms),
                                         _c.byref(sampling), tokens.numel(), _stream(stream)))


STATIC_SCRATCH_BYTES = 12 << 20


PATH_AUTO, PATH_KERNELS, PATH_PERSISTENT = 0, 1, 2


def set_decode_path(path: int):
    """ftts_set_decode_path: 0 automatic, 1 one kernel per phase, 2 the persistent step."""
    _check(lib().ftts_set_decode_path(path))


def decode_path(model, batch: int) -> int:
    """ftts_decode_path: 1 (one kernel per phase) or 2 (persistent step) for this model and batch."""
    r = lib().ftts_decode_path(_c.byref(model.c), int(batch))
    _check(r if r < 0 else 0)
    return r


def check_workspace(ws, stream=None):
    """ftts_check_workspace: raises if a persistent step on `ws` timed out waiting."""
    _check(lib().ftts_check_workspace(_ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))


# Byte offset of the persistent step's abort word in a workspace (int32, 0 = no failure).
ABORT_WORD_OFFSET = 4


def abort_word(ws):
    """A one-element int32 view of the workspace's abort word, for an asynchronous
    device-to-host copy (ftts_check_workspace reads the same word after a sync)."""
    return ws.view(torch.uint8)[ABORT_WORD_OFFSET:ABORT_WORD_OFFSET + 4].view(torch.int32)


# Most decode steps captured into one HIP graph.  A batched step is about 125
# kernel nodes; a single graph of a whole 755-step generation (about 94k nodes)
# once ended its process without a result, while graphs of 16-64 steps have
# always run, so longer loops are split into graphs of at most this many steps.
MAX_GRAPH_STEPS = 64


def graph_steps(n: int) -> int:
    """Check a steps-per-graph request against MAX_GRAPH_STEPS; returns it."""
    n = int(n)
    if n < 1 or n > MAX_GRAPH_STEPS:
        raise ValueError(f"steps per HIP graph must be in [1, {MAX_GRAPH_STEPS}] (got {n})")
    return n


def advance(tokens, positions, seq_lens, sampled, remaining=None, stop_token=0, history=None, step_counter=None,
            stream=None, retire_on_stop=False):
    """ftts_advance: device-side bookkeeping between decode steps (retire_on_stop: a
    sequence that samples stop_token retires at once, not only when its budget ends)."""
    B = tokens.numel()
    max_steps = history.shape[0] if history is not None else 0
    _check(lib().ftts_advance(_ptr(tokens), _ptr(positions), _ptr(seq_lens), _ptr(sampled), _ptr(remaining),
                              stop_token, 1 if retire_on_stop else 0, _ptr(history), _ptr(step_counter), max_steps,
                              B, _stream(stream)))


# --------------------------------------------------------------------------- device state
def make_config(shape, wdtype: int, eps: float = 1e-5) -> Config:
    return Config(shape.n_layer, shape.d_model, shape.n_head, shape.d_head, shape.d_ff, shape.vocab, shape.n_pos,
                  PAGE, wdtype, 128, eps)


def act_dtype(wdtype: int):
    return torch.float32 if wdtype == F32 else torch.bfloat16


class DeviceModel:
    """Model weights resident in HBM plus the ftts_weights struct pointing at them.

    `weights` is the numpy dict of the seeded input generator (fp32 arrays; in
    the 16-bit modes their values must be bf16-representable).  For W8A16 and
    W4A16 the four per-layer matrices are quantised on the GPU by
    ftts_quantize_weights from the fp32 values given here.  Every per-layer
    tensor kind is one stacked allocation [n_layer, ...], so layer l of a kind
    sits at a fixed stride (what the persistent decode step requires).
    """

    LN_KINDS = ("ln1_g", "ln1_b", "ln2_g", "ln2_b")
    LINEARS = ("qkv", "out", "fc1", "fc2")

    def __init__(self, weights: dict, shape, wdtype: int, device="cuda", stream=None):
        self.shape, self.wdtype = shape, wdtype
        self.cfg = make_config(shape, wdtype)
        adt = act_dtype(wdtype)
        L = shape.n_layer
        self.tensors = {}

        def up(a, dtype=adt):
            t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(device)
            return t if dtype == torch.float32 else t.to(dtype)

        def stacked(key):
            return up(np.stack([lw[key] for lw in weights["layers"]]))

        for k in self.LN_KINDS:
            self.tensors[k] = stacked(k)
        for name in self.LINEARS:
            self.tensors["b_" + name] = stacked("b_" + name)
            N, K = weights["layers"][0]["w_" + name].shape
            if wdtype in (F32, BF16):
                self.tensors["w_" + name] = stacked("w_" + name)
                continue
            if wdtype == W8A16:
                codes = torch.empty((L, N, K), dtype=torch.int8, device=device)
                scales = torch.empty((L, N), dtype=torch.int16, device=device)
                zeros = None
            else:
                codes = torch.empty((L, N, K // 8), dtype=torch.int32, device=device)
                scales = torch.empty((L, N, K // 128), dtype=torch.int16, device=device)
                zeros = torch.empty((L, N, K // 128), dtype=torch.int16, device=device)
            for l, lw in enumerate(weights["layers"]):
                w32 = up(lw["w_" + name], torch.float32)
                quantize_weights(wdtype, w32, codes[l], scales[l], zeros[l] if zeros is not None else None,
                                 stream=stream)
                torch.cuda.current_stream().synchronize()
                del w32
            self.tensors["w_" + name] = codes
            self.tensors["s_" + name] = scales
            if zeros is not None:
                self.tensors["z_" + name] = zeros
        for k in ("tok_emb", "pos_emb", "lnf_g", "lnf_b", "b_head"):
            self.tensors[k] = up(weights[k])
        self.tensors["w_head"] = up(weights["w_head"])  # never quantised

        def ptr(key, l):
            t = self.tensors.get(key)
            return None if t is None else t[l].data_ptr()

        self.layers = (Layer * L)()
        for l in range(L):
            Ly = self.layers[l]
            Ly.ln1_g, Ly.ln1_b = ptr("ln1_g", l), ptr("ln1_b", l)
            Ly.ln2_g, Ly.ln2_b = ptr("ln2_g", l), ptr("ln2_b", l)
            for name in self.LINEARS:
                setattr(Ly, name, Linear(ptr("w_" + name, l), ptr("s_" + name, l), ptr("z_" + name, l),
                                         ptr("b_" + name, l)))
        c = Weights()
        c.cfg = self.cfg
        c.tok_emb = self.tensors["tok_emb"].data_ptr()
        c.pos_emb = self.tensors["pos_emb"].data_ptr()
        c.layers = self.layers
        c.lnf_g, c.lnf_b = self.tensors["lnf_g"].data_ptr(), self.tensors["lnf_b"].data_ptr()
        c.head = Linear(self.tensors["w_head"].data_ptr(), None, None, self.tensors["b_head"].data_ptr())
        self.c = c

    def quantised(self, name, l):
        """(codes, scales, zeros) device tensors of linear `name` in layer l (quantised modes)."""
        z = self.tensors.get("z_" + name)
        return self.tensors["w_" + name][l], self.tensors["s_" + name][l], None if z is None else z[l]

    def weight_bytes(self) -> int:
        """Bytes of every parameter tensor held on the device."""
        return sum(t.numel() * t.element_size() for t in self.tensors.values())


class PagePool:
    """Host-side page allocator over a fixed number of KV pages (a free list)."""

    def __init__(self, n_pages: int):
        self.free = list(range(n_pages - 1, -1, -1))

    def alloc(self, n: int):
        if n > len(self.free):
            raise FTTSError(-5, "KV pool exhausted")
        return [self.free.pop() for _ in range(n)]

    def release(self, pages):
        self.free.extend(reversed(list(pages)))


class KVCache:
    """The paged KV pool [n_layer][n_pages][2][n_head][64][64] and its C view."""

    def __init__(self, shape, wdtype: int, n_pages: int, device="cuda", fill=None):
        dt = act_dtype(wdtype)
        dims = (shape.n_layer, n_pages, 2, shape.n_head, PAGE, shape.d_head)
        self.pool = (torch.full(dims, fill, dtype=dt, device=device) if fill is not None
                     else torch.zeros(dims, dtype=dt, device=device))
        self.n_pages = n_pages
        self.c = KvPool(self.pool.data_ptr(), n_pages)


class PageTableView:
    """Device block table [B][max_pages] and seq_lens [B] with their C view."""

    def __init__(self, block_table, seq_lens):
        self.block_table = block_table.to(torch.int32).contiguous()
        self.seq_lens = seq_lens.to(torch.int32).contiguous()
        self.c = PageTable(self.block_table.data_ptr(), self.seq_lens.data_ptr(), self.block_table.shape[1])


# ---- flow-matching DiT step ---------------------------------------------------------------

def make_dit_config(shape, eps: float = 1e-5) -> DitConfig:
    return DitConfig(shape.n_layer, shape.d_model, shape.n_head, shape.d_head, shape.d_ff, shape.n_mel,
                     shape.d_cond, shape.t_dim, eps)


def dit_workspace_bytes(cfg: DitConfig, max_frames: int) -> int:
    n = lib().ftts_dit_workspace_bytes(_c.byref(cfg), max_frames)
    if n == 0:
        raise FTTSError(-2, "invalid DiT config or frame count")
    return n


def dit_step(model, x, cond, t: float, dt: float, cfg_w: float, x_out, v_out, ws, lens=None, stream=None):
    """One guided Euler step (ftts_dit_step) over the utterances packed in x, of
    `lens` frames each (default: one utterance of all of x's rows)."""
    lens = [x.shape[0]] if lens is None else list(lens)
    arr = (i32 * max(len(lens), 1))(*lens)
    _check(lib().ftts_dit_step(_c.byref(model.c), _ptr(x), _ptr(cond), arr, len(lens), t, dt, cfg_w, _ptr(x_out),
                               _ptr(v_out), _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)))


class DitDeviceModel:
    """DiT weights resident in HBM (bf16) plus the ftts_dit_weights struct pointing at them.

    `weights` is the dict of ``workload.dit_master_weights``; its values must be
    bf16-representable (``workload.bf16_round``) so that the oracle can take the
    very same numbers.
    """

    GLOBAL = ("w_in", "b_in", "w_t1", "b_t1", "w_t2", "b_t2", "lnf_g", "lnf_b", "w_out_mel", "b_out_mel")
    LAYER = ("ln1_g", "ln1_b", "w_qkv", "b_qkv", "w_out", "b_out", "ln2_g", "ln2_b", "w_fc1", "b_fc1", "w_fc2",
             "b_fc2")

    def __init__(self, weights: dict, shape, device="cuda"):
        self.shape = shape
        self.cfg = make_dit_config(shape)

        def up(a):
            return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(device).to(torch.bfloat16)

        self.tensors = {k: up(weights[k]) for k in self.GLOBAL}
        for k in self.LAYER:
            self.tensors[k] = up(np.stack([lw[k] for lw in weights["layers"]]))
        T = self.tensors
        self.layers = (Layer * shape.n_layer)()
        for l in range(shape.n_layer):
            Ly = self.layers[l]
            Ly.ln1_g, Ly.ln1_b = T["ln1_g"][l].data_ptr(), T["ln1_b"][l].data_ptr()
            Ly.ln2_g, Ly.ln2_b = T["ln2_g"][l].data_ptr(), T["ln2_b"][l].data_ptr()
            for name in ("qkv", "out", "fc1", "fc2"):
                setattr(Ly, name, Linear(T["w_" + name][l].data_ptr(), None, None, T["b_" + name][l].data_ptr()))
        c = DitWeights()
        c.cfg = self.cfg
        c.in_ = Linear(T["w_in"].data_ptr(), None, None, T["b_in"].data_ptr())
        c.t1 = Linear(T["w_t1"].data_ptr(), None, None, T["b_t1"].data_ptr())
        c.t2 = Linear(T["w_t2"].data_ptr(), None, None, T["b_t2"].data_ptr())
        c.layers = self.layers
        c.lnf_g, c.lnf_b = T["lnf_g"].data_ptr(), T["lnf_b"].data_ptr()
        c.mel = Linear(T["w_out_mel"].data_ptr(), None, None, T["b_out_mel"].data_ptr())
        self.c = c

    def weight_bytes(self) -> int:
        return sum(t.numel() * t.element_size() for t in self.tensors.values())
