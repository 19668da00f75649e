"""Host-side checks of the C ABI that need no GPU: the library loads, exports
every function include/ftts.h declares, sizes workspaces, and rejects bad
arguments before anything is enqueued (every call below fails validation, so
no kernel is launched and no pointer is dereferenced)."""
import ctypes
import os

import pytest

from paper_2607_21042_amd import ftts, workload

FAKE = 0x100000  # aligned, never dereferenced: every call here fails validation first


def test_library_exports_every_header_function():
    names = ftts.header_functions()
    assert set(names) >= {"ftts_prefill", "ftts_decode_step", "ftts_quantize_weights", "ftts_sample",
                          "ftts_workspace_bytes", "ftts_last_error", "ftts_version"}
    L = ftts.lib()
    for n in names:
        assert hasattr(L, n), n
    assert "gfx950" in ftts.version()


def test_workspace_bytes_grows_with_batch_and_rows():
    cfg = ftts.make_config(workload.INDEXTTS2, ftts.BF16)
    a = ftts.workspace_bytes(cfg, 1, 0)
    b = ftts.workspace_bytes(cfg, 32, 0)
    c = ftts.workspace_bytes(cfg, 1, 512)
    assert 0 < a < b and a < c
    assert a % 256 == 0
    with pytest.raises(ftts.FTTSError):
        ftts.workspace_bytes(cfg, 0, 0)
    with pytest.raises(ftts.FTTSError):
        ftts.workspace_bytes(cfg, ftts.MAX_BATCH + 1, 0)


@pytest.mark.parametrize("field,value,code", [
    ("d_head", 32, -7), ("page_size", 16, -7), ("n_head", 3, -2), ("d_model", 200, -2),
    ("d_ff", 100, -2), ("wdtype", 9, -3), ("vocab", 1, -2), ("n_layer", 0, -2), ("ln_eps", 0.0, -5)])
def test_bad_config_rejected(field, value, code):
    cfg = ftts.make_config(workload.TINY, ftts.F32)
    setattr(cfg, field, value)
    assert ftts.lib().ftts_workspace_bytes(ctypes.byref(cfg), 1, 0) == 0
    w = _fake_weights(cfg)
    rc = _decode(w, B=1)
    assert rc == code, ftts.lib().ftts_last_error()


def _fake_weights(cfg):
    n = max(cfg.n_layer, 1)
    layers = (ftts.Layer * n)()
    for L in layers:
        L.ln1_g = L.ln1_b = L.ln2_g = L.ln2_b = FAKE
        for lin in (L.qkv, L.out, L.fc1, L.fc2):
            lin.w = lin.bias = lin.scale = lin.zero = FAKE
    w = ftts.Weights()
    w.cfg = cfg
    w.tok_emb = w.pos_emb = w.lnf_g = w.lnf_b = FAKE
    w.layers = layers
    w.head.w = w.head.bias = FAKE
    w._layers = layers
    return w


def _decode(w, B=1, samp=None, ws_bytes=1 << 30, tokens=FAKE, uniforms=FAKE, pt=None, kv=None, ws=FAKE):
    pt = pt or ftts.PageTable(FAKE, FAKE, 4)
    kv = kv or ftts.KvPool(FAKE, 16)
    samp = samp or ftts.Sampling(1.0, 1, 1.0)
    return ftts.lib().ftts_decode_step(ctypes.byref(w), tokens, FAKE, ctypes.byref(pt), ctypes.byref(kv), FAKE,
                                       FAKE, uniforms, ctypes.byref(samp), B, ws, ws_bytes, None)


def test_decode_argument_errors():
    cfg = ftts.make_config(workload.TINY, ftts.F32)
    w = _fake_weights(cfg)
    assert _decode(w, B=0) == -2
    assert _decode(w, B=ftts.MAX_BATCH + 1) == -2
    assert _decode(w, tokens=None) == -1
    assert _decode(w, samp=ftts.Sampling(1.0, 0, 1.0)) == -5
    assert _decode(w, samp=ftts.Sampling(1.0, ftts.MAX_TOP_K + 1, 1.0)) == -5
    assert _decode(w, samp=ftts.Sampling(0.0, 5, 0.9)) == -5
    assert _decode(w, samp=ftts.Sampling(1.0, 5, 1.5)) == -5
    assert _decode(w, samp=ftts.Sampling(1.0, 5, 0.9), uniforms=None) == -1
    assert _decode(w, ws_bytes=16) == -8
    assert _decode(w, ws=FAKE + 4) == -4
    assert _decode(w, pt=ftts.PageTable(FAKE, FAKE, 0)) == -2
    assert _decode(w, kv=ftts.KvPool(None, 4)) == -1
    assert "kv.base" in ftts.lib().ftts_last_error().decode()
    w.head.w = FAKE + 8
    assert _decode(w) == -4
    w.head.w = FAKE
    # the hidden-state variant takes the same checks, plus the alignment of hidden_out
    pt, kv, samp = ftts.PageTable(FAKE, FAKE, 4), ftts.KvPool(FAKE, 16), ftts.Sampling(1.0, 1, 1.0)
    hid = ftts.lib().ftts_decode_step_hidden
    args = lambda h, B: (ctypes.byref(w), FAKE, FAKE, ctypes.byref(pt), ctypes.byref(kv), FAKE, h, FAKE,  # noqa: E731
                         FAKE, ctypes.byref(samp), B, FAKE, 1 << 30, None)
    assert hid(*args(FAKE + 8, 1)) == -4
    assert "hidden_out" in ftts.lib().ftts_last_error().decode()
    assert hid(*args(FAKE, 0)) == -2
    w.layers[1].fc2.bias = None
    assert _decode(w) == -1


def test_quantised_modes_need_scales():
    cfg = ftts.make_config(workload.TINY, ftts.W4A16)
    w = _fake_weights(cfg)
    w.layers[0].qkv.zero = None
    assert _decode(w) == -1
    cfg.group_size = 64
    w = _fake_weights(cfg)
    assert _decode(w) == -7


def test_prefill_argument_errors():
    cfg = ftts.make_config(workload.TINY, ftts.F32)
    w = _fake_weights(cfg)
    pt = ftts.PageTable(FAKE, None, 1)
    kv = ftts.KvPool(FAKE, 4)
    L = ftts.lib()

    def call(lens, B=None):
        arr = (ctypes.c_int32 * max(len(lens), 1))(*lens)
        return L.ftts_prefill(ctypes.byref(w), FAKE, arr, len(lens) if B is None else B, ctypes.byref(pt),
                              ctypes.byref(kv), FAKE, FAKE, 1 << 30, None)

    assert call([0]) == -5
    assert call([65]) == -5          # more rows than max_pages * 64
    assert call([], B=0) == -2
    assert L.ftts_prefill(ctypes.byref(w), FAKE, None, 1, ctypes.byref(pt), ctypes.byref(kv), FAKE, FAKE,
                          1 << 30, None) == -1

    def ids(cond_lens, text_lens, text_vocab=50, text_pos0=0, text_ids=FAKE, cond=FAKE):
        cl = (ctypes.c_int32 * len(cond_lens))(*cond_lens)
        tl = (ctypes.c_int32 * len(text_lens))(*text_lens)
        return L.ftts_prefill_ids(ctypes.byref(w), cond, cl, text_ids, tl, text_vocab, text_pos0, len(cond_lens),
                                  ctypes.byref(pt), ctypes.byref(kv), FAKE, FAKE, 1 << 30, None)

    assert ids([0], [0]) == -5                          # an empty prefix
    assert ids([-1], [3]) == -5
    assert ids([2], [3], text_pos0=-1) == -5
    assert ids([2], [3], text_pos0=workload.TINY.n_pos - 2) == -5   # text positions past n_pos
    assert ids([2], [3], text_ids=None) == -1
    assert ids([2], [3], text_vocab=0) == -5
    assert ids([2], [0], cond=None) == -1
    assert ids([40], [30]) == -5                        # 70 rows > max_pages * 64


def test_quantize_and_sample_argument_errors():
    L = ftts.lib()
    assert L.ftts_quantize_weights(7, FAKE, 4, 128, 128, FAKE, FAKE, FAKE, None) == -3
    assert L.ftts_quantize_weights(ftts.W4A16, FAKE, 4, 100, 128, FAKE, FAKE, FAKE, None) == -2
    assert L.ftts_quantize_weights(ftts.W4A16, FAKE, 4, 256, 64, FAKE, FAKE, FAKE, None) == -7
    assert L.ftts_quantize_weights(ftts.W4A16, FAKE, 4, 256, 128, FAKE, FAKE, None, None) == -1
    assert L.ftts_quantize_weights(ftts.W8A16, FAKE, 4, 24, 128, FAKE, FAKE, None, None) == -2
    assert L.ftts_quantize_weights(ftts.W8A16, None, 4, 32, 128, FAKE, FAKE, None, None) == -1
    s = ftts.Sampling(1.0, 10, 0.9)
    assert L.ftts_sample(FAKE, 1, 5, ctypes.byref(s), FAKE, FAKE, None) == -5   # top_k > V
    assert L.ftts_sample(FAKE, 0, 50, ctypes.byref(s), FAKE, FAKE, None) == -2
    assert L.ftts_sample(FAKE, 1, 50000, ctypes.byref(s), FAKE, FAKE, None) == -2
    assert L.ftts_sample(None, 1, 50, ctypes.byref(s), FAKE, FAKE, None) == -1


def test_page_pool_allocator():
    p = ftts.PagePool(4)
    a = p.alloc(3)
    assert sorted(a) == [0, 1, 2]
    with pytest.raises(ftts.FTTSError):
        p.alloc(2)
    p.release(a)
    assert len(p.alloc(4)) == 4


def test_decode_path_query():
    """ftts_decode_path answers from host data only: fp32 weights never take the
    persistent step, a bad batch is refused, and path 1 is always honoured."""
    L = ftts.lib()
    w = _fake_weights(ftts.make_config(workload.TINY, ftts.F32))
    assert L.ftts_decode_path(ctypes.byref(w), 1) == 1
    assert L.ftts_decode_path(ctypes.byref(w), 0) == -5
    assert L.ftts_decode_path(ctypes.byref(w), ftts.MAX_BATCH + 1) == -5
    try:
        ftts.set_decode_path(ftts.PATH_PERSISTENT)
        assert L.ftts_decode_path(ctypes.byref(w), 1) == -7
        ftts.set_decode_path(ftts.PATH_KERNELS)
        assert L.ftts_decode_path(ctypes.byref(w), 1) == 1
    finally:
        ftts.set_decode_path(ftts.PATH_AUTO)


def _fake_dit(shape):
    cfg = ftts.make_dit_config(shape)
    layers = (ftts.Layer * shape.n_layer)()
    for L in layers:
        L.ln1_g = L.ln1_b = L.ln2_g = L.ln2_b = FAKE
        for lin in (L.qkv, L.out, L.fc1, L.fc2):
            lin.w = lin.bias = FAKE
    w = ftts.DitWeights()
    w.cfg = cfg
    for lin in (w.in_, w.t1, w.t2, w.mel):
        lin.w = lin.bias = FAKE
    w.lnf_g = w.lnf_b = FAKE
    w.layers = layers
    w._layers = layers
    return w


def _dit_step(w, T=8, t=0.5, ws_bytes=1 << 30, x=FAKE, x_out=FAKE, cond=FAKE, lens=None):
    lens = [T] if lens is None else lens
    arr = (ctypes.c_int32 * max(len(lens), 1))(*lens)
    return ftts.lib().ftts_dit_step(ctypes.byref(w), x, cond, arr, len(lens), t, 0.1, 1.0, x_out, None, FAKE,
                                    ws_bytes, None)


def test_dit_workspace_bytes():
    """Grows with the frame count, covers the split-K scratch of every smaller
    call, and is 0 for a config the step rejects."""
    cfg = ftts.make_dit_config(workload.DIT_96M)
    sizes = [ftts.dit_workspace_bytes(cfg, T) for T in (1, 2, 37, 64, 500, 4096)]
    assert all(a < b for a, b in zip(sizes, sizes[1:]))
    assert sizes[0] % 256 == 0
    L = ftts.lib()
    assert L.ftts_dit_workspace_bytes(ctypes.byref(cfg), 0) == 0
    for field, value in [("d_head", 32), ("n_head", 5), ("n_mel", 100), ("d_cond", 33), ("t_dim", 3),
                         ("t_dim", 2048), ("d_ff", 96), ("n_layer", 0), ("ln_eps", 0.0)]:
        bad = ftts.make_dit_config(workload.DIT_96M)
        setattr(bad, field, value)
        assert L.ftts_dit_workspace_bytes(ctypes.byref(bad), 16) == 0, field


def test_dit_step_argument_errors():
    w = _fake_dit(workload.DIT_TINY)
    L = ftts.lib()
    assert _dit_step(w, T=0) == -2
    assert _dit_step(w, lens=[]) == -2
    assert _dit_step(w, lens=[4] * 33) == -2
    assert _dit_step(w, lens=[4, 0, 4]) == -2
    need = ftts.dit_workspace_bytes(w.cfg, 4 + 9 + 30)
    assert _dit_step(w, lens=[4, 9, 30], ws_bytes=need - 1) == -8
    assert _dit_step(w, t=float("inf")) == -5
    assert _dit_step(w, x=None) == -1
    assert _dit_step(w, x_out=FAKE + 8) == -4
    assert _dit_step(w, cond=None) == -1
    need = ftts.dit_workspace_bytes(w.cfg, 8)
    assert _dit_step(w, ws_bytes=need - 1) == -8
    assert b"workspace" in L.ftts_last_error()
    w.layers[1].fc2.bias = None
    assert _dit_step(w) == -1
    w.cfg.d_head = 32
    assert _dit_step(w) == -7


def test_graph_step_cap():
    """Steps per captured HIP graph are capped on the host: the binding refuses
    larger requests, and bench.py exits with an error before touching a GPU."""
    import subprocess
    import sys
    from paper_2607_21042_amd import ftts
    assert ftts.graph_steps(1) == 1
    assert ftts.graph_steps(ftts.MAX_GRAPH_STEPS) == ftts.MAX_GRAPH_STEPS
    for bad in (0, -3, ftts.MAX_GRAPH_STEPS + 1, 755):
        with pytest.raises(ValueError):
            ftts.graph_steps(bad)
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--graph-steps", "755"],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 2, r.stdout + r.stderr
    assert "steps per HIP graph" in r.stdout


def test_abort_word_offset_matches_header():
    """The binding's asynchronous view of the abort word sits where the header says."""
    from paper_2607_21042_amd import ftts
    with open(ftts.HEADER_PATH) as fh:
        text = fh.read()
    assert "byte offset\n * 4 of the workspace" in text or "byte offset 4" in text.replace("\n *", "")
    assert ftts.ABORT_WORD_OFFSET == 4
