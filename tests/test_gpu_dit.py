"""GPU parity of the flow-matching DiT step (ftts_dit_step) against the DiT
oracle, both on the same bf16-rounded weights and the same seeded inputs.

Bar (bf16 weights and activations, fp32 accumulation and residual stream): the
guided velocity within DIT_REL_TOL of the oracle's, normwise, and within
DIT_ABS_TOL element-wise; the Euler update x + dt v is then checked through v
(its own rounding is fp32).  The derivation of both numbers is written beside
them in tests/helpers.py.
"""
import sys

import numpy as np
import pytest

from oracle import dit as odit
from paper_2607_21042_amd import workload
from tests import helpers

pytestmark = pytest.mark.gpu


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available()
    return torch


_MODELS = {}


def device_model(torch, shape):
    """(device model, oracle) for a shape, built once per module."""
    from paper_2607_21042_amd import ftts
    if shape not in _MODELS:
        w = workload.bf16_weights(workload.dit_master_weights(shape, seed=20))
        _MODELS[shape] = (ftts.DitDeviceModel(w, shape), odit.DiT(w, shape.n_head, shape.d_head, dtype=np.float64))
    return _MODELS[shape]


def run_step(torch, shape, T, t, dt, cfg_w, seed, in_place=False, want_v=True):
    from paper_2607_21042_amd import ftts
    dm, ora = device_model(torch, shape)
    x, cond = workload.dit_inputs(shape, T, seed=seed)
    xg = torch.from_numpy(x).cuda()
    cg = torch.from_numpy(cond).cuda().to(torch.bfloat16)
    xo = xg if in_place else torch.empty_like(xg)
    vo = torch.empty_like(xg) if want_v else None
    ws = torch.empty(ftts.dit_workspace_bytes(dm.cfg, T), dtype=torch.uint8, device="cuda")
    say(f"dit step: T={T} d={shape.d_model} layers={shape.n_layer} t={t} dt={dt} w={cfg_w} in_place={in_place}")
    ftts.dit_step(dm, xg, cg, t, dt, cfg_w, xo, vo, ws)
    torch.cuda.synchronize()
    x_ref, v_ref = ora.step(x, cond, t, dt, cfg_w)
    return (xo.cpu().numpy(), None if vo is None else vo.cpu().numpy(), x_ref, v_ref, x)


def check(v, v_ref, label):
    ok, rel, err = helpers.dit_tolerance_ok(v, v_ref)
    say(f"  {label}: normwise rel err {rel:.3e}, max abs err {err:.3e}, max |v| {np.max(np.abs(v_ref)):.3f}")
    assert ok, (label, rel, err)


@pytest.mark.parametrize("T", [1, 37, 97, 300])
def test_dit_step_tiny(torch_cuda, T):
    """Two blocks of width 256.  Attention works in 32-key tiles split over 4
    waves: one frame (3 waves idle), two tiles, four tiles with a single key in
    the last, and ten tiles with a ragged tail (waves with 2 and 3 tiles)."""
    xo, vo, x_ref, v_ref, x = run_step(torch_cuda, workload.DIT_TINY, T, 0.3, 0.04, 1.7, seed=21 + T)
    check(vo, v_ref, f"v T={T}")
    # x' - x = dt v: compare the update itself through the velocity's bar
    check((xo.astype(np.float64) - x) / 0.04, (x_ref - x) / 0.04, f"(x'-x)/dt T={T}")


def test_dit_step_in_place_without_velocity(torch_cuda):
    """x_out may alias x and v_out may be NULL: same update as the out-of-place call."""
    sh = workload.DIT_TINY
    xo1, _, _, _, x = run_step(torch_cuda, sh, 129, 0.8, -0.1, 2.5, seed=5)
    xo2, vo2, x_ref, _, _ = run_step(torch_cuda, sh, 129, 0.8, -0.1, 2.5, seed=5, in_place=True, want_v=False)
    assert vo2 is None
    np.testing.assert_array_equal(xo1, xo2)
    check((xo2.astype(np.float64) - x) / -0.1, (x_ref - x) / -0.1, "in place")


def test_dit_step_guidance_limits(torch_cuda):
    """w = 1 gives the conditional branch and w = 0 the unconditional one; the
    two differ (the conditioning reaches the output)."""
    sh = workload.DIT_TINY
    _, v1, _, v1_ref, _ = run_step(torch_cuda, sh, 64, 0.5, 0.02, 1.0, seed=9)
    _, v0, _, v0_ref, _ = run_step(torch_cuda, sh, 64, 0.5, 0.02, 0.0, seed=9)
    check(v1, v1_ref, "w=1")
    check(v0, v0_ref, "w=0")
    assert np.max(np.abs(v1_ref - v0_ref)) > 10 * helpers.DIT_ABS_TOL


def test_dit_step_96m(torch_cuda):
    """The 96M-parameter shape (13 blocks of width 768, conditioning width 1280)
    over 500 frames, the frame count the step is measured on."""
    xo, vo, x_ref, v_ref, x = run_step(torch_cuda, workload.DIT_96M, 500, 0.64, 0.04, 2.0, seed=31)
    check(vo, v_ref, "v 96M T=500")
    check((xo.astype(np.float64) - x) / 0.04, (x_ref - x) / 0.04, "(x'-x)/dt 96M")


def run_batch(torch, shape, lens, t, dt, cfg_w, seed):
    """One call over several packed utterances; each checked against its own oracle step."""
    from paper_2607_21042_amd import ftts
    dm, ora = device_model(torch, shape)
    parts = [workload.dit_inputs(shape, n, seed=seed + i) for i, n in enumerate(lens)]
    x = np.concatenate([p[0] for p in parts])
    cond = np.concatenate([p[1] for p in parts])
    xg = torch.from_numpy(x).cuda()
    cg = torch.from_numpy(cond).cuda().to(torch.bfloat16)
    xo, vo = torch.empty_like(xg), torch.empty_like(xg)
    ws = torch.empty(ftts.dit_workspace_bytes(dm.cfg, int(sum(lens))), dtype=torch.uint8, device="cuda")
    say(f"dit batch: lens={lens} d={shape.d_model} layers={shape.n_layer} t={t} dt={dt} w={cfg_w}")
    ftts.dit_step(dm, xg, cg, t, dt, cfg_w, xo, vo, ws, lens=lens)
    torch.cuda.synchronize()
    vo = vo.cpu().numpy()
    off = 0
    for i, (n, (xi, ci)) in enumerate(zip(lens, parts)):
        _, v_ref = ora.step(xi, ci, t, dt, cfg_w)
        check(vo[off:off + n], v_ref, f"utterance {i} ({n} frames)")
        off += n


def test_dit_step_batch_tiny(torch_cuda):
    """Utterances attend only to their own frames: a batch of four lengths (one
    of a single frame) matches four separate oracle steps."""
    run_batch(torch_cuda, workload.DIT_TINY, [37, 1, 130, 64], 0.45, 0.05, 1.6, seed=40)


def test_dit_step_batch_wide_grid(torch_cuda):
    """32 utterances of 257-400 frames: enough 128-query tiles (>= 256 with the
    heads) that the attention shares each K and V tile among 128 queries instead
    of splitting the keys over waves; ragged lengths in every tile position."""
    lens = [257 + (37 * i) % 144 for i in range(32)]
    run_batch(torch_cuda, workload.DIT_TINY, lens, 0.7, 0.03, 1.3, seed=70)


def test_dit_step_batch_96m(torch_cuda):
    """Two utterances of the 96M shape in one step."""
    run_batch(torch_cuda, workload.DIT_96M, [431, 257], 0.2, 0.04, 1.7, seed=50)


def test_dit_step_without_conditioning(torch_cuda):
    """d_cond = 0 (cond may be NULL): both guidance branches are the same
    computation, so the velocity does not depend on the guidance strength.  Also
    the smallest state width (64 mel bins) and the largest time-feature width
    (1024)."""
    import torch
    from paper_2607_21042_amd import ftts
    sh = workload.DitShape(n_layer=1, d_model=128, n_head=2, d_head=64, d_ff=256, n_mel=64, d_cond=0, t_dim=1024)
    w = workload.bf16_weights(workload.dit_master_weights(sh, seed=20))
    dm = ftts.DitDeviceModel(w, sh)
    ora = odit.DiT(w, sh.n_head, sh.d_head, dtype=np.float64)
    x, cond = workload.dit_inputs(sh, 45, seed=3)
    xg = torch.from_numpy(x).cuda()
    ws = torch.empty(ftts.dit_workspace_bytes(dm.cfg, 45), dtype=torch.uint8, device="cuda")
    vs = []
    for cfg_w in (0.0, 3.0):
        xo, vo = torch.empty_like(xg), torch.empty_like(xg)
        say(f"dit step without conditioning: T=45 w={cfg_w}")
        ftts.dit_step(dm, xg, None, 0.4, 0.1, cfg_w, xo, vo, ws)
        torch.cuda.synchronize()
        _, v_ref = ora.step(x, cond, 0.4, 0.1, cfg_w)
        check(vo.cpu().numpy(), v_ref, f"d_cond=0 w={cfg_w}")
        vs.append(vo.cpu().numpy())
    np.testing.assert_allclose(vs[0], vs[1], rtol=0, atol=1e-6)


def test_dit_step_rejects_bad_calls(torch_cuda):
    """A workspace too small, no frames or a non-finite time fail before any launch."""
    import torch
    from paper_2607_21042_amd import ftts
    dm, _ = device_model(torch, workload.DIT_TINY)
    x = torch.zeros((40, workload.DIT_TINY.n_mel), device="cuda")
    c = torch.zeros((40, workload.DIT_TINY.d_cond), device="cuda", dtype=torch.bfloat16)
    small = torch.empty(ftts.dit_workspace_bytes(dm.cfg, 39), dtype=torch.uint8, device="cuda")
    with pytest.raises(ftts.FTTSError) as e:
        ftts.dit_step(dm, x, c, 0.1, 0.1, 1.0, x, None, small)
    assert e.value.code == -8  # FTTS_E_WORKSPACE
    ws = torch.empty(ftts.dit_workspace_bytes(dm.cfg, 40), dtype=torch.uint8, device="cuda")
    with pytest.raises(ftts.FTTSError):
        ftts.dit_step(dm, x[:0], c[:0], 0.1, 0.1, 1.0, x[:0], None, ws)
    with pytest.raises(ftts.FTTSError):
        ftts.dit_step(dm, x, c, float("nan"), 0.1, 1.0, x, None, ws)


def test_dit_steps_replay_from_a_graph(torch_cuda):
    """Three Euler steps captured into one HIP graph: every replay (with eager
    work and synchronisations between them) equals the eager steps bit for bit
    (fixed split-K summation order; the step clears its scratch with kernels)."""
    import torch
    from paper_2607_21042_amd import ftts
    sh = workload.DIT_TINY
    dm, _ = device_model(torch, sh)
    lens = [70, 33]
    x0_np, cond_np = workload.dit_inputs(sh, sum(lens), seed=60)
    x0 = torch.from_numpy(x0_np).cuda()
    cond = torch.from_numpy(cond_np).cuda().to(torch.bfloat16)
    ws = torch.empty(ftts.dit_workspace_bytes(dm.cfg, sum(lens)), dtype=torch.uint8, device="cuda")
    x = torch.empty_like(x0)

    def solve():
        x.copy_(x0)
        for k in range(3):
            ftts.dit_step(dm, x, cond, 0.1 + 0.2 * k, 0.2, 1.5, x, None, ws, lens=lens)

    say("dit graph: eager reference")
    solve()
    torch.cuda.synchronize()
    ref = x.clone()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        solve()
    for r in range(3):
        x.fill_(float("nan"))
        torch.cuda.synchronize()
        say(f"dit graph: replay {r}")
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(x, ref), r
        solve()  # eager work between replays
        torch.cuda.synchronize()
        assert torch.equal(x, ref)
