"""The allocation-free decode entry point (ftts_decode_step_static) against
ftts_decode_step with a workspace: same inputs, bit-identical logits and ids,
on two calls in a row -- a batch of 9 (the matrix-core linears, whose split-K
partials and counters live in the scratch) and then a smaller batch of 1 (the
persistent step, whose control words and exchange buffers live there) -- and
the static scratch's limit is enforced before anything runs."""
import sys

import numpy as np
import pytest

from paper_2607_21042_amd import workload
from tests import helpers

pytestmark = pytest.mark.gpu

MID = workload.ModelShape(n_layer=2, d_model=1280, n_head=20, d_head=64, d_ff=5120, vocab=1024)


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def test_static_scratch_matches_workspace_path():
    import torch
    from paper_2607_21042_amd import ftts
    assert torch.cuda.is_available()
    inputs = workload.bf16_weights(workload.master_weights(MID, seed=0))
    dm = ftts.DeviceModel(inputs, MID, ftts.BF16)
    rng = np.random.default_rng(50)
    for B, steps, samp in ((9, 3, ftts.Sampling(0.8, 30, 0.8)), (1, 3, ftts.Sampling(1.0, 1, 1.0))):
        lens = [int(x) for x in rng.integers(20, 200, size=B)]
        say(f"static scratch: B={B} ({'persistent' if ftts.decode_path(dm, B) == 2 else 'kernel per phase'}), "
            f"prefixes {lens}")
        flat = workload.prefix_embeddings(lens, MID.d_model, seed=51)
        bt_np, n_pages = helpers.make_block_table([n + steps for n in lens], seed=3)
        kv = ftts.KVCache(MID, ftts.BF16, n_pages)
        pt = ftts.PageTableView(torch.from_numpy(bt_np).cuda(), torch.zeros(B, dtype=torch.int32, device="cuda"))
        ws = torch.empty(ftts.workspace_bytes(dm.cfg, B, sum(lens)), dtype=torch.uint8, device="cuda")
        ftts.prefill(dm, torch.from_numpy(flat).cuda().to(torch.bfloat16), lens, pt, kv, None, ws)
        pt.seq_lens.copy_(torch.tensor(lens, dtype=torch.int32))
        tok = torch.full((B,), MID.start_token, dtype=torch.int32, device="cuda")
        pos = torch.zeros(B, dtype=torch.int32, device="cuda")
        uni = torch.from_numpy(workload.uniforms(steps, B, seed=52)).cuda()
        la = torch.empty((B, MID.vocab), dtype=torch.float32, device="cuda")
        lb = torch.empty_like(la)
        sa = torch.empty(B, dtype=torch.int32, device="cuda")
        sb = torch.empty_like(sa)
        for t in range(steps):
            # the same step twice on the same state (each writes the same K/V slot)
            ftts.decode_step_static(dm, tok, pos, pt, kv, la, sa, uni[t], samp)
            ftts.decode_step(dm, tok, pos, pt, kv, lb, sb, uni[t], samp, ws)
            torch.cuda.synchronize()
            np.testing.assert_array_equal(la.cpu().numpy(), lb.cpu().numpy())
            np.testing.assert_array_equal(sa.cpu().numpy(), sb.cpu().numpy())
            assert bool((sa >= 0).all())
            tok.copy_(sa)
            pos.add_(1)
            pt.seq_lens.add_(1)
        if ftts.decode_path(dm, B) == 2:
            ftts.check_workspace(ws)
        say(f"  {steps} steps bit-identical")


def test_static_scratch_limit_is_checked():
    """A model and batch whose scratch need exceeds the static array (the 1280-wide
    decoder with a 16,384-row vocabulary at batch 64) are refused with
    FTTS_E_WORKSPACE before anything is enqueued."""
    import torch
    from paper_2607_21042_amd import ftts
    big = workload.ModelShape(n_layer=1, d_model=1280, n_head=20, d_head=64, d_ff=5120, vocab=16384)
    cfg = ftts.make_config(big, ftts.BF16)
    need = ftts.workspace_bytes(cfg, 64, 0)
    assert need > ftts.STATIC_SCRATCH_BYTES
    w = ftts.Weights()
    w.cfg = cfg
    tok = torch.zeros(64, dtype=torch.int32, device="cuda")
    rc = ftts.lib().ftts_decode_step_static(ftts._c.byref(w), tok.data_ptr(), tok.data_ptr(), None, None, None,
                                            None, None, None, 64, None)
    assert rc == -8, (rc, ftts.lib().ftts_last_error())
    assert b"static scratch" in ftts.lib().ftts_last_error()
