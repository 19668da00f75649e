"""GPU parity at the configurations' real lengths.

* Batched decode (the MFMA linears and the paged attention kernel of batches of
  8 and more) over contexts of 600-1,300 tokens, so that each of an attention
  workgroup's 8 waves walks two or three KV pages; sampling with top-k 30,
  top-p 0.8, temperature 0.8 and host uniforms, STOP forced by the device-side
  step bookkeeping, pages scattered over the pool.
* The batched paged workload at 24 layers: 32 sequences with prefixes drawn
  U[128, 512], sampled closed-loop.
* The three batch-1 configurations at full length (512 greedy steps, teacher-
  forced on the oracle's own greedy tokens), with the page table the benchmark
  uses, so the persistent step splits each head's attention over 2 workgroups.

Bars as in test_gpu_parity: bf16-storage logits within 3e-2 absolute of the
fp32 oracle on the same dequantised weights; greedy choices equal except at
oracle near-ties; sampled choices equal to the oracle sampler's on the GPU's
own logits and uniforms, except draws within 1e-5 of a cumulative-sum boundary
(counted); page placement bit-for-bit irrelevant.
"""
import sys

import numpy as np
import pytest

from oracle import gpt as ogpt
from oracle import sample as osample
from paper_2607_21042_amd import workload
from tests import helpers

pytestmark = pytest.mark.gpu

MID = workload.ModelShape(n_layer=2, d_model=1280, n_head=20, d_head=64, d_ff=5120, vocab=1024)
TOP_K, TOP_P, TEMP = 30, 0.8, 0.8


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def torch_cuda():
    import torch
    assert torch.cuda.is_available()
    return torch


def wd(name):
    from paper_2607_21042_amd import ftts
    return {"f32": ftts.F32, "bf16": ftts.BF16, "w8a16": ftts.W8A16, "w4a16": ftts.W4A16}[name]


def model_inputs(mode, master):
    if mode == "bf16":
        return workload.bf16_weights(master)
    return workload.quantisable_weights(master)


def closed_loop(dm, shape, prefixes, budgets, T, uniforms, block_table, n_pages):
    """Prefill, then T decode steps whose sampled ids are fed back on the device
    (ftts_advance; a sequence's budget-th id is forced to STOP and the slot
    retires).  Returns per-step logits [T][B][V], the sampler's own ids [T][B]
    (before STOP forcing) and the fed-back history [T][B] (-1 once retired)."""
    import torch
    from paper_2607_21042_amd import ftts
    B = len(prefixes)
    lens = [p.shape[0] for p in prefixes]
    kv = ftts.KVCache(shape, dm.wdtype, n_pages)
    bt = torch.from_numpy(block_table).cuda()
    seq_lens = torch.tensor(lens, dtype=torch.int32, device="cuda")
    pt = ftts.PageTableView(bt, seq_lens)
    adt = ftts.act_dtype(dm.wdtype)
    prefix = torch.from_numpy(np.concatenate(prefixes).astype(np.float32)).cuda().to(adt)
    ws = torch.empty(ftts.workspace_bytes(dm.cfg, B, sum(lens)), dtype=torch.uint8, device="cuda")
    V = shape.vocab
    last = torch.empty((B, V), dtype=torch.float32, device="cuda")
    ftts.prefill(dm, prefix, lens, pt, kv, last, ws)
    pt.seq_lens.copy_(torch.tensor(lens, dtype=torch.int32))
    samp = ftts.Sampling(TEMP, TOP_K, TOP_P)
    tok = torch.full((B,), shape.start_token, dtype=torch.int32, device="cuda")
    pos = torch.zeros(B, dtype=torch.int32, device="cuda")
    rem = torch.tensor(budgets, dtype=torch.int32, device="cuda")
    sampled = torch.empty(B, dtype=torch.int32, device="cuda")
    logits = torch.empty((T, B, V), dtype=torch.float32, device="cuda")
    raw = torch.empty((T, B), dtype=torch.int32, device="cuda")
    hist = torch.full((T, B), -7, dtype=torch.int32, device="cuda")
    ctr = torch.zeros(1, dtype=torch.int32, device="cuda")
    un = torch.from_numpy(np.ascontiguousarray(uniforms, np.float32)).cuda()
    for t in range(T):
        ftts.decode_step(dm, tok, pos, pt, kv, logits[t], sampled, un[t], samp, ws)
        raw[t].copy_(sampled)
        ftts.advance(tok, pos, pt.seq_lens, sampled, rem, shape.stop_token, hist, ctr)
    torch.cuda.synchronize()
    if ftts.decode_path(dm, B) == 2:
        ftts.check_workspace(ws)
    return logits.cpu().numpy(), raw.cpu().numpy(), hist.cpu().numpy()


def check_closed_loop(om, shape, prefixes, budgets, uniforms, logits, raw, hist, mode):
    """Every active step's logits against the oracle teacher-forced on the ids the
    GPU fed itself; every sampled id against the oracle sampler on the GPU's
    logits; STOP at each budget's last step and nothing after it."""
    B = len(prefixes)
    T = logits.shape[0]
    worst, n_near, n_checked = 0.0, 0, 0
    for b in range(B):
        n = min(budgets[b], T)
        steps = list(range(n))
        fed = np.concatenate([[shape.start_token], hist[:n - 1, b]]).astype(np.int32)
        assert np.all(fed >= 0), (b, fed)
        _, ref = helpers.oracle_teacher_forced(om, prefixes[b], fed)
        for i, t in enumerate(steps):
            ok, err = helpers.tolerance_ok(logits[t, b], ref[i], mode)
            worst = max(worst, err)
            assert ok, ("logits", t, b, err)
            want, det = osample.sample(logits[t, b], TEMP, TOP_K, TOP_P, np.float32(uniforms[t, b]))
            n_checked += 1
            if int(raw[t, b]) != want:
                assert osample.near_boundary(det), ("sample", t, b, int(raw[t, b]), want)
                n_near += 1
            expect = shape.stop_token if t == budgets[b] - 1 else int(raw[t, b])
            assert int(hist[t, b]) == expect, ("history", t, b)
        if budgets[b] <= T:
            assert np.all(hist[n:, b] == -1), ("retired slot produced ids", b)
        if b % 8 == 7:
            say(f"  oracle checked {b + 1} of {B} sequences")
    assert n_near <= max(1, n_checked // 100), (n_near, n_checked)
    return worst, n_near, n_checked


def scattered_table(lens_total, seed):
    return helpers.make_block_table(lens_total, seed=seed, spare=5)


@pytest.fixture(scope="module")
def mid_master():
    return workload.master_weights(MID, seed=0)


@pytest.mark.parametrize("mode", ["bf16", "w8a16"])
def test_batched_long_contexts_sampled(torch_cuda, mid_master, mode):
    """12 sequences with prefixes of 600-1,280 tokens (10-21 pages: 2-3 per
    attention wave), 14 sampled steps, budgets of 5-14 steps so that most
    sequences hit their forced STOP and retire mid-run; the same run with
    another page placement is bit-identical."""
    from paper_2607_21042_amd import ftts
    B, T = 12, 14
    rng = np.random.default_rng(40)
    lens = [int(x) for x in rng.integers(600, 1281, size=B)]
    lens[0], lens[1] = 1280, 600
    budgets = [int(x) for x in rng.integers(5, T + 1, size=B)]
    budgets[0] = T
    inputs = model_inputs(mode, mid_master)
    flat = workload.prefix_embeddings(lens, MID.d_model, seed=41)
    prefixes = np.split(flat, np.cumsum(lens)[:-1])
    uni = workload.uniforms(T, B, seed=2)
    dm = ftts.DeviceModel(inputs, MID, wd(mode))
    assert ftts.decode_path(dm, B) == 1
    totals = [n + T for n in lens]
    bt0, n_pages = scattered_table(totals, seed=3)
    say(f"batched long contexts {mode}: {min(lens)}-{max(lens)} tokens, up to {bt0.shape[1]} pages")
    lg0, raw0, hist0 = closed_loop(dm, MID, prefixes, budgets, T, uni, bt0, n_pages)
    om = ogpt.GPT(helpers.oracle_weights(inputs, mode), MID.n_head, MID.d_head, dtype=np.float32)
    worst, near, n = check_closed_loop(om, MID, prefixes, budgets, uni, lg0, raw0, hist0, mode)
    say(f"  worst abs err {worst:.3g}; sampled ids checked {n}, near-boundary {near}")
    bt1, _ = scattered_table(totals, seed=9)
    lg1, raw1, hist1 = closed_loop(dm, MID, prefixes, budgets, T, uni, bt1, n_pages)
    np.testing.assert_array_equal(lg0, lg1)
    np.testing.assert_array_equal(hist0, hist1)


@pytest.fixture(scope="module")
def big_master():
    return workload.master_weights(workload.INDEXTTS2, seed=0)


def test_paged_batch32_24_layers(torch_cuda, big_master):
    """The batched paged workload at its real shape: 24 layers, 32 sequences with
    prefixes ~U[128, 512] (seed 3), pages scattered over one pool, 10 sampled
    steps (top-k 30, top-p 0.8, T 0.8, host uniforms of seed 2) fed back on the
    device; every logit and sampled id against the oracle."""
    from paper_2607_21042_amd import ftts
    shape = workload.INDEXTTS2
    B, T = 32, 10
    P, Tt = workload.batch_lengths(B, seed=3)
    lens = [int(p) for p in P]
    budgets = [int(t) for t in Tt]
    inputs = workload.bf16_weights(big_master)
    flat = workload.prefix_embeddings(lens, shape.d_model, seed=1)
    prefixes = np.split(flat, np.cumsum(lens)[:-1])
    uni = workload.uniforms(int(Tt.max()), B, seed=2)[:T]
    say(f"paged batch 32 at 24 layers: prefixes {min(lens)}-{max(lens)}, upload")
    dm = ftts.DeviceModel(inputs, shape, ftts.BF16)
    bt, n_pages = scattered_table([n + T for n in lens], seed=7)
    lg, raw, hist = closed_loop(dm, shape, prefixes, budgets, T, uni, bt, n_pages)
    del dm
    say("  oracle")
    om = ogpt.GPT(inputs, shape.n_head, shape.d_head, dtype=np.float32)
    worst, near, n = check_closed_loop(om, shape, prefixes, budgets, uni, lg, raw, hist, "bf16")
    say(f"  worst abs err {worst:.3g}; sampled ids checked {n}, near-boundary {near}")


@pytest.mark.parametrize("mode,P", [("bf16", 256), ("w8a16", 256), ("w4a16", 384)])
def test_batch1_full_length(torch_cuda, big_master, mode, P):
    """Batch 1 at 24 layers for the full 512 greedy steps, teacher-forced on the
    oracle's own greedy tokens, with the benchmark's page table (identity pages,
    ceil((P + 512) / 64) of them), which makes the persistent step split each
    head's attention over two workgroups."""
    from paper_2607_21042_amd import ftts
    shape = workload.INDEXTTS2
    T = 512
    inputs = model_inputs(mode, big_master)
    prefix = workload.prefix_embeddings([P], shape.d_model, seed=1)
    say(f"batch 1 full length {mode} P={P}: oracle greedy decode")
    om = ogpt.GPT(helpers.oracle_weights(inputs, mode), shape.n_head, shape.d_head, dtype=np.float32)
    cache, _ = om.prefill(prefix)
    tok, ref, fed = shape.start_token, [], []
    for t in range(T):
        fed.append(tok)
        lg, _ = om.decode_step(cache, tok, t)
        ref.append(lg.astype(np.float32))
        tok = int(np.argmax(lg))
        if t % 128 == 127:
            say(f"  oracle step {t + 1}")
    ref = np.stack(ref)
    fed = np.array(fed, dtype=np.int32)[:, None]
    say("  gpu run")
    dm = ftts.DeviceModel(inputs, shape, wd(mode))
    assert ftts.decode_path(dm, 1) == 2
    max_pages = -(-(P + T) // 64)
    bt = np.arange(max_pages, dtype=np.int32)[None, :]
    res = helpers.run_gpu(dm, shape, [prefix], fed, block_table=bt, n_pages=max_pages)
    ftts.check_workspace(res["ws"])
    worst, near = 0.0, 0
    for t in range(T):
        ok, err = helpers.tolerance_ok(res["logits"][t, 0], ref[t], mode)
        worst = max(worst, err)
        assert ok, ("step", t, err)
        agree, is_near = helpers.argmax_agrees(res["sampled"][t, 0], ref[t], mode)
        near += is_near
        assert agree, ("argmax", t, int(res["sampled"][t, 0]), int(np.argmax(ref[t])))
    say(f"  worst abs err {worst:.3g} over {T} steps, near ties {near}")
