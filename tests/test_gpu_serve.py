"""GPU: continuous batching (paper_2607_21042_amd.serve) over the C ABI.

More requests than decode slots, so requests are admitted while others decode;
every request's ids are checked against the oracle teacher-forced on the ids the
GPU produced (argmax equal away from near-ties), its hidden states against the
oracle's, its budget against the forced STOP, its streamed windows against its
ids, and every page must come back to the pool.
"""
import sys

import numpy as np
import pytest

from oracle import gpt as ogpt
from paper_2607_21042_amd import workload
from tests import helpers

pytestmark = pytest.mark.gpu


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.mark.parametrize("mode,slots,graphs", [("f32", 3, False), ("f32", 3, True), ("bf16", 3, True),
                                               ("bf16", 9, True)])
def test_continuous_batching_matches_oracle(mode, slots, graphs):
    import torch
    from paper_2607_21042_amd import ftts, serve
    assert torch.cuda.is_available()
    shape = workload.TINY
    master = workload.master_weights(shape, seed=0)
    inputs = master if mode == "f32" else workload.bf16_weights(master)
    wdt = ftts.F32 if mode == "f32" else ftts.BF16
    dm = ftts.DeviceModel(inputs, shape, wdt)
    om = ogpt.GPT(helpers.oracle_weights(inputs, mode), shape.n_head, shape.d_head, dtype=np.float32)
    lens = [40, 1, 70, 129, 5, 33, 64, 17, 90, 2, 48, 11]
    budgets = [10, 25, 7, 12, 30, 3, 9, 14, 5, 21, 6, 13]
    flat = workload.prefix_embeddings(lens, shape.d_model, seed=1, bf16=(mode != "f32"))
    prefixes = np.split(flat, np.cumsum(lens)[:-1])
    n_pages = 3 * slots + 4                      # tight enough that admission sometimes waits for pages
    sch = serve.Scheduler(dm, shape, max_slots=slots, n_pages=n_pages, max_ctx=max(lens) + max(budgets),
                          sampling=ftts.Sampling(1.0, 1, 1.0), chunk=4, overlap=1, hidden=True, graphs=graphs)
    reqs = [sch.submit(serve.Request(prefix=p, max_new=n)) for p, n in zip(prefixes, budgets)]
    say(f"serve {mode} slots={slots} graphs={graphs}")
    sch.run()
    assert not sch.busy()
    assert len(sch.pool.free) == n_pages
    assert any(r.admitted_at > 0 for r in reqs)
    near = 0
    for r, p in zip(reqs, prefixes):
        assert r.done and len(r.tokens) == r.max_new, (r.rid, len(r.tokens))
        assert r.tokens[-1] == shape.stop_token
        fed = np.array([shape.start_token] + r.tokens[:-1], dtype=np.int32)
        _, ref, ref_hid = helpers.oracle_teacher_forced(om, p, fed, with_hidden=True)
        for j in range(r.max_new - 1):             # the last id is the forced STOP
            ok, is_near = helpers.argmax_agrees(r.tokens[j], ref[j], mode)
            near += is_near
            assert ok, (r.rid, j, r.tokens[j], int(np.argmax(ref[j])))
        for j in range(r.max_new):
            ok, err = helpers.tolerance_ok(r.hidden[j], ref_hid[j], mode)
            assert ok, ("hidden", r.rid, j, err)
        # streamed windows: each repeats `overlap` ids of the previous one and they tile the ids
        joined = []
        for w0, ids in r.chunks:
            assert w0 == max(0, len(joined) - 1)
            np.testing.assert_array_equal(ids[:len(joined) - w0], joined[w0:])
            joined = joined[:w0] + list(ids)
        assert joined == r.tokens
    say(f"  {sch.n_chunks} chunks, near ties {near}")


def test_requests_end_at_a_sampled_stop_code():
    """With stop_on_token a request ends at the first stop code it samples (the
    slot is freed on the device at that step and its pages come back), before
    its budget; requests that never sample it run to the forced STOP.  The stop
    code here is an id the same requests produced in a first run, so several of
    them meet it early; every id is checked against the oracle as above."""
    import dataclasses
    import torch
    from paper_2607_21042_amd import ftts, serve
    shape = workload.TINY
    inputs = workload.bf16_weights(workload.master_weights(shape, seed=0))
    dm = ftts.DeviceModel(inputs, shape, ftts.BF16)
    om = ogpt.GPT(helpers.oracle_weights(inputs, "bf16"), shape.n_head, shape.d_head, dtype=np.float32)
    lens = [40, 9, 70, 33, 64, 17]
    budgets = [24, 24, 24, 24, 24, 24]
    flat = workload.prefix_embeddings(lens, shape.d_model, seed=1, bf16=True)
    prefixes = np.split(flat, np.cumsum(lens)[:-1])

    def run(stop_on, stop):
        sch = serve.Scheduler(dm, shape, max_slots=3, n_pages=16, max_ctx=max(lens) + max(budgets),
                              sampling=ftts.Sampling(1.0, 1, 1.0), chunk=4, overlap=0, graphs=True,
                              stop_on_token=stop_on, stop_token=stop)
        reqs = [sch.submit(serve.Request(prefix=p, max_new=n)) for p, n in zip(prefixes, budgets)]
        sch.run()
        assert not sch.busy() and len(sch.pool.free) == 16
        return reqs

    first = run(False, None)
    # the id met earliest (over the first half of the budgets) by the most requests
    counts = {}
    for r in first:
        for t in set(r.tokens[:12]):
            counts[t] = counts.get(t, 0) + 1
    stop = max(sorted(counts), key=lambda t: counts[t])
    say(f"stop code {stop}: met by {counts[stop]} of {len(first)} requests in their first 12 ids")
    reqs = run(True, stop)
    early = 0
    for r, p in zip(reqs, prefixes):
        assert r.done and 1 <= len(r.tokens) <= r.max_new
        assert r.tokens[-1] in (stop, shape.stop_token)
        assert stop not in r.tokens[:-1], (r.rid, r.tokens)
        if len(r.tokens) < r.max_new:
            early += 1
            assert r.tokens[-1] == stop
        else:
            assert r.tokens[-1] in (stop, shape.stop_token)
        fed = np.array([shape.start_token] + r.tokens[:-1], dtype=np.int32)
        _, ref, _ = helpers.oracle_teacher_forced(om, p, fed, with_hidden=True)
        n_check = len(r.tokens) if len(r.tokens) < r.max_new else r.max_new - 1
        for j in range(n_check):
            ok, _ = helpers.argmax_agrees(r.tokens[j], ref[j], "bf16")
            assert ok, (r.rid, j, r.tokens[j], int(np.argmax(ref[j])))
    assert early >= 1
    say(f"  {early} of {len(reqs)} requests ended at the sampled stop code")
