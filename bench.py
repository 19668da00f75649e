#!/usr/bin/env python3
"""Decode throughput of the IndexTTS-2-shaped GPT on one MI355X.

One bench step is one whole generation job: prefill of the conditioning
prefix, then `--decode` greedy decode steps for every sequence of the batch,
each step's sampled ids fed straight back as the next step's tokens (device to
device, no host round trip).  Inputs are seeded synthetic tensors resident in
HBM before timing starts.  The JSON line reports generated tokens per second
over the whole job, the HBM roofline of the decode step's dominant kernel, and
the CPU oracle's rate on a bounded sample of the same workload.

Roofline: when the persistent single-launch step serves the batch, that kernel
is the whole decode step and is timed per launch with HIP events on the stream
it runs on; otherwise the step (several kernels, replayed from a HIP graph) is
timed per replay.  `achieved` is the algorithmic bytes of a step divided by
that time.  `traffic` is the HBM bytes per launch measured by rocprofv3
counters (stored next to the kernel-trace summaries under profiles/), reported
only for the workload they were taken on and only while the kernel sources
are unchanged since.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "GPT decode tokens/s on 1 MI355X at batch 1 & 32; achieved HBM GB/s vs peak"
HBM_PEAK_GBS = 8000.0
EV_EVERY = 16  # persistent decode: timing events around every 16th step
COUNTERS = os.path.join(ROOT, "profiles", "decode_counters.json")


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=3, help="timed generation jobs")
    p.add_argument("--warmup", type=int, default=1)
    p.add_argument("--mode", default="bf16", choices=["bf16", "w8a16", "w4a16", "f32"])
    p.add_argument("--batch", type=int, default=1)
    p.add_argument("--prefix", type=int, default=256)
    p.add_argument("--decode", type=int, default=512)
    p.add_argument("--cpu-steps", type=int, default=512,
                   help="decode steps timed for the CPU oracle baseline (default: the whole 512-step run)")
    p.add_argument("--graph-steps", type=int, default=32, help="decode steps per HIP graph (kernel-per-phase path)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-legs", action="store_true",
                   help="headline workload only (by default the bf16 batch-1 run is followed by the W8A16 and "
                        "W4A16 batch-1, W8A16 batch-8 and batched paged batch-32 legs in the same JSON line)")
    p.add_argument("--paged", action="store_true",
                   help="the batched paged workload instead: --batch sequences (default 32) with prefix lengths "
                        "~U[128,512], targets ~U[256,768] then STOP, top-k 30 / top-p 0.8 / T 0.8 sampling")
    p.add_argument("--eager", action="store_true",
                   help="launch every kernel-per-phase decode step directly instead of replaying HIP graphs "
                        "(the counter runs)")
    p.add_argument("--serve", action="store_true",
                   help="continuous batching instead: --requests utterances (default 64) with the --paged length "
                        "mix through --batch decode slots (default 32), chunks of 16 steps, top-k 30 sampling")
    p.add_argument("--requests", type=int, default=64)
    p.add_argument("--dit", action="store_true",
                   help="flow-matching DiT (96M shape): guided Euler steps over --frames mel frames")
    p.add_argument("--frames", type=int, default=500, help="DiT: mel frames per utterance")
    p.add_argument("--dit-batch", type=int, default=1, help="DiT: utterances per step")
    p.add_argument("--euler", type=int, default=25, help="Euler steps per DiT job")
    p.add_argument("--graph", action="store_true", help="DiT: replay each job's steps from one HIP graph")
    p.add_argument("--copy-calibration", action="store_true",
                   help="only run a plain device copy of known size (scales the rocprofv3 byte counters)")
    return p.parse_args()


def copy_calibration():
    """Four plain device-to-device copies of 256 MiB each, one kernel apiece:
    a counter run over this gives FETCH_SIZE / WRITE_SIZE for known traffic."""
    import torch
    n = 256 << 20
    src = torch.ones(n // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(4):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration": {"bytes_read_per_copy": n, "bytes_written_per_copy": n, "copies": 4}}))


MEGA_SOURCES = ("decode_mega.hip", "ftts_internal.hpp", "gemv_impl.hpp", "kv_page.hpp")
BATCHED_SOURCES = ("bgemm.hip", "attention.hip", "misc.hip", "ftts.hip", "ftts_internal.hpp", "kv_page.hpp")


def kernel_sources_sha(files=MEGA_SOURCES) -> str:
    """Hash of the sources a decode path's kernels are built from."""
    csrc = os.path.join(ROOT, "paper_2607_21042_amd", "csrc")
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(fh.read())
    with open(os.path.join(ROOT, "include", "ftts.h"), "rb") as fh:
        h.update(fh.read())
    return h.hexdigest()


def measured_traffic(workload: str, sha: str):
    """HBM bytes per timed unit from the committed counter runs, if one was taken
    on this workload and the kernel sources are unchanged since."""
    try:
        with open(COUNTERS) as fh:
            entries = json.load(fh)["entries"]
    except (OSError, ValueError, KeyError):
        return None
    for c in entries:
        if c.get("workload") == workload and c.get("source_sha256") == sha:
            return c.get("hbm_bytes_per_unit")
    return None


def algorithmic_step_bytes(shape, dm, B, ctx_lens, kv_elem):
    """Bytes one decode step must move: every parameter once, the KV rows it
    attends over (the new one included), its KV writes, the embedding rows read
    and the fp32 logits written."""
    per_tok_kv = shape.n_layer * 2 * shape.d_model * kv_elem
    kv_read = sum(c + 1 for c in ctx_lens) * per_tok_kv
    kv_write = B * per_tok_kv
    emb = B * 2 * shape.d_model * kv_elem
    logits = B * shape.vocab * 4
    embed_tables = (shape.vocab + shape.n_pos) * shape.d_model * kv_elem  # read sparsely, not streamed
    return dm.weight_bytes() - embed_tables + kv_read + kv_write + emb + logits


def cpu_baseline(inputs, shape, mode, prefixes, n_steps, sampling=None, batch=None):
    """The numpy fp32 oracle, as it stands, on the host cores: an untimed prefill
    of each prefix, then n_steps decode steps per sequence, one sequence after
    another (greedy, or the oracle sampler with `sampling` = (T, k, p) and
    seeded uniforms), timed.  `batch` names the GPU batch the sample stands for."""
    import threadpoolctl
    from oracle import gpt as ogpt
    from oracle import quant as oquant
    from oracle import sample as osample

    cores = len(os.sched_getaffinity(0))
    with threadpoolctl.threadpool_limits(cores):
        w = inputs if mode in ("f32", "bf16") else oquant.dequantized_model(
            inputs, "w8" if mode == "w8a16" else "w4")
        om = ogpt.GPT(w, shape.n_head, shape.d_head, dtype=np.float32)
        caches = [om.prefill(p)[0] for p in prefixes]
        uni = np.random.default_rng(2).random((n_steps, len(prefixes)), dtype=np.float32)
        t0 = time.perf_counter()
        for b, cache in enumerate(caches):
            tok = shape.start_token
            for t in range(n_steps):
                logits, _ = om.decode_step(cache, tok, t)
                if sampling is None:
                    tok = int(np.argmax(logits))
                else:
                    tok = osample.sample(logits.astype(np.float32), *sampling, uni[t, b])[0]
        dt = time.perf_counter() - t0
        used = max((i.get("num_threads", 1) for i in threadpoolctl.threadpool_info()), default=1)
    n_tok = n_steps * len(prefixes)
    how = "greedy" if sampling is None else "top-k {1} / top-p {2} / T {0} sampled".format(*sampling)
    lens = sorted({p.shape[0] for p in prefixes})
    sample = (f"{n_steps} {how} decode steps of {len(prefixes)} sequence(s) after an untimed prefill of "
              f"{'/'.join(str(x) for x in lens)} rows, numpy fp32 oracle on the same {mode} weights")
    if batch is not None and batch != len(prefixes):
        sample += f" (the oracle runs sequences one at a time: its rate for the batch of {batch} is the same)"
    return {"value": round(n_tok / dt, 3), "unit": "tokens/s", "cores": int(min(used, cores)), "kind": "oracle",
            "sample": sample}


MFMA_BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 matrix peak


def prefill_report(shape, lens, ms):
    """Prefill throughput against the dense bf16 matrix peak: the four linears
    of every layer over all prefix rows, causal attention (Q K^T and P V over
    the lower triangle) and the LM head on each sequence's last row."""
    d, F, H = shape.d_model, shape.d_ff, shape.n_head
    rows = int(sum(lens))
    lin = 2 * rows * (3 * d * d + d * d + 2 * d * F)
    att = sum(2 * 2 * (int(p) * (int(p) + 1) // 2) * shape.d_head * H for p in lens)
    flops = shape.n_layer * (lin + att) + 2 * len(lens) * d * shape.vocab
    tflops = flops / (ms / 1e3) / 1e12
    return {"ms": round(ms, 3), "rows": rows, "gflop": round(flops / 1e9, 1), "tflops": round(tflops, 1),
            "peak_tflops": MFMA_BF16_PEAK_TFLOPS, "mfma_frac": round(tflops / MFMA_BF16_PEAK_TFLOPS, 4)}


def paged_batch(args, torch, ftts, workload, shape, dm, mode, wdtype, inputs):
    """The batched paged workload: one job = ragged prefill of every sequence, then
    decode steps until every sequence has produced its target length (the last
    token forced to STOP), sampling with host uniforms.  The decode steps are
    replayed from HIP graphs of 32 steps; tokens/s counts only tokens of active
    sequences."""
    B = args.batch
    P, Tt = workload.batch_lengths(B, seed=3)
    T_max = int(Tt.max())
    adt = ftts.act_dtype(wdtype)
    prefix = torch.from_numpy(workload.prefix_embeddings(P.tolist(), shape.d_model, seed=1,
                                                         bf16=(mode != "f32"))).cuda().to(adt)
    need = [math.ceil((int(p) + int(t)) / 64) for p, t in zip(P, Tt)]
    max_pages = max(need)
    n_pages = sum(need)
    perm = np.random.default_rng(7).permutation(n_pages)  # pages of a shared pool, scattered
    bt_np = np.full((B, max_pages), -1, np.int32)
    k = 0
    for b, n in enumerate(need):
        bt_np[b, :n] = perm[k:k + n]
        k += n
    bt = torch.from_numpy(bt_np).cuda()
    kv = ftts.KVCache(shape, wdtype, n_pages)
    logits = torch.empty((B, shape.vocab), dtype=torch.float32, device="cuda")
    last = torch.empty((B, shape.vocab), dtype=torch.float32, device="cuda")
    ws = torch.empty(ftts.workspace_bytes(dm.cfg, B, int(P.sum())), dtype=torch.uint8, device="cuda")
    samp = ftts.Sampling(0.8, 30, 0.8)
    uni = torch.from_numpy(workload.uniforms(T_max, B, seed=2)).cuda()
    tokens = torch.empty(B, dtype=torch.int32, device="cuda")
    positions = torch.empty(B, dtype=torch.int32, device="cuda")
    seq_lens = torch.empty(B, dtype=torch.int32, device="cuda")
    sampled = torch.empty(B, dtype=torch.int32, device="cuda")
    remaining = torch.empty(B, dtype=torch.int32, device="cuda")
    history = torch.empty((T_max, B), dtype=torch.int32, device="cuda")
    counter = torch.empty(1, dtype=torch.int32, device="cuda")
    pt = ftts.PageTableView(bt, seq_lens)
    pt.seq_lens = seq_lens
    pt.c = ftts.PageTable(bt.data_ptr(), seq_lens.data_ptr(), max_pages)
    P_dev = torch.from_numpy(P).cuda()
    T_dev = torch.from_numpy(Tt).cuda()

    def reset_and_prefill(pev=None):
        tokens.fill_(shape.start_token)
        positions.zero_()
        seq_lens.copy_(P_dev)
        remaining.copy_(T_dev)
        counter.zero_()
        if pev is not None:
            pev[0].record(torch.cuda.current_stream())
        ftts.prefill(dm, prefix, P.tolist(), pt, kv, last, ws)
        if pev is not None:
            pev[1].record(torch.cuda.current_stream())

    def step(t):
        ftts.decode_step(dm, tokens, positions, pt, kv, logits, sampled, uni[t], samp, ws)
        ftts.advance(tokens, positions, seq_lens, sampled, remaining, shape.stop_token, history, counter)

    reset_and_prefill()
    step(0)
    torch.cuda.synchronize()
    # One graph per --graph-steps steps (each step reads its own row of uniforms):
    # a graph of every step would be a single chain of ~94k kernel nodes, beyond
    # the cap on steps per graph.
    S = ftts.graph_steps(args.graph_steps)
    graphs = []
    for g0 in range(0, T_max if not args.eager else 0, S):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for t in range(g0, min(g0 + S, T_max)):
                step(t)
        graphs.append(g)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()

    class _All:
        def replay(self):
            if args.eager:
                for t in range(T_max):
                    step(t)
            for g in graphs:
                g.replay()
    graph = _All()
    for _ in range(args.warmup):
        reset_and_prefill()
        graph.replay()
    torch.cuda.synchronize()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    pevs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    wall0 = time.perf_counter()
    t0.record(stream)
    for k in range(args.steps):
        reset_and_prefill(pevs[k])
        evs[k][0].record(stream)
        graph.replay()
        evs[k][1].record(stream)
    t1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    hist = history.cpu().numpy()
    assert all(hist[int(Tt[b]) - 1, b] == shape.stop_token for b in range(B)), "STOP not forced"
    job_ms = t0.elapsed_time(t1) / args.steps
    decode_ms = float(np.mean([a.elapsed_time(b) for a, b in evs]))
    n_tok = int(Tt.sum())
    kv_elem = 4 if mode == "f32" else 2
    per_tok_kv = shape.n_layer * 2 * shape.d_model * kv_elem
    weights = dm.weight_bytes() - (shape.vocab + shape.n_pos) * shape.d_model * kv_elem
    total_bytes = 0.0
    for t in range(T_max):
        act = Tt > t
        total_bytes += weights + int(((P + t + 1) * act).sum()) * per_tok_kv + int(act.sum()) * (
            per_tok_kv + 2 * shape.d_model * kv_elem + shape.vocab * 4)
    achieved = total_bytes / (decode_ms / 1e3) / 1e9
    workload_name = (f"indextts2-gpt {mode} paged batch={B} prefix~U[128,512] target~U[256,768]+STOP "
                     f"top-k 30 top-p 0.8 T 0.8")
    out = {
        "metric": METRIC, "value": round(n_tok / (job_ms / 1e3), 2), "unit": "tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(job_ms, 3), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": {"f32": "f32", "bf16": "bf16", "w8a16": "int8-w/bf16",
                                                          "w4a16": "int4-w/bf16"}[mode],
        "data": "synthetic: seeded random-init IndexTTS-2-shaped GPT; paged KV from a shared pool",
        "config": {"workload": workload_name, "batch": B, "tokens": n_tok, "decode_steps": T_max,
                   "decode_path": "kernel-per-phase" if ftts.decode_path(dm, B) == 1 else "persistent"},
        "decode_tokens_per_s": round(n_tok / (decode_ms / 1e3), 2),
        "decode_ms_per_step": round(decode_ms / T_max, 4),
        "prefill_ms": round(job_ms - decode_ms, 3),
        "prefill": prefill_report(shape, P, float(np.mean([a.elapsed_time(b) for a, b in pevs]))),
        "wall_s": round(wall, 3),
        "roofline": {"bound": "hbm", "kernel": (f"decode step, kernel per phase ({T_max} steps, "
                                                + ("launched eagerly)" if args.eager else f"{S} per HIP graph)")),
                     "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "algorithmic_bytes_per_step": int(total_bytes / T_max),
                     "traffic": measured_traffic(workload_name, kernel_sources_sha(BATCHED_SOURCES))},
    }
    if not args.no_cpu_baseline:
        flat = workload.prefix_embeddings(P[:2].tolist(), shape.d_model, seed=1, bf16=(mode != "f32"))
        seqs = np.split(flat, [int(P[0])])
        out["cpu_baseline"] = cpu_baseline(inputs, shape, mode, seqs, 64, sampling=(0.8, 30, 0.8), batch=B)
    return out


def serve_run(args, torch, ftts, workload, shape, dm, mode):
    """Continuous batching: more utterances than decode slots, admitted as slots
    and pages free up; ids streamed in chunks.  Times whole runs (prefills,
    decode chunks and the host's bookkeeping between them)."""
    from paper_2607_21042_amd import serve
    R, S = args.requests, args.batch
    P, Tt = workload.batch_lengths(R, seed=3)
    flat = workload.prefix_embeddings(P.tolist(), shape.d_model, seed=1, bf16=(mode != "f32"))
    prefixes = np.split(flat, np.cumsum(P)[:-1])
    uni = workload.uniforms(int(Tt.max()), R, seed=2)
    max_ctx = int((P + Tt).max())
    n_pages = S * ((max_ctx + 63) // 64) + 8
    samp = ftts.Sampling(0.8, 30, 0.8)

    def one_run():
        sch = serve.Scheduler(dm, shape, max_slots=S, n_pages=n_pages, max_ctx=max_ctx, sampling=samp, chunk=16,
                              overlap=4, max_prefill_rows=S * 512)
        reqs = [sch.submit(serve.Request(prefix=p, max_new=int(t), uniforms=uni[:, i]))
                for i, (p, t) in enumerate(zip(prefixes, Tt))]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        sch.run()
        torch.cuda.synchronize()
        dt = time.perf_counter() - t0
        assert all(r.done and len(r.tokens) == r.max_new and r.tokens[-1] == shape.stop_token for r in reqs)
        return dt, sch.n_chunks

    for _ in range(args.warmup):
        one_run()
    runs = [one_run() for _ in range(args.steps)]
    dt = float(np.mean([r[0] for r in runs]))
    n_tok = int(Tt.sum())
    return {
        "metric": METRIC, "value": round(n_tok / dt, 2), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(dt * 1e3, 3), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": {"f32": "f32", "bf16": "bf16", "w8a16": "int8-w/bf16",
                                       "w4a16": "int4-w/bf16"}[mode],
        "data": "synthetic: seeded random-init IndexTTS-2-shaped GPT; continuous batching over a shared page pool",
        "config": {"workload": f"indextts2-gpt {mode} continuous batching: {R} utterances, {S} slots, "
                               f"prefix~U[128,512] target~U[256,768]+STOP, chunks of 16 (overlap 4), "
                               f"top-k 30 top-p 0.8 T 0.8", "requests": R, "slots": S, "tokens": n_tok,
                   "chunks": runs[-1][1]},
        "wall_s": round(dt, 3),
    }


def dit_flops(shape, lens):
    """Algorithmic flops of one guided Euler step over utterances of `lens` frames
    (both branches): 2 M N K per linear at M = 2 sum(lens) rows, 4 T^2 d per
    block, branch and utterance of T frames for the attention (Q K^T and P V),
    and the M-independent time MLP."""
    M, d = 2 * sum(lens), shape.d_model
    lin = sum(N * K for _, N, K in shape.matrices()) * shape.n_layer + d * (shape.n_mel + shape.d_cond) \
        + shape.n_mel * d
    att = sum(4.0 * T * T * d for T in lens)
    return 2.0 * M * lin + shape.n_layer * 2 * att + 2.0 * (d * shape.t_dim + d * d)


def dit_run(args, torch, ftts, workload):
    """One job = --euler guided Euler steps of the 96M DiT for --dit-batch
    utterances of --frames frames each (t from 0 to 1 in equal steps), state and
    conditioning resident in HBM."""
    shape = workload.DIT_96M
    T, K, B = args.frames, args.euler, args.dit_batch
    lens = [T] * B
    w = workload.bf16_weights(workload.dit_master_weights(shape, seed=20))
    dm = ftts.DitDeviceModel(w, shape)
    x0_np, cond_np = workload.dit_inputs(shape, T * B, seed=21)
    x0 = torch.from_numpy(x0_np).cuda()
    x = torch.empty_like(x0)
    cond = torch.from_numpy(cond_np).cuda().to(torch.bfloat16)
    ws = torch.empty(ftts.dit_workspace_bytes(dm.cfg, T * B), dtype=torch.uint8, device="cuda")
    stream = torch.cuda.current_stream()
    cfg_w, dt = 1.7, 1.0 / K

    def solve(evs=None):
        x.copy_(x0)
        for k in range(K):
            if evs is not None:
                evs[k][0].record(stream)
            ftts.dit_step(dm, x, cond, k * dt, dt, cfg_w, x, None, ws, lens=lens)
            if evs is not None:
                evs[k][1].record(stream)

    graph = None
    if args.graph:
        solve()
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            solve()
    for _ in range(args.warmup):
        if graph:
            graph.replay()
        else:
            solve()
    torch.cuda.synchronize()
    evs = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(K)]
           for _ in range(args.steps)]
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    wall0 = time.perf_counter()
    t0.record(stream)
    for j in range(args.steps):
        if graph:
            graph.replay()
        else:
            solve(evs[j])
    t1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    job_ms = t0.elapsed_time(t1) / args.steps
    step_ms = job_ms / K if graph else float(np.mean([[a.elapsed_time(b) for a, b in r] for r in evs]))
    fl = dit_flops(shape, lens)
    achieved = fl / (step_ms / 1e3) / 1e12
    peak = 2500.0
    out = {
        "metric": "DiT guided Euler steps/s on 1 MI355X (96M flow-matching DiT); achieved TFLOP/s vs bf16 MFMA peak",
        "value": round(1e3 / step_ms, 2), "unit": "steps/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(job_ms, 3), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic: seeded random-init 96M DiT (13x768, 12 heads, FFN 3072, 128 mel, cond 1280)",
        "config": {"workload": f"dit-96m bf16 batch={B} frames={T} euler={K} cfg both branches in one batch",
                   "batch": B, "frames": T, "euler_steps": K, "graph": bool(graph)},
        "ms_per_euler_step": round(step_ms, 4),
        "frames_per_s": round(B * T * 1e3 / step_ms, 1),
        "wall_s": round(wall, 3),
        "roofline": {"bound": "mfma", "kernel": "whole guided Euler step (GEMMs, attention, LayerNorms)",
                     "achieved": round(achieved, 2), "peak": peak, "unit": "TFLOP/s",
                     "frac": round(achieved / peak, 4), "flops_per_step": fl, "traffic": None},
    }
    if not args.no_cpu_baseline:
        import threadpoolctl
        from oracle import dit as odit
        cores = len(os.sched_getaffinity(0))
        with threadpoolctl.threadpool_limits(cores):
            ora = odit.DiT(w, shape.n_head, shape.d_head, dtype=np.float64)
            c0 = time.perf_counter()
            ora.step(x0_np[:T], cond_np[:T], 0.0, dt, cfg_w)  # one utterance; the rate below scales by B
            cpu_s = (time.perf_counter() - c0) * B
            used = max((i.get("num_threads", 1) for i in threadpoolctl.threadpool_info()), default=1)
        out["cpu_baseline"] = {"value": round(1.0 / cpu_s, 4), "unit": "steps/s", "cores": int(min(used, cores)),
                               "kind": "oracle", "sample": f"one guided Euler step of one {T}-frame utterance, "
                                                           f"numpy fp64 oracle on the same bf16 weights, "
                                                           f"scaled to the batch of {B}"}
    return out


DTYPE_NAMES = {"f32": "f32", "bf16": "bf16", "w8a16": "int8-w/bf16", "w4a16": "int4-w/bf16"}


def model_inputs(workload, master, mode):
    if mode == "f32":
        return master
    if mode == "bf16":
        return workload.bf16_weights(master)
    return workload.quantisable_weights(master)


def fixed_batch(torch, ftts, workload, shape, inputs, mode, B, P, T, steps, warmup, graph_steps=32,
                cpu_steps=0, cpu_seqs=1, eager=False):
    """B sequences with the same prefix length P, T greedy steps each; one job =
    prefill + T steps with the sampled ids fed back on the device.  The
    persistent step is timed per launch; the kernel-per-phase step per graph
    replay of `graph_steps` steps."""
    wdtype = {"f32": ftts.F32, "bf16": ftts.BF16, "w8a16": ftts.W8A16, "w4a16": ftts.W4A16}[mode]
    dm = ftts.DeviceModel(inputs, shape, wdtype)
    adt = ftts.act_dtype(wdtype)
    prefix_np = workload.prefix_embeddings([P] * B, shape.d_model, seed=1, bf16=(mode != "f32"))
    prefix = torch.from_numpy(prefix_np).cuda().to(adt)

    max_pages = math.ceil((P + T) / 64)
    n_pages = B * max_pages
    bt = torch.arange(n_pages, dtype=torch.int32, device="cuda").reshape(B, max_pages)
    kv = ftts.KVCache(shape, wdtype, n_pages)
    logits = torch.empty((B, shape.vocab), dtype=torch.float32, device="cuda")
    last = torch.empty((B, shape.vocab), dtype=torch.float32, device="cuda")
    ws = torch.empty(ftts.workspace_bytes(dm.cfg, B, B * P), dtype=torch.uint8, device="cuda")
    greedy = ftts.Sampling(1.0, 1, 1.0)
    # Generation state; every decode step reads and updates it on the device.
    tokens = torch.empty(B, dtype=torch.int32, device="cuda")
    positions = torch.empty(B, dtype=torch.int32, device="cuda")
    seq_lens = torch.empty(B, dtype=torch.int32, device="cuda")
    sampled = torch.empty(B, dtype=torch.int32, device="cuda")
    history = torch.empty((T, B), dtype=torch.int32, device="cuda")
    counter = torch.empty(1, dtype=torch.int32, device="cuda")
    pt = ftts.PageTableView(bt, seq_lens)
    pt.seq_lens = seq_lens  # keep the same storage: the graph reads these pointers
    pt.c = ftts.PageTable(bt.data_ptr(), seq_lens.data_ptr(), max_pages)
    persistent = ftts.decode_path(dm, B) == 2
    # kernel-per-phase steps replay HIP graphs unless `eager` (counter runs)
    direct = persistent or eager
    # Launch timing: an event pair around every EV_EVERY-th directly launched step
    # (a pair on every step adds ~6 us per step to the whole job), around every
    # replay on the graph path.
    ev_every = EV_EVERY if direct else 1

    def reset():
        tokens.fill_(shape.start_token)
        positions.zero_()
        seq_lens.fill_(P)
        counter.zero_()

    def step_kernel():
        ftts.decode_step(dm, tokens, positions, pt, kv, logits, sampled, None, greedy, ws)

    def step_advance():
        ftts.advance(tokens, positions, seq_lens, sampled, None, shape.stop_token, history, counter)

    stream = torch.cuda.current_stream()
    S = 1
    graph = None
    reset()
    ftts.prefill(dm, prefix, [P] * B, pt, kv, last, ws)
    for _ in range(2):
        step_kernel()
        step_advance()
    torch.cuda.synchronize()
    if not direct:
        # several kernels per step: capture S steps into one graph
        S = ftts.graph_steps(graph_steps) if T % graph_steps == 0 else 1
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for _ in range(S):
                step_kernel()
                step_advance()
        torch.cuda.synchronize()

    def job(evs=None, pev=None):
        reset()
        if pev is not None:
            pev[0].record(stream)
        ftts.prefill(dm, prefix, [P] * B, pt, kv, last, ws)
        if pev is not None:
            pev[1].record(stream)
        if direct:
            for t in range(T):
                timed = evs is not None and t % ev_every == 0
                if timed:
                    evs[t // ev_every][0].record(stream)
                step_kernel()
                if timed:
                    evs[t // ev_every][1].record(stream)
                step_advance()
        else:
            for r in range(T // S):
                if evs is not None:
                    evs[r][0].record(stream)
                graph.replay()
                if evs is not None:
                    evs[r][1].record(stream)

    for _ in range(warmup):
        job()
    torch.cuda.synchronize()
    n_units = len(range(0, T, ev_every)) if direct else T // S
    evs = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n_units)]
           for _ in range(steps)]
    pevs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    t_start.record(stream)
    for k in range(steps):
        job(evs[k], pevs[k])
    t_end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    if persistent:
        ftts.check_workspace(ws)
    total_ms = t_start.elapsed_time(t_end)
    job_ms = total_ms / steps
    value = B * T / (job_ms / 1e3)

    kv_elem = 4 if mode == "f32" else 2
    step_bytes = np.array([algorithmic_step_bytes(shape, dm, B, [P + t] * B, kv_elem) for t in range(T)], np.float64)
    unit_ms = np.array([[a.elapsed_time(b) for a, b in row] for row in evs], np.float64)  # [steps][units]
    if persistent:
        unit_bytes = step_bytes[::ev_every]
        kernel = "decode_mega_kernel (persistent single-launch decode step)"
        sha = kernel_sources_sha(MEGA_SOURCES)
    elif eager:
        unit_bytes = step_bytes[::ev_every]
        kernel = "decode step, kernel per phase (launched eagerly)"
        sha = None  # the committed counters are per graph replay
    else:
        unit_bytes = step_bytes.reshape(T // S, S).sum(axis=1)
        kernel = f"decode step, kernel per phase ({S} steps per graph replay)"
        sha = kernel_sources_sha(BATCHED_SOURCES)
    launch_us = float(unit_ms.mean() * 1e3)
    achieved = float(unit_bytes.sum() * steps / (unit_ms.sum() / 1e3) / 1e9)
    # decode time per job: the timed launches' mean times the step count (persistent)
    decode_ms = float(unit_ms.mean() * T) if direct else float(unit_ms.sum(axis=1).mean())
    workload_name = f"indextts2-gpt {mode} batch={B} prefix={P} greedy decode={T}"
    out = {
        "metric": METRIC, "value": round(value, 2), "unit": "tokens/s", "n_gpus": 1, "steps": steps,
        "warmup": warmup, "ms_per_step": round(job_ms, 3), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": DTYPE_NAMES[mode],
        "data": "synthetic: seeded random-init IndexTTS-2-shaped GPT (24x1280, 20 heads, FFN 5120, vocab 8194)",
        "config": {"workload": workload_name, "batch": B, "prefix": P, "decode_tokens": T, "weights": mode,
                   "decode_path": "persistent" if persistent else "kernel-per-phase"},
        "decode_tokens_per_s": round(B * T / (decode_ms / 1e3), 2),
        "decode_ms_per_token_step": round(decode_ms / T, 4),
        "prefill_ms": round(job_ms - decode_ms, 3),
        "prefill": prefill_report(shape, [P] * B, float(np.mean([a.elapsed_time(b) for a, b in pevs]))),
        "wall_s": round(wall, 3),
        "roofline": {"bound": "hbm", "kernel": kernel, "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "launch_us": round(launch_us, 2),
                     "launches_timed_per_job": n_units,
                     "algorithmic_bytes_per_launch": int(unit_bytes.mean()),
                     "traffic": measured_traffic(workload_name, sha)},
    }
    del dm, kv, ws
    torch.cuda.empty_cache()
    if cpu_steps > 0:
        seqs = [prefix_np[b * P:(b + 1) * P] for b in range(min(cpu_seqs, B))]
        out["cpu_baseline"] = cpu_baseline(inputs, shape, mode, seqs, cpu_steps, batch=B)
    return out


LEG_KEYS = ("config", "dtype", "value", "unit", "ms_per_step", "decode_tokens_per_s", "decode_ms_per_token_step",
            "decode_ms_per_step", "prefill_ms", "prefill", "roofline", "cpu_baseline", "steps", "warmup")


def legs(args, torch, ftts, workload, shape, master):
    """The rest of the metric, measured in the same run after the headline:
    W8A16 and W4A16 at batch 1, W8A16 at batch 8, and the batched paged
    workload at batch 32.  Each leg is a few whole jobs (prefill + all decode
    steps) after one untimed job."""
    out = {}
    for name, mode, B, P in (("w8a16_b1", "w8a16", 1, 256), ("w4a16_b1", "w4a16", 1, 384),
                             ("w8a16_b8", "w8a16", 8, 256)):
        t0 = time.perf_counter()
        inputs = model_inputs(workload, master, mode)
        r = fixed_batch(torch, ftts, workload, shape, inputs, mode, B, P, 512, steps=3, warmup=1,
                        cpu_steps=0 if args.no_cpu_baseline else 64, cpu_seqs=1 if B == 1 else 2)
        r["leg_wall_s"] = round(time.perf_counter() - t0, 1)
        out[name] = {k: r[k] for k in LEG_KEYS + ("leg_wall_s",) if k in r}
        print(f"leg {name}: {r['value']} tokens/s, {r['decode_ms_per_token_step']} ms per step",
              file=sys.stderr, flush=True)
        del inputs
    t0 = time.perf_counter()
    inputs = workload.bf16_weights(master)
    dm = ftts.DeviceModel(inputs, shape, ftts.BF16)
    pa = argparse.Namespace(**vars(args))
    pa.batch, pa.steps, pa.warmup = 32, 2, 1
    r = paged_batch(pa, torch, ftts, workload, shape, dm, "bf16", ftts.BF16, inputs)
    del dm
    torch.cuda.empty_cache()
    r["leg_wall_s"] = round(time.perf_counter() - t0, 1)
    out["bf16_b32_paged"] = {k: r[k] for k in LEG_KEYS + ("leg_wall_s",) if k in r}
    print(f"leg bf16_b32_paged: {r['value']} tokens/s", file=sys.stderr, flush=True)
    return out


def main():
    args = parse()
    if args.copy_calibration:
        copy_calibration()
        return
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on exactly one GPU; --gpus must be 1",
                          "n_gpus": args.gpus}))
        sys.exit(2)
    import torch
    from paper_2607_21042_amd import ftts, workload

    try:
        ftts.graph_steps(args.graph_steps)
    except ValueError as e:
        print(json.dumps({"error": str(e)}))
        sys.exit(2)
    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU visible"}))
        sys.exit(1)
    if args.dit:
        print(json.dumps(dit_run(args, torch, ftts, workload)), flush=True)
        return
    shape = workload.INDEXTTS2
    mode = args.mode
    wdtype = {"f32": ftts.F32, "bf16": ftts.BF16, "w8a16": ftts.W8A16, "w4a16": ftts.W4A16}[mode]
    master = workload.master_weights(shape, seed=0)
    inputs = model_inputs(workload, master, mode)
    if args.paged or args.serve:
        dm = ftts.DeviceModel(inputs, shape, wdtype)
        if args.batch == 1:
            args.batch = 32
        if args.paged:
            r = paged_batch(args, torch, ftts, workload, shape, dm, mode, wdtype, inputs)
        else:
            r = serve_run(args, torch, ftts, workload, shape, dm, mode)
        print(json.dumps(r), flush=True)
        return
    out = fixed_batch(torch, ftts, workload, shape, inputs, mode, args.batch, args.prefix, args.decode, args.steps,
                      args.warmup, graph_steps=args.graph_steps,
                      cpu_steps=0 if args.no_cpu_baseline else args.cpu_steps, eager=args.eager)
    headline = mode == "bf16" and args.batch == 1 and args.prefix == 256 and args.decode == 512
    if headline and not args.no_legs:
        out["legs"] = legs(args, torch, ftts, workload, shape, master)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
