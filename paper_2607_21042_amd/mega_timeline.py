"""Per-phase timeline of the persistent decode step (batch 1).

    python -m paper_2607_21042_amd.build --trace
    python -m paper_2607_21042_amd.mega_timeline [--mode bf16|w8a16|w4a16] [--prefix 256] [--steps 64]

Runs a prefill and `--steps` greedy steps of the 24-layer IndexTTS-2-shaped GPT
(seeded random weights) on libftts_trace.so, whose step stamps the GPU's 100 MHz
wall clock at fixed points of every layer (thread 0 of wave 0 of every group,
and of the copy wave of the GEMV groups), and prints the medians of the last
step over layers 2-21, in microseconds from the layer's first barrier.
"""
from __future__ import annotations

import argparse
import ctypes
import os
import sys

import numpy as np

PKG = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(PKG))

from paper_2607_21042_amd import ftts, workload  # noqa: E402

MARKS_PER_LAYER, GROUPS = 20, 256
SLOTS = 1 + 50 * MARKS_PER_LAYER + 8
GEMV = ["P0 start", "x gathered", "LN1 done", "P1 start (q/k/v out)", "o gathered", "P3 start (x out)",
        "x gathered", "LN2 done", "P4 start (h out)", "h gathered", "FC2 out"]
COPY = ["P0", "q/k/v share in", "P1", "out-proj share in", "P3", "FC1 share in", "P4", "FC2 share in"]
ATTN = ["layer start", "q/k/v gathered", "wave 0 done", "output published"]


def main() -> None:
    p = argparse.ArgumentParser()
    p.add_argument("--mode", default="bf16", choices=["bf16", "w8a16", "w4a16"])
    p.add_argument("--prefix", type=int, default=256)
    p.add_argument("--steps", type=int, default=64)
    args = p.parse_args()
    ftts.LIB_PATH = os.path.join(PKG, "libftts_trace.so")
    L = ftts.lib()
    read = L.ftts_mega_trace_read
    read.argtypes = [ctypes.c_void_p, ctypes.c_size_t]
    read.restype = ctypes.c_int

    import torch
    shape = workload.INDEXTTS2
    wd = {"bf16": ftts.BF16, "w8a16": ftts.W8A16, "w4a16": ftts.W4A16}[args.mode]
    master = workload.master_weights(shape, seed=0)
    inputs = workload.bf16_weights(master) if args.mode == "bf16" else workload.quantisable_weights(master)
    dm = ftts.DeviceModel(inputs, shape, wd)
    assert ftts.decode_path(dm, 1) == 2, "the persistent step does not serve this model"
    P, T = args.prefix, args.steps
    prefix = torch.from_numpy(workload.prefix_embeddings([P], shape.d_model, seed=1)).cuda().to(torch.bfloat16)
    maxp = (P + T + 63) // 64
    bt = torch.arange(maxp, dtype=torch.int32, device="cuda").reshape(1, maxp)
    seq = torch.zeros(1, dtype=torch.int32, device="cuda")
    pt = ftts.PageTableView(bt, seq)
    pt.c = ftts.PageTable(bt.data_ptr(), seq.data_ptr(), maxp)
    kv = ftts.KVCache(shape, wd, maxp)
    ws = torch.empty(ftts.workspace_bytes(dm.cfg, 1, P), dtype=torch.uint8, device="cuda")
    last = torch.empty((1, shape.vocab), device="cuda")
    logits = torch.empty((1, shape.vocab), device="cuda")
    tok = torch.full((1,), shape.start_token, dtype=torch.int32, device="cuda")
    pos = torch.zeros(1, dtype=torch.int32, device="cuda")
    out = torch.empty(1, dtype=torch.int32, device="cuda")
    ftts.prefill(dm, prefix, [P], pt, kv, last, ws)
    seq.fill_(P)
    greedy = ftts.Sampling(1.0, 1, 1.0)
    for _ in range(T):
        ftts.decode_step(dm, tok, pos, pt, kv, logits, out, None, greedy, ws)
        torch.cuda.synchronize()
        tok.copy_(out)
        pos.add_(1)
        seq.add_(1)
    ftts.check_workspace(ws)

    buf = np.zeros((GROUPS, 2, SLOTS), dtype=np.uint64)
    if read(buf.ctypes.data, buf.nbytes) != 0:
        raise SystemExit("libftts_trace.so holds no timeline (build it with --trace)")
    n_att = 20
    tr = buf[:, 0].astype(np.int64)
    cw = buf[:, 1].astype(np.int64)
    nl = shape.n_layer
    layer = lambda t, g: t[g, 1:1 + nl * MARKS_PER_LAYER].reshape(nl, MARKS_PER_LAYER).astype(np.float64)
    print(f"# persistent step timeline, {args.mode}, prefix {P}, after {T} steps (context {P + T})")
    span = (tr[n_att:, 3 + nl * MARKS_PER_LAYER].max() - tr[:, 0].min()) / 100.0
    print(f"step span (first group's prologue end to the argmax): {span:.1f} us")
    gv = np.stack([layer(tr, g) for g in range(n_att, GROUPS)])       # [groups][layers][marks]
    rel = (gv - gv[:, :, :1]) / 100.0
    per_layer = (gv[:, 1:, 0] - gv[:, :-1, 0]) / 100.0
    print(f"layer period (median over GEMV groups, layers 2-21): {np.median(per_layer[:, 1:21]):.2f} us")
    med = np.median(rel[:, 2:22, :len(GEMV)], axis=(0, 1))
    print("\n| GEMV groups | us |\n|---|---|")
    for name, v in zip(GEMV, med):
        print(f"| {name} | {v:.2f} |")
    cv = np.stack([layer(cw, g) for g in range(n_att, GROUPS)])
    cmed = np.median((cv[:, 2:22, :len(COPY)] - gv[:, 2:22, :1]) / 100.0, axis=(0, 1))
    print("\n| copy wave | us |\n|---|---|")
    for name, v in zip(COPY, cmed):
        print(f"| {name} | {v:.2f} |")
    av = np.stack([layer(tr, g) for g in range(n_att)])
    amed = np.median((av[:, 2:22, :len(ATTN)] - np.median(gv[:, 2:22, :1], axis=0)[None]) / 100.0, axis=(0, 1))
    amax = np.median(np.max((av[:, 2:22, :len(ATTN)] - np.median(gv[:, 2:22, :1], axis=0)[None]) / 100.0, axis=0),
                     axis=0)
    print("\n| attention groups (from the GEMV groups' P0) | median us | slowest group us |\n|---|---|---|")
    for name, v, x in zip(ATTN, amed, amax):
        print(f"| {name} | {v:.2f} | {x:.2f} |")


if __name__ == "__main__":
    main()
