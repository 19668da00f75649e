"""Continuous batching of the GPT decode step with chunked streaming output.

The serving engine batches utterances in flight (Sec. II-C: the GPT runs on an
engine with in-flight batching) and streams semantic tokens downstream in
chunks of a configurable size whose windows overlap by a configurable number of
tokens, several utterances per step (Sec. II-D, batched streaming).

A fixed set of decode slots shares one paged KV pool.  Every decode step runs
``ftts_decode_step`` over all slots (a free slot carries token -1 and touches
nothing) followed by ``ftts_advance`` on the device, so a chunk of steps needs
no host round trip.  Between chunks the host

* hands the previous chunk's sampled ids (and hidden states) to each request,
  one device-to-host copy per chunk, while the current chunk already runs;
* retires requests whose budget ran out (``ftts_advance`` forced STOP at their
  last step and freed the slot on the device) or, with ``stop_on_token``, that
  sampled the stop code (the device freed the slot at that step), and returns
  their pages;
* admits waiting requests into free slots: their pages (prefix + budget) come
  from the host page pool, their prefixes are prefilled together in one
  ``ftts_prefill`` call, and their slot state (START token, position 0, KV slot,
  budget) is written by device copies ordered after the running chunk.

Nothing here computes model arithmetic: every step of the path runs in the HIP
library; this module only moves ids, pages and slot bookkeeping.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np
import torch

from . import ftts


@dataclass
class Request:
    """One utterance: its prefix rows (conditioning + text, already embedded) and
    its decode budget.  ``uniforms`` [max_new] drive sampling (top_k > 1)."""
    prefix: np.ndarray
    max_new: int
    uniforms: np.ndarray | None = None
    rid: int = -1
    tokens: list = field(default_factory=list)    # every emitted id, in order
    hidden: list = field(default_factory=list)    # [d] fp32 per emitted id (when asked for)
    chunks: list = field(default_factory=list)    # (first index, ids) windows handed downstream
    admitted_at: int = -1                         # chunk index of admission
    finished_at: int = -1                         # chunk index whose results completed it

    @property
    def done(self) -> bool:
        return self.finished_at >= 0


class Scheduler:
    """In-flight batching over ``max_slots`` decode slots.

    model      ftts.DeviceModel; shape its ModelShape.
    n_pages    KV pages in the shared pool (64 tokens each).
    max_ctx    longest prefix + budget a request may have (sizes the block table).
    sampling   ftts.Sampling shared by all requests.
    chunk      decode steps per chunk (ids are handed out once per chunk).
    overlap    ids repeated from the previous window at the start of each emitted window.
    hidden     also collect each step's last-layer hidden state (ftts_decode_step_hidden).
    graphs     replay each chunk's steps from a captured HIP graph (one per buffer parity)
               instead of launching every kernel from the host.
    stop_on_token  end a request when it samples the stop code (stop_token, default the
               shape's), not only when its budget runs out.
    """

    def __init__(self, model, shape, max_slots: int, n_pages: int, max_ctx: int, sampling, chunk: int = 16,
                 overlap: int = 0, hidden: bool = False, max_prefill_rows: int | None = None, graphs: bool = True,
                 stop_on_token: bool = False, stop_token: int | None = None):
        if chunk < 1 or overlap < 0 or overlap >= chunk:
            raise ValueError("need chunk >= 1 and 0 <= overlap < chunk")
        if graphs:
            ftts.graph_steps(chunk)                 # a chunk is one captured graph
        self.model, self.shape, self.B, self.chunk, self.overlap = model, shape, max_slots, chunk, overlap
        self.stop_token = shape.stop_token if stop_token is None else stop_token
        self.stop_on_token = stop_on_token
        self.sampling, self.want_hidden = sampling, hidden
        self.max_pages = (max_ctx + ftts.PAGE - 1) // ftts.PAGE
        self.pool = ftts.PagePool(n_pages)
        self.kv = ftts.KVCache(shape, model.wdtype, n_pages)
        B, dev = max_slots, "cuda"
        i32 = dict(dtype=torch.int32, device=dev)
        self.block_table = torch.full((B, self.max_pages), -1, **i32)
        self.pt = ftts.PageTableView(self.block_table, torch.zeros(B, **i32))
        self.tokens = torch.full((B,), -1, **i32)
        self.positions = torch.zeros(B, **i32)
        self.remaining = torch.zeros(B, **i32)
        self.sampled = torch.empty(B, **i32)
        self.counter = torch.zeros(1, **i32)
        self.history = [torch.full((chunk, B), -1, **i32) for _ in range(2)]  # double-buffered per chunk
        self.hidden_buf = ([torch.zeros((chunk, B, shape.d_model), dtype=torch.float32, device=dev)
                            for _ in range(2)] if hidden else None)
        self.uni = [torch.zeros((chunk, B), dtype=torch.float32, device=dev) for _ in range(2)]
        self.logits = torch.empty((B, shape.vocab), dtype=torch.float32, device=dev)
        rows = max_prefill_rows if max_prefill_rows is not None else B * max_ctx
        self.ws = torch.empty(ftts.workspace_bytes(model.cfg, B, rows), dtype=torch.uint8, device=dev)
        self.host_hist = [torch.empty((chunk, B), dtype=torch.int32).pin_memory() for _ in range(2)]
        self.host_hid = ([torch.empty((chunk, B, shape.d_model), dtype=torch.float32).pin_memory()
                          for _ in range(2)] if hidden else None)
        self.host_abort = [torch.zeros(1, dtype=torch.int32).pin_memory() for _ in range(2)]
        self.done_ev = [torch.cuda.Event() for _ in range(2)]
        self.slot_req: list[Request | None] = [None] * B
        self.slot_pages: list[list[int]] = [[] for _ in range(B)]
        self.slot_steps = [0] * B               # steps a slot's request has been given (host view)
        self.waiting: list[Request] = []
        self.n_chunks = 0
        self.next_rid = 0
        self.use_graphs = graphs
        self.graphs = [None, None]

    # -- requests ----------------------------------------------------------------------------
    def submit(self, req: Request) -> Request:
        need = req.prefix.shape[0] + req.max_new
        if req.max_new < 1 or req.prefix.shape[0] < 1 or need > self.max_pages * ftts.PAGE:
            raise ValueError("request does not fit max_ctx")
        req.rid = self.next_rid
        self.next_rid += 1
        self.waiting.append(req)
        return req

    def busy(self) -> bool:
        return bool(self.waiting) or any(r is not None for r in self.slot_req)

    # -- admission ---------------------------------------------------------------------------
    def _admit(self):
        free = [s for s in range(self.B) if self.slot_req[s] is None]
        group = []
        while free and self.waiting:
            req = self.waiting[0]
            n = -(-(req.prefix.shape[0] + req.max_new) // ftts.PAGE)
            if n > len(self.pool.free):
                break                            # wait for pages to come back
            self.waiting.pop(0)
            s = free.pop(0)
            self.slot_pages[s] = self.pool.alloc(n)
            self.slot_req[s] = req
            self.slot_steps[s] = 0
            req.admitted_at = self.n_chunks
            group.append((s, req))
        if not group:
            return
        slots = [s for s, _ in group]
        lens = [r.prefix.shape[0] for _, r in group]
        bt = np.full((len(group), self.max_pages), -1, dtype=np.int32)
        for i, s in enumerate(slots):
            bt[i, :len(self.slot_pages[s])] = self.slot_pages[s]
        bt_d = torch.from_numpy(bt).cuda()
        adt = ftts.act_dtype(self.model.wdtype)
        prefix = torch.from_numpy(np.concatenate([r.prefix for _, r in group]).astype(np.float32)).cuda().to(adt)
        pt = ftts.PageTableView(bt_d, torch.zeros(len(group), dtype=torch.int32, device="cuda"))
        ftts.prefill(self.model, prefix, lens, pt, self.kv, None, self.ws)
        idx = torch.tensor(slots, dtype=torch.int64, device="cuda")
        self.block_table.index_copy_(0, idx, bt_d)
        self.pt.seq_lens.index_copy_(0, idx, torch.tensor(lens, dtype=torch.int32, device="cuda"))
        self.tokens.index_fill_(0, idx, self.shape.start_token)
        self.positions.index_fill_(0, idx, 0)
        self.remaining.index_copy_(0, idx, torch.tensor([r.max_new for _, r in group], dtype=torch.int32,
                                                       device="cuda"))

    # -- one chunk of decode steps -----------------------------------------------------------
    def _launch_chunk(self, k: int):
        buf = k & 1
        if self.sampling.top_k != 1:
            u = np.zeros((self.chunk, self.B), dtype=np.float32)
            for s, r in enumerate(self.slot_req):
                if r is not None and r.uniforms is not None:
                    j0 = self.slot_steps[s]
                    take = r.uniforms[j0:j0 + self.chunk]
                    u[:len(take), s] = take
            self.uni[buf].copy_(torch.from_numpy(u))
        if self.use_graphs:
            if self.graphs[buf] is None:
                torch.cuda.synchronize()
                g = torch.cuda.CUDAGraph()
                with torch.cuda.graph(g):
                    self._steps(buf)
                self.graphs[buf] = g
                torch.cuda.synchronize()
            self.graphs[buf].replay()
        else:
            self._steps(buf)
        self.host_hist[buf].copy_(self.history[buf], non_blocking=True)
        self.host_abort[buf].copy_(ftts.abort_word(self.ws), non_blocking=True)
        if self.want_hidden:
            self.host_hid[buf].copy_(self.hidden_buf[buf], non_blocking=True)
        self.done_ev[buf].record()
        for s, r in enumerate(self.slot_req):
            if r is not None:
                self.slot_steps[s] += self.chunk

    def _steps(self, buf: int):
        """The device work of one chunk (captured once per buffer parity when graphs are on)."""
        self.history[buf].fill_(-1)
        self.counter.zero_()
        for t in range(self.chunk):
            ftts.decode_step(self.model, self.tokens, self.positions, self.pt, self.kv, self.logits, self.sampled,
                             self.uni[buf][t], self.sampling, self.ws,
                             hidden_out=self.hidden_buf[buf][t] if self.want_hidden else None)
            ftts.advance(self.tokens, self.positions, self.pt.seq_lens, self.sampled, self.remaining,
                         self.stop_token, self.history[buf], self.counter, retire_on_stop=self.stop_on_token)

    def _collect(self, k: int):
        """Hand chunk k's ids to their requests; retire the finished ones."""
        buf = k & 1
        self.done_ev[buf].synchronize()
        if int(self.host_abort[buf][0]) != 0:
            # a persistent step gave up waiting (its rows carry id -1): stop serving
            raise ftts.FTTSError(-6, f"decode chunk {k}: a persistent decode step timed out; "
                                     "its ids are invalid (ftts_prefill on a fresh workspace clears this)")
        hist = self.host_hist[buf].numpy()
        hid = self.host_hid[buf].numpy() if self.want_hidden else None
        for s, r in enumerate(self.slot_req):
            if r is None or r.admitted_at > k:
                continue
            got = [t for t in range(self.chunk) if hist[t, s] >= 0]
            start = len(r.tokens)
            r.tokens.extend(int(hist[t, s]) for t in got)
            if hid is not None:
                r.hidden.extend(hid[t, s].copy() for t in got)
            if got:
                w0 = max(0, start - self.overlap)
                r.chunks.append((w0, np.array(r.tokens[w0:], dtype=np.int32)))
            ended = self.stop_on_token and got and r.tokens[-1] == self.stop_token  # sampled stop code
            if len(r.tokens) >= r.max_new or ended:  # (or the budget's last step forced it on the device)
                r.finished_at = k
                self.pool.release(self.slot_pages[s])
                self.slot_pages[s] = []
                self.slot_req[s] = None

    def run(self, max_chunks: int = 1 << 30):
        """Serve until every submitted request is done.  Chunk k runs on the GPU
        while the host collects chunk k - 1 and admits into the slots it freed."""
        self._admit()
        pending = None
        while self.busy() and self.n_chunks < max_chunks:
            k = self.n_chunks
            self._launch_chunk(k)
            self.n_chunks += 1
            if pending is not None:
                self._collect(pending)
                # slots freed by chunk k-1 may still be active in chunk k only if their
                # budget was not used up (they are not freed then); admitting here is safe
                self._admit()
            pending = k
            if not any(r is not None for r in self.slot_req) and not self.waiting:
                break
        if pending is not None:
            self._collect(pending)
            while self.busy() and self.n_chunks < max_chunks:   # drain what the last admission added
                k = self.n_chunks
                self._launch_chunk(k)
                self.n_chunks += 1
                self._collect(k)
                self._admit()
