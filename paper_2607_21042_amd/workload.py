"""Seeded synthetic inputs for the IndexTTS-2-shaped GPT decode path.

This module is the only code shared by the CPU oracle's tests, the GPU path's
tests and the benchmark.  It draws random numbers and converts them to the
storage dtype of the inputs; it holds none of the method's arithmetic (no
normalisation, no attention, no quantisation, no sampling).

Shapes follow the paper's model class: a decoder-only GPT-2 style network
(Sec. II-A), conditioned on a prefix of embeddings that are not tokens
(Sec. II-C, first adaptation), emitting semantic codec tokens.  The paper gives
only the parameter count of its GPT (512M, Sec. III-A); the 24 x 1280 shape used
here has 494.6M parameters.

Every tensor is drawn from its own PCG64 stream, seeded with ``[seed, id]``, so
tensors are independent of generation order and can be drawn in parallel.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass

import numpy as np


@dataclass(frozen=True)
class ModelShape:
    n_layer: int
    d_model: int
    n_head: int
    d_head: int
    d_ff: int
    vocab: int
    n_pos: int = 1024

    @property
    def start_token(self) -> int:
        # The last two rows of the semantic vocabulary are the start and stop
        # codes (8192 codes + 2 specials for the 8194-row vocabulary).
        return self.vocab - 2

    @property
    def stop_token(self) -> int:
        return self.vocab - 1

    def matrices(self):
        """(name, N, K) of the four per-layer linears, weights stored [N][K]."""
        d, f = self.d_model, self.d_ff
        return [("qkv", 3 * d, d), ("out", d, d), ("fc1", f, d), ("fc2", d, f)]

    def n_params(self) -> int:
        d, f, V = self.d_model, self.d_ff, self.vocab
        per_layer = sum(N * K + N for _, N, K in self.matrices()) + 4 * d
        return (V * d + self.n_pos * d + self.n_layer * per_layer + 2 * d
                + V * d + V)


# Tiny GPT-2 style decoder: 2 layers, d=256, 4 heads of 64, FFN 1024, vocab 1024.
TINY = ModelShape(n_layer=2, d_model=256, n_head=4, d_head=64, d_ff=1024, vocab=1024)
# IndexTTS-2-shaped Text-to-Semantic GPT: 24 layers, d=1280, 20 heads of 64,
# FFN 5120, semantic vocabulary 8194.
INDEXTTS2 = ModelShape(n_layer=24, d_model=1280, n_head=20, d_head=64, d_ff=5120, vocab=8194)

INIT_STD = 0.02


def bf16_round(a: np.ndarray) -> np.ndarray:
    """Round fp32 values to the nearest bfloat16 (ties to even), returned as fp32.

    Used only to make inputs that are exactly representable in bf16, so the
    same numbers can be handed to a bf16 GPU buffer and to an fp32 CPU array.
    """
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32).reshape(a.shape)


def bf16_bits(a: np.ndarray) -> np.ndarray:
    """Upper 16 bits of fp32 values that are already bf16-representable."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    bits = a.view(np.uint32)
    if np.any(bits & 0xFFFF):
        raise ValueError("values are not bf16-representable; call bf16_round first")
    return (bits >> 16).astype(np.uint16)


def _normal(seed: int, tid: int, shape, std: float, mean: float = 0.0) -> np.ndarray:
    rng = np.random.default_rng([seed, tid])
    a = rng.standard_normal(shape, dtype=np.float32)
    a *= np.float32(std)
    if mean:
        a += np.float32(mean)
    return a


def _weight_specs(shape: ModelShape):
    """(key, layer or None, tensor shape, mean) in a fixed order; index = stream id."""
    d, V = shape.d_model, shape.vocab
    specs = [("tok_emb", None, (V, d), 0.0), ("pos_emb", None, (shape.n_pos, d), 0.0)]
    for l in range(shape.n_layer):
        specs += [("ln1_g", l, (d,), 1.0), ("ln1_b", l, (d,), 0.0)]
        for name, N, K in shape.matrices():
            if name == "fc1":
                specs += [("ln2_g", l, (d,), 1.0), ("ln2_b", l, (d,), 0.0)]
            specs += [("w_" + name, l, (N, K), 0.0), ("b_" + name, l, (N,), 0.0)]
    specs += [("lnf_g", None, (d,), 1.0), ("lnf_b", None, (d,), 0.0),
              ("w_head", None, (V, d), 0.0), ("b_head", None, (V,), 0.0)]
    return specs


def master_weights(shape: ModelShape, seed: int = 0, threads: int | None = None) -> dict:
    """fp32 master weights, every tensor ~N(0, 0.02) (LayerNorm gains 1 + N(0, 0.02)).

    Returns ``{"tok_emb", "pos_emb", "layers": [ {ln1_g, ln1_b, w_qkv, b_qkv, w_out,
    b_out, ln2_g, ln2_b, w_fc1, b_fc1, w_fc2, b_fc2} ], "lnf_g", "lnf_b",
    "w_head", "b_head"}``.  Linear weights are [N][K] (output row, input column);
    the qkv rows are ordered [q | k | v], each block split into heads of d_head.
    """
    specs = _weight_specs(shape)
    threads = threads or min(8, os.cpu_count() or 1)

    def draw(i):
        key, _, shp, mean = specs[i]
        return _normal(seed, i, shp, INIT_STD, mean)

    with ThreadPoolExecutor(threads) as ex:
        arrays = list(ex.map(draw, range(len(specs))))
    out: dict = {"layers": [dict() for _ in range(shape.n_layer)]}
    for (key, layer, _, _), a in zip(specs, arrays):
        if layer is None:
            out[key] = a
        else:
            out["layers"][layer][key] = a
    return out


def map_weights(w: dict, fn, keys=None) -> dict:
    """Apply ``fn`` to every array (or to those named in ``keys``)."""
    def conv(k, a):
        return fn(a) if keys is None or k in keys else a
    out = {k: conv(k, v) for k, v in w.items() if k != "layers"}
    out["layers"] = [{k: conv(k, v) for k, v in lw.items()} for lw in w["layers"]]
    return out


def bf16_weights(master: dict, threads: int = 8) -> dict:
    """All parameters rounded to bf16 values (kept as fp32 arrays)."""
    flat = []
    for k, v in master.items():
        if k != "layers":
            flat.append((None, k, v))
    for l, lw in enumerate(master["layers"]):
        for k, v in lw.items():
            flat.append((l, k, v))
    with ThreadPoolExecutor(threads) as ex:
        rounded = list(ex.map(lambda t: bf16_round(t[2]), flat))
    out: dict = {"layers": [dict() for _ in master["layers"]]}
    for (l, k, _), r in zip(flat, rounded):
        if l is None:
            out[k] = r
        else:
            out["layers"][l][k] = r
    return out


def prefix_embeddings(lens, d_model: int, seed: int = 1, bf16: bool = True) -> np.ndarray:
    """Conditioning prefix rows ~N(0, 1), packed [sum(lens), d_model] in sequence order."""
    rng = np.random.default_rng(seed)
    a = rng.standard_normal((int(np.sum(lens)), d_model), dtype=np.float32)
    return bf16_round(a) if bf16 else a


def uniforms(n_steps: int, batch: int, seed: int = 2) -> np.ndarray:
    """Host-side sampling uniforms in [0, 1), one per (step, sequence)."""
    # Generated directly as float32 so that no value rounds up to 1.0.
    return np.random.default_rng(seed).random((n_steps, batch), dtype=np.float32)


def batch_lengths(batch: int, seed: int = 3, prefix=(128, 512), target=(256, 768)):
    """Per-sequence prefix lengths and decode target lengths, uniform on the closed ranges."""
    rng = np.random.default_rng(seed)
    p = rng.integers(prefix[0], prefix[1] + 1, size=batch).astype(np.int32)
    t = rng.integers(target[0], target[1] + 1, size=batch).astype(np.int32)
    return p, t


def text_table(shape: ModelShape, n_text: int, seed: int = 9) -> np.ndarray:
    """Rows of a text-token embedding block [n_text, d_model] ~N(0, 0.02), bf16-representable.
    Appended after the semantic rows of tok_emb it forms the merged token table."""
    rng = np.random.default_rng(seed)
    return bf16_round(rng.standard_normal((n_text, shape.d_model), dtype=np.float32) * np.float32(INIT_STD))


def text_ids(lens, n_text: int, seed: int = 10) -> np.ndarray:
    """Packed text-token ids in [0, n_text) for sequences of the given lengths."""
    return np.random.default_rng(seed).integers(0, n_text, size=int(np.sum(lens))).astype(np.int32)


def random_tokens(n_steps: int, batch: int, vocab: int, seed: int = 4) -> np.ndarray:
    """Teacher-forcing token ids in [0, vocab - 2) (no special codes), shape [n_steps, batch]."""
    return np.random.default_rng(seed).integers(0, vocab - 2, size=(n_steps, batch)).astype(np.int32)


def random_logits(batch: int, vocab: int, seed: int = 5, scale: float = 3.0) -> np.ndarray:
    """fp32 logits for exercising a sampler on its own, shape [batch, vocab]."""
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((batch, vocab), dtype=np.float32) * np.float32(scale))


LINEAR_KEYS = ("w_qkv", "w_out", "w_fc1", "w_fc2")


def quantisable_weights(master: dict, threads: int = 8) -> dict:
    """Inputs of a weight-only-quantised model: the four per-layer matrices keep
    their fp32 master values (each side quantises them itself); every other
    tensor is rounded to bf16."""
    out = bf16_weights({k: v for k, v in master.items()} | {"layers": [
        {k: v for k, v in lw.items() if k not in LINEAR_KEYS} for lw in master["layers"]]}, threads)
    for lw_out, lw in zip(out["layers"], master["layers"]):
        for k in LINEAR_KEYS:
            lw_out[k] = lw[k]
    return out


# ---- Semantic-to-Mel flow-matching DiT (synthetic shape) ---------------------------------
@dataclass(frozen=True)
class DitShape:
    n_layer: int
    d_model: int
    n_head: int
    d_head: int
    d_ff: int
    n_mel: int      # mel bins of the state being integrated
    d_cond: int     # width of the per-frame conditioning rows (GPT hidden states)
    t_dim: int = 256  # sinusoidal timestep features

    def matrices(self):
        d, f = self.d_model, self.d_ff
        return [("qkv", 3 * d, d), ("out", d, d), ("fc1", f, d), ("fc2", d, f)]

    def n_params(self) -> int:
        d = self.d_model
        per_layer = sum(N * K + N for _, N, K in self.matrices()) + 4 * d
        return (d * (self.n_mel + self.d_cond) + d + d * self.t_dim + d + d * d + d
                + self.n_layer * per_layer + 2 * d + self.n_mel * d + self.n_mel)


# Tiny DiT for parity: 2 blocks of width 256.  The 96M-parameter shape: 13 pre-LN
# blocks of width 768 (12 heads of 64, FFN 3072), 128 mel bins, conditioned on the
# GPT's 1280-wide hidden states.
DIT_TINY = DitShape(n_layer=2, d_model=256, n_head=4, d_head=64, d_ff=1024, n_mel=128, d_cond=256)
DIT_96M = DitShape(n_layer=13, d_model=768, n_head=12, d_head=64, d_ff=3072, n_mel=128, d_cond=1280)


def dit_master_weights(shape: DitShape, seed: int = 20) -> dict:
    """fp32 DiT weights ~N(0, 0.02) (LayerNorm gains 1 + N(0, 0.02)), one stream per tensor.

    ``{"w_in" [d][n_mel + d_cond], "b_in", "w_t1" [d][t_dim], "b_t1", "w_t2" [d][d], "b_t2",
    "layers": [ {ln1_g, ln1_b, w_qkv, b_qkv, w_out, b_out, ln2_g, ln2_b, w_fc1, b_fc1, w_fc2,
    b_fc2} ], "lnf_g", "lnf_b", "w_out_mel" [n_mel][d], "b_out_mel"}``.
    """
    d = shape.d_model
    specs = [("w_in", None, (d, shape.n_mel + shape.d_cond), 0.0), ("b_in", None, (d,), 0.0),
             ("w_t1", None, (d, shape.t_dim), 0.0), ("b_t1", None, (d,), 0.0),
             ("w_t2", None, (d, d), 0.0), ("b_t2", None, (d,), 0.0)]
    for l in range(shape.n_layer):
        specs += [("ln1_g", l, (d,), 1.0), ("ln1_b", l, (d,), 0.0)]
        for name, N, K in shape.matrices():
            if name == "fc1":
                specs += [("ln2_g", l, (d,), 1.0), ("ln2_b", l, (d,), 0.0)]
            specs += [("w_" + name, l, (N, K), 0.0), ("b_" + name, l, (N,), 0.0)]
    specs += [("lnf_g", None, (d,), 1.0), ("lnf_b", None, (d,), 0.0),
              ("w_out_mel", None, (shape.n_mel, d), 0.0), ("b_out_mel", None, (shape.n_mel,), 0.0)]
    out: dict = {"layers": [dict() for _ in range(shape.n_layer)]}
    for i, (key, layer, shp, mean) in enumerate(specs):
        a = _normal(seed, i, shp, INIT_STD, mean)
        if layer is None:
            out[key] = a
        else:
            out["layers"][layer][key] = a
    return out


def dit_inputs(shape: DitShape, T: int, seed: int = 21):
    """The state x [T][n_mel] ~N(0, 1) (fp32) and conditioning rows cond [T][d_cond] ~N(0, 1)
    rounded to bf16 (the GPU takes them as bf16)."""
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((T, shape.n_mel), dtype=np.float32)
    cond = bf16_round(rng.standard_normal((T, shape.d_cond), dtype=np.float32))
    return x, cond
