"""Oracle: one Euler step of the Semantic-to-Mel flow-matching DiT with
classifier-free guidance.

TEST INFRASTRUCTURE ONLY -- see the package docstring.

What is computed (Sec. II-A: the Semantic-to-Mel module is conditional flow
matching with a Diffusion Transformer, conditioned on GPT hidden states among
others; at inference an Euler ODE solver with classifier-free guidance refines
the mel over several steps; Sec. III-A: the DiT has 96M parameters):

  time         e(t) = W_t2 silu(W_t1 s(t) + b_t1) + b_t2, with s(t) the sinusoidal
               features [cos(1000 t f_i), sin(1000 t f_i)], f_i = 10000^(-i/half)
  input        h = [x | c] W_in^T + b_in + e(t)      (one row per frame)
  each block   h = h + Attn(LN1(h)),  h = h + W_fc2 gelu(LN2(h) W_fc1^T + b_fc1) + b_fc2
               Attn: per head, softmax(q k^T / sqrt(dh)) v over ALL frames (no mask)
  output       v(x, c, t) = LN_f(h) W_mel^T + b_mel
  guidance     v = v(x, 0, t) + w (v(x, c, t) - v(x, 0, t))
  Euler step   x' = x + dt v

Readings of points the paper leaves open (each pinned by a test):
  * the block is the pre-LN transformer block of the GPT (biased-variance
    LayerNorm, eps 1e-5, tanh GELU, biases everywhere), without a causal mask;
  * frames carry no positional embedding (the step is equivariant under a
    permutation of the frames);
  * the time embedding is the sinusoid-plus-MLP form above, added to every row;
  * the unconditional branch zeroes the conditioning rows; guidance strength w
    scales the conditional-minus-unconditional difference (w = 1: conditional).

Arithmetic is plain numpy in the dtype of the weights handed in; one matrix
product per linear and the attention written from its definition.
"""
from __future__ import annotations

import numpy as np

from .gpt import gelu, layer_norm, linear, softmax


def timestep_features(t: float, dim: int, dtype=np.float64) -> np.ndarray:
    """[cos(1000 t f_i) for i < dim/2, sin(1000 t f_i) for i < dim/2], f_i = 10000^(-i/(dim/2))."""
    half = dim // 2
    f = np.exp(-np.log(10000.0) * np.arange(half, dtype=np.float64) / half)
    a = 1000.0 * float(t) * f
    return np.concatenate([np.cos(a), np.sin(a)]).astype(dtype)


def silu(u):
    return u / (u.dtype.type(1.0) + np.exp(-u))


def attention(q, k, v):
    """softmax(q k^T / sqrt(dh)) v over all keys, for [T][dh] arrays."""
    s = (q @ k.T) / q.dtype.type(np.sqrt(q.shape[-1]))
    return softmax(s) @ v


class DiT:
    """w: the dict of ``workload.dit_master_weights`` (or its bf16-rounded copy)."""

    def __init__(self, w: dict, n_head: int, d_head: int, dtype=np.float32):
        self.dt = np.dtype(dtype)
        cast = lambda a: np.asarray(a, dtype=self.dt)
        self.g = {k: cast(v) for k, v in w.items() if k != "layers"}
        self.layers = [{k: cast(v) for k, v in lw.items()} for lw in w["layers"]]
        self.H, self.dh = n_head, d_head

    def time_embedding(self, t: float) -> np.ndarray:
        g = self.g
        s = timestep_features(t, g["w_t1"].shape[1], self.dt)
        return linear(silu(linear(s, g["w_t1"], g["b_t1"])), g["w_t2"], g["b_t2"])

    def block(self, h: np.ndarray, L: dict) -> np.ndarray:
        d = h.shape[1]
        a = layer_norm(h, L["ln1_g"], L["ln1_b"])
        qkv = linear(a, L["w_qkv"], L["b_qkv"])
        q, k, v = qkv[:, :d], qkv[:, d:2 * d], qkv[:, 2 * d:]
        heads = [attention(q[:, i * self.dh:(i + 1) * self.dh], k[:, i * self.dh:(i + 1) * self.dh],
                           v[:, i * self.dh:(i + 1) * self.dh]) for i in range(self.H)]
        h = h + linear(np.concatenate(heads, axis=1), L["w_out"], L["b_out"])
        a = layer_norm(h, L["ln2_g"], L["ln2_b"])
        return h + linear(gelu(linear(a, L["w_fc1"], L["b_fc1"])), L["w_fc2"], L["b_fc2"])

    def velocity(self, x: np.ndarray, cond: np.ndarray, t: float) -> np.ndarray:
        g = self.g
        inp = np.concatenate([np.asarray(x, self.dt), np.asarray(cond, self.dt)], axis=1)
        h = linear(inp, g["w_in"], g["b_in"]) + self.time_embedding(t)
        for L in self.layers:
            h = self.block(h, L)
        return linear(layer_norm(h, g["lnf_g"], g["lnf_b"]), g["w_out_mel"], g["b_out_mel"])

    def step(self, x: np.ndarray, cond: np.ndarray, t: float, dt: float, w_cfg: float):
        """One guided Euler step: returns (x', v)."""
        vc = self.velocity(x, cond, t)
        vu = self.velocity(x, np.zeros_like(cond), t)
        v = vu + self.dt.type(w_cfg) * (vc - vu)
        return np.asarray(x, self.dt) + self.dt.type(dt) * v, v
