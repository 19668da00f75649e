"""Oracle: the GPT-2 style decoder of IndexTTS-2's Text-to-Semantic module.

TEST INFRASTRUCTURE ONLY -- see the package docstring.

What is computed (Sec. II-A: the Text-to-Semantic module is a decoder-only
autoregressive GPT of the GPT-2 family; Sec. II-C: conditioning enters as a
prefix of embeddings, and positions are custom):

  input rows   prefix rows are the conditioning embeddings as given, with no
               position embedding added; a decoded row is
               tok_emb[token] + pos_emb[position], the semantic tokens using
               their own position range starting at 0.
  each layer   a = LN1(x);  [q | k | v] = a W_qkv^T + b_qkv
               per head h (columns h*dh .. h*dh+dh-1 of each block):
                   o_h = softmax(q_h K_h^T / sqrt(dh), causal) V_h
               x = x + concat_h(o_h) W_out^T + b_out
               x = x + gelu(LN2(x) W_fc1^T + b_fc1) W_fc2^T + b_fc2
  head         logits = LN_f(x) W_head^T + b_head

Readings of points the paper leaves open (each pinned by a test):
  * LayerNorm uses the biased variance and eps = 1e-5.
  * GELU is GPT-2's tanh form.
  * Every linear, the LM head included, has a bias; the head is untied.
  * The prefix gets no positional embedding at all.

Arithmetic is plain numpy in the dtype of the weights handed in (fp64 for
self-checks, fp32 for parity); there is no blocking, fusion or reordering
beyond one matrix product per linear.
"""
from __future__ import annotations

import numpy as np

LN_EPS = 1e-5


def layer_norm(x, g, b, eps=LN_EPS):
    """(x - mean) / sqrt(var + eps) * g + b over the last axis, biased variance."""
    mean = x.mean(axis=-1, keepdims=True)
    var = ((x - mean) ** 2).mean(axis=-1, keepdims=True)
    return (x - mean) / np.sqrt(var + x.dtype.type(eps)) * g + b


def gelu(u):
    """GPT-2's tanh approximation of the Gaussian error linear unit."""
    t = u.dtype.type
    c = t(np.sqrt(2.0 / np.pi))
    return t(0.5) * u * (t(1.0) + np.tanh(c * (u + t(0.044715) * u * u * u)))


def softmax(s):
    """Softmax over the last axis (max-subtracted, which leaves the value unchanged)."""
    e = np.exp(s - s.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


def linear(a, w, b):
    """a W^T + b with W stored [out][in]."""
    return a @ w.T + b


def causal_attention(q, k, v, n_head, d_head):
    """Causal multi-head attention over T rows: q, k, v are [T, n_head*d_head]."""
    T = q.shape[0]
    scale = q.dtype.type(1.0 / np.sqrt(d_head))
    out = np.empty_like(q)
    mask = np.triu(np.ones((T, T), dtype=bool), k=1)
    for h in range(n_head):
        c = slice(h * d_head, (h + 1) * d_head)
        s = (q[:, c] @ k[:, c].T) * scale
        s = np.where(mask, -np.inf, s)
        out[:, c] = softmax(s) @ v[:, c]
    return out


def attend_last(q, K, V, n_head, d_head):
    """Attention of one query row over all cached rows (the newest one included)."""
    scale = q.dtype.type(1.0 / np.sqrt(d_head))
    out = np.empty_like(q)
    for h in range(n_head):
        c = slice(h * d_head, (h + 1) * d_head)
        s = (K[:, c] @ q[c]) * scale
        out[c] = softmax(s) @ V[:, c]
    return out


class GPT:
    """The decoder forward on given weights (see module docstring).

    ``weights`` is the dict layout produced by the seeded input generator:
    tok_emb [V,d], pos_emb [n_pos,d], layers[l] = {ln1_g, ln1_b, w_qkv [3d,d],
    b_qkv, w_out [d,d], b_out, ln2_g, ln2_b, w_fc1 [f,d], b_fc1, w_fc2 [d,f],
    b_fc2}, lnf_g, lnf_b, w_head [V,d], b_head.  Quantised models pass their
    dequantised matrices here.
    """

    def __init__(self, weights, n_head, d_head, dtype=np.float32, eps=LN_EPS):
        cast = lambda a: np.ascontiguousarray(a, dtype=dtype)  # noqa: E731
        self.dtype = np.dtype(dtype)
        self.n_head, self.d_head, self.eps = n_head, d_head, eps
        self.tok_emb = cast(weights["tok_emb"])
        self.pos_emb = cast(weights["pos_emb"])
        self.layers = [{k: cast(v) for k, v in lw.items()} for lw in weights["layers"]]
        self.lnf_g, self.lnf_b = cast(weights["lnf_g"]), cast(weights["lnf_b"])
        self.w_head, self.b_head = cast(weights["w_head"]), cast(weights["b_head"])
        self.d_model = self.tok_emb.shape[1]

    # -- input rows -----------------------------------------------------------
    def embed(self, tokens, positions):
        """Rows for decoded tokens: token embedding plus own-range position embedding."""
        tokens = np.asarray(tokens)
        positions = np.asarray(positions)
        return self.tok_emb[tokens] + self.pos_emb[positions]

    def assemble_prefix(self, cond, text_ids, text_pos0):
        """The model's own prefix from ids (Sec. II-C, the first three serving
        adaptations): the conditioning rows as given, with no position
        embedding, then one row per text token.  Text and semantic codes share
        one token table with the text block after the semantic vocabulary (its
        size: the LM head's rows), so text id t is row vocab + t; text token i
        takes position row text_pos0 + i, the text range of the position table."""
        cond = np.asarray(cond, dtype=self.dtype).reshape(-1, self.d_model)
        text_ids = np.asarray(text_ids, dtype=np.int64)
        vocab = self.w_head.shape[0]
        text = self.tok_emb[vocab + text_ids] + self.pos_emb[text_pos0 + np.arange(len(text_ids))]
        return np.concatenate([cond, text.reshape(-1, self.d_model)], axis=0)

    def rows(self, prefix, tokens=(), positions=None):
        """Prefix rows (as given, no positions) followed by decoded-token rows."""
        prefix = np.asarray(prefix, dtype=self.dtype)
        tokens = np.asarray(tokens, dtype=np.int64)
        if positions is None:
            positions = np.arange(len(tokens))
        if len(tokens) == 0:
            return prefix
        return np.concatenate([prefix, self.embed(tokens, positions)], axis=0)

    def head(self, x):
        """Final LayerNorm and LM head; returns (logits, normalised hidden state)."""
        hn = layer_norm(x, self.lnf_g, self.lnf_b, self.eps)
        return linear(hn, self.w_head, self.b_head), hn

    # -- full causal forward over a whole sequence ------------------------------
    def full_forward(self, x):
        """Causal forward over rows x [T, d]; returns (logits [T,V], final hidden [T,d])."""
        x = np.array(x, dtype=self.dtype)
        d = self.d_model
        for lw in self.layers:
            a = layer_norm(x, lw["ln1_g"], lw["ln1_b"], self.eps)
            qkv = linear(a, lw["w_qkv"], lw["b_qkv"])
            o = causal_attention(qkv[:, :d], qkv[:, d:2 * d], qkv[:, 2 * d:],
                                 self.n_head, self.d_head)
            x = x + linear(o, lw["w_out"], lw["b_out"])
            a = layer_norm(x, lw["ln2_g"], lw["ln2_b"], self.eps)
            x = x + linear(gelu(linear(a, lw["w_fc1"], lw["b_fc1"])), lw["w_fc2"], lw["b_fc2"])
        return self.head(x)

    # -- incremental (KV-cache) forward ------------------------------------------
    def new_cache(self):
        """Per-layer lists of cached key and value rows (layout-free)."""
        return {"k": [np.zeros((0, self.d_model), self.dtype) for _ in self.layers],
                "v": [np.zeros((0, self.d_model), self.dtype) for _ in self.layers]}

    def prefill(self, prefix):
        """Run the prefix rows, filling a fresh cache; returns (cache, logits of the last row)."""
        x = np.array(prefix, dtype=self.dtype)
        cache = self.new_cache()
        d = self.d_model
        for i, lw in enumerate(self.layers):
            a = layer_norm(x, lw["ln1_g"], lw["ln1_b"], self.eps)
            qkv = linear(a, lw["w_qkv"], lw["b_qkv"])
            cache["k"][i] = qkv[:, d:2 * d].copy()
            cache["v"][i] = qkv[:, 2 * d:].copy()
            o = causal_attention(qkv[:, :d], qkv[:, d:2 * d], qkv[:, 2 * d:],
                                 self.n_head, self.d_head)
            x = x + linear(o, lw["w_out"], lw["b_out"])
            a = layer_norm(x, lw["ln2_g"], lw["ln2_b"], self.eps)
            x = x + linear(gelu(linear(a, lw["w_fc1"], lw["b_fc1"])), lw["w_fc2"], lw["b_fc2"])
        logits, _ = self.head(x[-1])
        return cache, logits

    def decode_step(self, cache, token, position):
        """Append one decoded row to the cache and return (logits, final hidden) for it."""
        x = self.embed(token, position).astype(self.dtype)
        d = self.d_model
        for i, lw in enumerate(self.layers):
            a = layer_norm(x, lw["ln1_g"], lw["ln1_b"], self.eps)
            qkv = linear(a, lw["w_qkv"], lw["b_qkv"])
            cache["k"][i] = np.concatenate([cache["k"][i], qkv[None, d:2 * d]], axis=0)
            cache["v"][i] = np.concatenate([cache["v"][i], qkv[None, 2 * d:]], axis=0)
            o = attend_last(qkv[:d], cache["k"][i], cache["v"][i], self.n_head, self.d_head)
            x = x + linear(o, lw["w_out"], lw["b_out"])
            a = layer_norm(x, lw["ln2_g"], lw["ln2_b"], self.eps)
            x = x + linear(gelu(linear(a, lw["w_fc1"], lw["b_fc1"])), lw["w_fc2"], lw["b_fc2"])
        return self.head(x)

    def greedy_decode(self, prefix, n_steps, start_token):
        """Prefill, then n_steps greedy steps feeding start_token first; returns tokens [n_steps]."""
        cache, _ = self.prefill(prefix)
        tok, out = start_token, []
        for t in range(n_steps):
            logits, _ = self.decode_step(cache, tok, t)
            tok = int(np.argmax(logits))
            out.append(tok)
        return np.array(out, dtype=np.int32)
