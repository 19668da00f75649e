"""Oracle: choosing the next token from fp32 logits.

TEST INFRASTRUCTURE ONLY -- see the package docstring.

The paper relies on the serving engine's sampling (Sec. I lists efficient
sampling strategies among its features) and prints no parameters.  This
module fixes one reading, step by step, in fp32:

greedy (top_k == 1): the index of the largest raw logit, lowest index on ties.

otherwise, with temperature T, top_k k and top_p p:
  1. z_i = logit_i / T                        (one IEEE fp32 division each)
  2. keep the k largest z, ordered by decreasing z, lower index first on ties
  3. e_i = exp(z_i - z_1) for the kept ones, in that order
  4. c_i = e_1 + ... + e_i, summed one term at a time in fp32
  5. n = the smallest i with c_i >= p * c_k   (the crossing token is kept)
  6. r = u * c_n; the result is the first kept index j <= n with c_j > r,
     or the n-th if none is
u is a host-supplied uniform in [0, 1).
"""
from __future__ import annotations

import numpy as np


def greedy(logits):
    """Index of the largest value, lowest index on ties."""
    return int(np.argmax(np.asarray(logits, dtype=np.float32)))


def top_k_order(z, k):
    """Indices of the k largest values, in decreasing value, lower index first on ties."""
    order = np.argsort(-z, kind="stable")
    return order[:k]


def sample(logits, temperature, top_k, top_p, u):
    """One draw as described in the module docstring; returns (token, detail dict)."""
    logits = np.asarray(logits, dtype=np.float32)
    V = logits.shape[0]
    if top_k == 1:
        return greedy(logits), {"n": 1, "cum": None, "r": None}
    k = V if top_k <= 0 or top_k > V else top_k
    z = logits / np.float32(temperature)
    top = top_k_order(z, k)
    zt = z[top]
    e = np.exp(zt - zt[0]).astype(np.float32)
    cum = np.empty(k, dtype=np.float32)
    acc = np.float32(0.0)
    for i in range(k):
        acc = np.float32(acc + e[i])
        cum[i] = acc
    thresh = np.float32(np.float32(top_p) * cum[k - 1])
    n = k
    for i in range(k):
        if cum[i] >= thresh:
            n = i + 1
            break
    r = np.float32(np.float32(u) * cum[n - 1])
    j = n - 1
    for i in range(n):
        if cum[i] > r:
            j = i
            break
    return int(top[j]), {"n": n, "cum": cum, "r": r, "thresh": thresh, "top": top[:n].copy()}


def near_boundary(detail, rel=1e-5):
    """True when the draw r, or the top-p threshold, lies within rel * c_k of one of
    the cumulative sums, i.e. when a one-ulp change in an exponential could change
    the pick."""
    if detail.get("cum") is None:
        return False
    cum, r, t = detail["cum"], detail["r"], detail["thresh"]
    tol = rel * cum[-1]
    return bool(np.any(np.abs(cum - r) <= tol) or np.any(np.abs(cum - t) <= tol))
