"""CPU pins of the DiT step oracle (oracle/dit.py) against facts that do not
come from the oracle itself: special values of the timestep features, brute
force attention, closed forms of degenerate weights, the symmetry the step must
have (no positions, no mask), and the limits of the guidance formula."""
import math

import numpy as np

from oracle import dit as odit
from oracle import gpt as ogpt
from paper_2607_21042_amd import workload

SH = workload.DitShape(n_layer=2, d_model=128, n_head=2, d_head=64, d_ff=256, n_mel=16, d_cond=32, t_dim=32)


def model(dtype=np.float64, zero_blocks=False):
    w = workload.dit_master_weights(SH, seed=3)
    if zero_blocks:
        for L in w["layers"]:
            for k in L:
                if k.startswith("w_") or k.startswith("b_"):
                    L[k] = np.zeros_like(L[k])
    return odit.DiT(w, SH.n_head, SH.d_head, dtype=dtype), w


def test_timestep_features_special_values():
    """t = 0: every cosine is 1 and every sine 0; the first frequency is 1, so at
    t = pi/1000 the first feature is cos(pi) = -1 and its sine partner 0."""
    s0 = odit.timestep_features(0.0, 32)
    np.testing.assert_array_equal(s0[:16], np.ones(16))
    np.testing.assert_array_equal(s0[16:], np.zeros(16))
    s = odit.timestep_features(math.pi / 1000.0, 32)
    assert abs(s[0] + 1.0) < 1e-15 and abs(s[16]) < 1e-12
    # the last frequency is 10000^(-15/16): its phase at t = 1 is 1000 * that
    s1 = odit.timestep_features(1.0, 32)
    assert abs(s1[15] - math.cos(1000.0 * 10000.0 ** (-15 / 16))) < 1e-12


def test_attention_matches_brute_force():
    """Every output row is the softmax-weighted sum over all keys, written out per element."""
    rng = np.random.default_rng(0)
    q, k, v = (rng.standard_normal((5, 4)) for _ in range(3))
    out = odit.attention(q, k, v)
    for i in range(5):
        w = [math.exp(sum(q[i, c] * k[j, c] for c in range(4)) / 2.0) for j in range(5)]
        z = sum(w)
        for c in range(4):
            assert abs(out[i, c] - sum(w[j] * v[j, c] for j in range(5)) / z) < 1e-12


def test_identity_blocks_reduce_to_projections():
    """With every block weight and bias zero each block is the identity, so v is
    LN_f(input projection + time embedding) through the mel projection."""
    m, w = model(zero_blocks=True)
    x, cond = workload.dit_inputs(SH, 7, seed=4)
    t = 0.3
    s = odit.timestep_features(t, SH.t_dim)
    e = w["w_t2"].astype(np.float64) @ (lambda u: u / (1 + np.exp(-u)))(
        w["w_t1"].astype(np.float64) @ s + w["b_t1"]) + w["b_t2"]
    h = np.concatenate([x, cond], axis=1).astype(np.float64) @ w["w_in"].T.astype(np.float64) + w["b_in"] + e
    mu = h.mean(axis=1, keepdims=True)
    var = ((h - mu) ** 2).mean(axis=1, keepdims=True)
    y = (h - mu) / np.sqrt(var + 1e-5) * w["lnf_g"] + w["lnf_b"]
    ref = y @ w["w_out_mel"].T.astype(np.float64) + w["b_out_mel"]
    np.testing.assert_allclose(m.velocity(x, cond, t), ref, rtol=1e-12, atol=1e-12)


def test_frames_permute_with_the_output():
    """No positions and no mask: permuting the frames permutes the velocity rows."""
    m, _ = model()
    x, cond = workload.dit_inputs(SH, 9, seed=5)
    p = np.random.default_rng(6).permutation(9)
    v = m.velocity(x, cond, 0.7)
    np.testing.assert_allclose(m.velocity(x[p], cond[p], 0.7), v[p], rtol=1e-10, atol=1e-12)
    # a causal mask would break this: the first frame alone would see only itself
    v1 = m.velocity(x[:1], cond[:1], 0.7)
    assert np.max(np.abs(v1[0] - v[0])) > 1e-6


def test_guidance_limits_and_euler():
    """w = 1 gives the conditional velocity, w = 0 the unconditional one (zero
    conditioning), w = 2 extrapolates past the conditional one; dt = 0 leaves x."""
    m, _ = model()
    x, cond = workload.dit_inputs(SH, 6, seed=7)
    vc = m.velocity(x, cond, 0.25)
    vu = m.velocity(x, np.zeros_like(cond), 0.25)
    x1, v1 = m.step(x, cond, 0.25, 0.04, 1.0)
    np.testing.assert_allclose(v1, vc, rtol=1e-12, atol=1e-14)
    _, v0 = m.step(x, cond, 0.25, 0.04, 0.0)
    np.testing.assert_allclose(v0, vu, rtol=1e-12, atol=1e-14)
    _, v2 = m.step(x, cond, 0.25, 0.04, 2.0)
    np.testing.assert_allclose(v2, 2 * vc - vu, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(x1, x + 0.04 * vc, rtol=1e-12, atol=1e-14)
    x0, _ = m.step(x, cond, 0.25, 0.0, 3.0)
    np.testing.assert_array_equal(x0, x.astype(np.float64))


def test_block_is_the_gpt_block_without_mask():
    """On a single frame the causal mask changes nothing, so the DiT block equals
    the GPT oracle's layer on that frame (same LayerNorm, GELU, head split)."""
    m, w = model()
    g = ogpt.GPT({"tok_emb": np.zeros((2, SH.d_model)), "pos_emb": np.zeros((2, SH.d_model)),
                  "layers": w["layers"], "lnf_g": np.ones(SH.d_model), "lnf_b": np.zeros(SH.d_model),
                  "w_head": np.zeros((2, SH.d_model)), "b_head": np.zeros(2)}, SH.n_head, SH.d_head,
                 dtype=np.float64)
    h = np.random.default_rng(8).standard_normal((1, SH.d_model))
    logits, hid = g.full_forward(h)
    ref = h
    for L in m.layers:
        ref = m.block(ref, L)
    mu = ref.mean(axis=1, keepdims=True)
    var = ((ref - mu) ** 2).mean(axis=1, keepdims=True)
    np.testing.assert_allclose(hid, (ref - mu) / np.sqrt(var + 1e-5), rtol=1e-10, atol=1e-12)


def test_silu_known_values():
    """silu(u) = u * sigmoid(u): sigmoid(1) = e / (1 + e) = 0.7310585786300049,
    silu(-1) = -(1 - sigmoid(1)), silu(0) = 0, and the two tails (u and 0)."""
    u = np.array([1.0, -1.0, 0.0, 40.0, -40.0])
    s = odit.silu(u)
    np.testing.assert_allclose(s[:2], [0.7310585786300049, -0.2689414213699951], rtol=0, atol=1e-15)
    assert s[2] == 0.0
    assert abs(s[3] - 40.0) < 1e-12 and abs(s[4]) < 1e-15
