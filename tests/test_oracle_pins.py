"""Pins for the CPU oracle: each check ties it to something other than itself.

* Library routines for the textbook special cases: torch's layer_norm, tanh-GELU
  and scaled-dot-product attention, and Hugging Face's GPT-2 (the model class the
  paper builds on, Sec. II-A) for the whole decoder stack.
* Brute force with explicit loops on tiny inputs.
* Closed forms and invariants: normalised moments, odd-part identity of GELU,
  softmax special cases, incremental decode == full causal forward.
* Hand-worked quantiser and sampler examples (tests/golden/).
* Planted mistakes: a broken copy of an oracle function must fail the pins.
"""
import json
import math
import os

import numpy as np
import pytest
import torch

from oracle import gpt, quant, sample
from paper_2607_21042_amd import workload

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
SMALL = workload.ModelShape(n_layer=2, d_model=128, n_head=2, d_head=64, d_ff=256, vocab=64, n_pos=32)


def small_model(dtype=np.float64, shape=SMALL, seed=0):
    w = workload.master_weights(shape, seed=seed, threads=2)
    # Larger than the init std so that every term of the forward is exercised.
    w = workload.map_weights(w, lambda a: a * 5 if a.ndim == 2 else a)
    return w, gpt.GPT(w, shape.n_head, shape.d_head, dtype=dtype)


# --------------------------------------------------------------------------- LN / GELU
def test_layer_norm_matches_torch_and_closed_forms():
    rng = np.random.default_rng(10)
    x = rng.standard_normal((7, 96)) * 3 + 1.5
    g = rng.standard_normal(96)
    b = rng.standard_normal(96)
    ref = torch.nn.functional.layer_norm(torch.from_numpy(x), (96,), torch.from_numpy(g),
                                         torch.from_numpy(b), eps=1e-5).numpy()
    np.testing.assert_allclose(gpt.layer_norm(x, g, b), ref, rtol=0, atol=1e-12)
    y = gpt.layer_norm(x, np.ones(96), np.zeros(96))
    np.testing.assert_allclose(y.mean(axis=1), 0, atol=1e-12)
    np.testing.assert_allclose((y ** 2).mean(axis=1), 1, atol=1e-4)  # eps shrinks it slightly
    # invariant to shift and positive scale of the input
    np.testing.assert_allclose(gpt.layer_norm(4 * x - 7, g, b), gpt.layer_norm(x, g, b), atol=1e-5)


def test_gelu_matches_torch_and_identities():
    u = np.linspace(-8, 8, 2001)
    ref = torch.nn.functional.gelu(torch.from_numpy(u), approximate="tanh").numpy()
    np.testing.assert_allclose(gpt.gelu(u), ref, rtol=0, atol=1e-12)
    assert gpt.gelu(np.array([0.0]))[0] == 0.0
    # gelu(u) - gelu(-u) = u holds for u * Phi(u) and for its tanh approximation
    np.testing.assert_allclose(gpt.gelu(u) - gpt.gelu(-u), u, atol=1e-12)
    # the tanh form stays within 1e-3 of the exact u * Phi(u)
    exact = np.array([x * 0.5 * (1 + math.erf(x / math.sqrt(2))) for x in u])
    assert np.max(np.abs(gpt.gelu(u) - exact)) < 1e-3


# --------------------------------------------------------------------------- attention
def brute_attention(q, k, v, n_head, d_head):
    """Explicit loops: scores, running max, exponentials, weighted sum."""
    T = q.shape[0]
    out = np.zeros_like(q)
    for h in range(n_head):
        for i in range(T):
            scores = []
            for j in range(i + 1):
                s = 0.0
                for c in range(d_head):
                    s += q[i, h * d_head + c] * k[j, h * d_head + c]
                scores.append(s / math.sqrt(d_head))
            m = max(scores)
            w = [math.exp(s - m) for s in scores]
            tot = sum(w)
            for c in range(d_head):
                out[i, h * d_head + c] = sum(w[j] * v[j, h * d_head + c] for j in range(i + 1)) / tot
    return out


def test_causal_attention_brute_force():
    rng = np.random.default_rng(11)
    H, dh, T = 2, 8, 6
    q, k, v = (rng.standard_normal((T, H * dh)) for _ in range(3))
    np.testing.assert_allclose(gpt.causal_attention(q, k, v, H, dh), brute_attention(q, k, v, H, dh),
                               rtol=0, atol=1e-12)
    for i in range(T):  # the one-query form used by decode agrees with row i
        o = gpt.attend_last(q[i], k[:i + 1], v[:i + 1], H, dh)
        np.testing.assert_allclose(o, brute_attention(q, k, v, H, dh)[i], atol=1e-12)


def test_causal_attention_matches_torch_sdpa():
    rng = np.random.default_rng(12)
    H, dh, T = 3, 64, 40
    q, k, v = (rng.standard_normal((T, H * dh)) for _ in range(3))
    t = lambda a: torch.from_numpy(a).reshape(T, H, dh).transpose(0, 1)  # noqa: E731
    ref = torch.nn.functional.scaled_dot_product_attention(t(q), t(k), t(v), is_causal=True)
    ref = ref.transpose(0, 1).reshape(T, H * dh).numpy()
    np.testing.assert_allclose(gpt.causal_attention(q, k, v, H, dh), ref, rtol=0, atol=1e-12)


def test_attention_special_cases():
    rng = np.random.default_rng(13)
    H, dh = 2, 64
    q, k, v = (rng.standard_normal((1, H * dh)) for _ in range(3))
    # one cached row: the output is that row's value
    np.testing.assert_allclose(gpt.attend_last(q[0], k, v, H, dh), v[0], atol=1e-15)
    # identical keys: uniform weights, output = mean of the values
    K = np.repeat(k, 9, axis=0)
    V = rng.standard_normal((9, H * dh))
    np.testing.assert_allclose(gpt.attend_last(q[0], K, V, H, dh), V.mean(axis=0), atol=1e-12)
    # a dominant key selects its value
    K = rng.standard_normal((5, H * dh)) * 0.01
    K[3] = q[0] * 100
    np.testing.assert_allclose(gpt.attend_last(q[0], K, V[:5], H, dh), V[3], atol=1e-9)


# --------------------------------------------------------------------------- whole decoder
def hf_gpt2(weights, shape):
    from transformers import GPT2Config, GPT2Model
    cfg = GPT2Config(vocab_size=shape.vocab, n_positions=shape.n_pos, n_embd=shape.d_model,
                     n_layer=shape.n_layer, n_head=shape.n_head, n_inner=shape.d_ff,
                     activation_function="gelu_new", resid_pdrop=0.0, embd_pdrop=0.0,
                     attn_pdrop=0.0, layer_norm_epsilon=1e-5, bos_token_id=0, eos_token_id=0)
    m = GPT2Model(cfg, attn_implementation="eager") if "attn_implementation" in \
        GPT2Model.__init__.__code__.co_varnames else GPT2Model(cfg)
    m = m.double().eval()
    T = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float64))  # noqa: E731
    with torch.no_grad():
        m.wte.weight.copy_(T(weights["tok_emb"]))
        m.wpe.weight.zero_()  # positions are added by the caller (the prefix gets none)
        for blk, lw in zip(m.h, weights["layers"]):
            blk.ln_1.weight.copy_(T(lw["ln1_g"]))
            blk.ln_1.bias.copy_(T(lw["ln1_b"]))
            blk.attn.c_attn.weight.copy_(T(lw["w_qkv"].T))  # GPT-2's Conv1D stores [in, out]
            blk.attn.c_attn.bias.copy_(T(lw["b_qkv"]))
            blk.attn.c_proj.weight.copy_(T(lw["w_out"].T))
            blk.attn.c_proj.bias.copy_(T(lw["b_out"]))
            blk.ln_2.weight.copy_(T(lw["ln2_g"]))
            blk.ln_2.bias.copy_(T(lw["ln2_b"]))
            blk.mlp.c_fc.weight.copy_(T(lw["w_fc1"].T))
            blk.mlp.c_fc.bias.copy_(T(lw["b_fc1"]))
            blk.mlp.c_proj.weight.copy_(T(lw["w_fc2"].T))
            blk.mlp.c_proj.bias.copy_(T(lw["b_fc2"]))
        m.ln_f.weight.copy_(T(weights["lnf_g"]))
        m.ln_f.bias.copy_(T(weights["lnf_b"]))
    return m


def hf_reference(weights, shape, rows):
    m = hf_gpt2(weights, shape)
    with torch.no_grad():
        hid = m(inputs_embeds=torch.from_numpy(rows)[None]).last_hidden_state[0].numpy()
    return hid @ weights["w_head"].T.astype(np.float64) + weights["b_head"], hid


def test_full_forward_matches_hf_gpt2():
    w, model = small_model()
    prefix = workload.prefix_embeddings([10], SMALL.d_model, seed=1, bf16=False).astype(np.float64)
    toks = np.array([3, 17, 60, 1, 1])
    rows = model.rows(prefix, toks)
    logits, hid = model.full_forward(rows)
    ref_logits, ref_hid = hf_reference(w, SMALL, rows)
    np.testing.assert_allclose(hid, ref_hid, rtol=0, atol=1e-10)
    np.testing.assert_allclose(logits, ref_logits, rtol=0, atol=1e-10)
    # decoded rows carry their own-range positions 0, 1, 2, ...; the prefix has none
    np.testing.assert_allclose(rows[10 + 2], w["tok_emb"][60] + w["pos_emb"][2], atol=0)
    np.testing.assert_array_equal(rows[:10], prefix)


def test_input_assembly_merged_table_and_position_ranges():
    """Sec. II-C adaptations 1-3: conditioning rows pass through with no position
    embedding; a text id shifted past the semantic vocabulary into the merged
    table reads the separate text table's row; text positions start at text_pos0;
    semantic ids still read the semantic block."""
    w, _ = small_model()
    d, V = SMALL.d_model, SMALL.vocab
    rng = np.random.default_rng(3)
    text = rng.standard_normal((7, d))
    merged = dict(w)
    merged["tok_emb"] = np.concatenate([w["tok_emb"], text])
    m = gpt.GPT(merged, SMALL.n_head, SMALL.d_head, dtype=np.float64)
    cond = rng.standard_normal((3, d))
    ids = np.array([4, 0, 6, 4])
    rows = m.assemble_prefix(cond, ids, text_pos0=5)
    assert rows.shape == (3 + len(ids), d)
    np.testing.assert_array_equal(rows[:3], cond)
    for i, t in enumerate(ids):
        np.testing.assert_array_equal(rows[3 + i], text[t] + w["pos_emb"][5 + i])
    np.testing.assert_array_equal(m.embed([V - 1], [2])[0],
                                  w["tok_emb"][V - 1].astype(np.float64) + w["pos_emb"][2].astype(np.float64))
    # no text: the prefix is the conditioning alone; no conditioning: text rows alone
    np.testing.assert_array_equal(m.assemble_prefix(cond, [], 0), cond)
    np.testing.assert_array_equal(m.assemble_prefix(np.zeros((0, d)), [6], 0)[0], text[6] + w["pos_emb"][0])


@pytest.mark.parametrize("dtype,tol", [(np.float64, 1e-12), (np.float32, 1e-5)])
def test_prefill_then_decode_equals_full_forward(dtype, tol):
    w, model = small_model(dtype)
    prefix = workload.prefix_embeddings([9], SMALL.d_model, seed=1, bf16=False)
    toks = workload.random_tokens(6, 1, SMALL.vocab, seed=4)[:, 0]
    full, full_h = model.full_forward(model.rows(prefix, toks))
    cache, last = model.prefill(prefix)
    np.testing.assert_allclose(last, full[8], rtol=0, atol=tol * np.abs(full[8]).max())
    for t, tok in enumerate(toks):
        lg, hn = model.decode_step(cache, tok, t)
        ref = full[9 + t]
        assert np.max(np.abs(lg - ref)) <= tol * np.max(np.abs(ref))
        assert np.max(np.abs(hn - full_h[9 + t])) <= tol * np.max(np.abs(full_h[9 + t]))
    assert cache["k"][0].shape == (9 + len(toks), SMALL.d_model)


def test_greedy_decode_agrees_with_full_forward():
    w, model = small_model()
    prefix = workload.prefix_embeddings([5], SMALL.d_model, seed=1, bf16=False)
    toks = model.greedy_decode(prefix, 6, SMALL.start_token)
    fed = np.concatenate([[SMALL.start_token], toks[:-1]])
    full, _ = model.full_forward(model.rows(prefix, fed))
    np.testing.assert_array_equal(np.argmax(full[5:], axis=1), toks)


def test_planted_mistakes_fail_the_pins(monkeypatch):
    """Each broken variant of an oracle step must be caught by the GPT-2 comparison."""
    w, model = small_model()
    prefix = workload.prefix_embeddings([6], SMALL.d_model, seed=1, bf16=False).astype(np.float64)
    rows = model.rows(prefix, [5, 9])
    ref, _ = hf_reference(w, SMALL, rows)

    def caught():
        got, _ = gpt.GPT(w, SMALL.n_head, SMALL.d_head, dtype=np.float64).full_forward(rows)
        return np.max(np.abs(got - ref)) > 1e-6

    good_ln, good_gelu, good_attn, good_lin = gpt.layer_norm, gpt.gelu, gpt.causal_attention, gpt.linear
    mutants = {
        "ln unbiased variance": ("layer_norm", lambda x, g, b, eps=1e-5: (x - x.mean(-1, keepdims=True))
                                 / np.sqrt(x.var(-1, ddof=1, keepdims=True) + eps) * g + b),
        "ln drops beta": ("layer_norm", lambda x, g, b, eps=1e-5: good_ln(x, g, 0 * b, eps)),
        "gelu sign": ("gelu", lambda u: good_gelu(-u)),
        "erf gelu": ("gelu", lambda u: u * 0.5 * (1 + np.vectorize(math.erf)(u / math.sqrt(2)))),
        "no attention scale": ("causal_attention", lambda q, k, v, H, dh: good_attn(q * 8, k, v, H, dh)),
        "non-causal": ("causal_attention", lambda q, k, v, H, dh: np.concatenate(
            [gpt.attend_last(q[i], k, v, H, dh)[None] for i in range(q.shape[0])])),
        "k and v swapped": ("causal_attention", lambda q, k, v, H, dh: good_attn(q, v, k, H, dh)),
        "bias dropped": ("linear", lambda a, W, b: a @ W.T),
        "transposed weight": ("linear", lambda a, W, b: (a @ W + b) if W.shape[0] == W.shape[1]
                              else good_lin(a, W, b)),
    }
    assert not caught()
    for name, (fn, bad) in mutants.items():
        with monkeypatch.context() as mp:
            mp.setattr(gpt, fn, bad)
            assert caught(), name


# --------------------------------------------------------------------------- quantiser
def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def test_w8_golden():
    g = _golden("quant_examples.json")["w8"]
    w = np.array(g["rows"], dtype=np.float32)
    q, s = quant.quantize_w8(w)
    np.testing.assert_array_equal(q, np.array(g["codes"], dtype=np.int8))
    np.testing.assert_array_equal(s, np.array(g["scales"], dtype=np.float32))
    np.testing.assert_array_equal(quant.to_bits(s), [int(b, 16) for b in g["scale_bits"]])


def test_w4_golden():
    g = _golden("quant_examples.json")["w4"]
    G = g["group"]
    w = np.zeros((2, 2 * G), dtype=np.float32)
    for blk in g["rows_sparse"]:
        a, b = blk["cols"]
        w[blk["row"], a:b] = blk["fill"]
        for k, v in blk["values"].items():
            w[blk["row"], a + int(k)] = v
    q, s, z = quant.quantize_w4(w, G)
    np.testing.assert_array_equal(s, np.array(g["scales"], dtype=np.float32))
    np.testing.assert_array_equal(quant.to_bits(s), [[int(b, 16) for b in r] for r in g["scale_bits"]])
    np.testing.assert_array_equal(z, np.array(g["zeros"], dtype=np.float32))
    # zero-points are non-negative integers: +0 is the only encoding of zero
    np.testing.assert_array_equal(quant.to_bits(z), [[0x4040, 0x0000], [0x4170, 0x0000]])
    h = g["codes_head"]
    np.testing.assert_array_equal(q[0, :8], h["row0_group0"])
    np.testing.assert_array_equal(q[0, G:G + 4], h["row0_group1"])
    np.testing.assert_array_equal(q[1, :4], h["row1_group0"])
    np.testing.assert_array_equal(q[1, G:G + 4], h["row1_group1"])
    assert np.all(q[0, 5:G] == 3)


def test_bf16_rounding_against_torch():
    x = np.random.default_rng(20).standard_normal(100000).astype(np.float32) * 1e-2
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    np.testing.assert_array_equal(quant.bf16_rne(x), ref)


def test_w8_exact_dequant_bounds_and_nearest_code():
    w = np.random.default_rng(21).standard_normal((64, 256)).astype(np.float32) * 0.02
    q, s = quant.quantize_w8(w)
    assert q.dtype == np.int8 and np.all(np.abs(q.astype(int)) <= 127)
    deq = quant.dequantize_w8(q, s)
    # exact: fp64 product equals the fp32 product
    np.testing.assert_array_equal(deq.astype(np.float64), q.astype(np.float64) * s[:, None].astype(np.float64))
    assert np.all(np.abs(w - deq) <= s[:, None] * 0.5 * (1 + 1e-6))
    # every row reaches a code of magnitude 127 or 126 (bf16 rounding of the scale)
    assert np.all(np.abs(q.astype(int)).max(axis=1) >= 126)
    # brute force: each code is the nearest of all 255 candidates
    cand = np.arange(-127, 128, dtype=np.float64)
    for n in range(0, 64, 7):
        err = np.abs(w[n].astype(np.float64)[:, None] - cand[None, :] * float(s[n]))
        best = cand[np.argmin(err, axis=1)]
        off = best != q[n]
        # a mismatch can only be a near-tie, where fp32 w/s sits within rounding of x.5
        ratio = w[n].astype(np.float64) / float(s[n])
        assert np.all(np.abs(np.abs(ratio[off] - np.floor(ratio[off])) - 0.5) < 1e-5)


def test_w4_exact_dequant_bounds_and_idempotence():
    w = np.random.default_rng(22).standard_normal((16, 512)).astype(np.float32) * 0.02
    q, s, z = quant.quantize_w4(w)
    assert q.dtype == np.uint8 and q.max() <= 15
    deq = quant.dequantize_w4(q, s, z)
    s_el = np.repeat(s, 128, axis=1)
    z_el = np.repeat(z, 128, axis=1)
    np.testing.assert_array_equal(deq.astype(np.float64),
                                  (q.astype(np.float64) - z_el) * s_el.astype(np.float64))
    assert np.all(np.abs(w - deq) <= s_el * (0.5 + 1.0 / 16))
    # quantising dequantised weights again is a fixed point wherever the range is
    # reproduced exactly
    q2, s2, z2 = quant.quantize_w4(deq)
    same = (s2 == s) & (z2 == z)
    assert same.mean() > 0.5
    qb = q.reshape(16, 4, 128)[same]
    q2b = q2.reshape(16, 4, 128)[same]
    np.testing.assert_array_equal(qb, q2b)


def test_w8_idempotence():
    w = np.random.default_rng(23).standard_normal((32, 128)).astype(np.float32)
    q, s = quant.quantize_w8(w)
    q2, s2 = quant.quantize_w8(quant.dequantize_w8(q, s))
    # amax of the dequantised row is 127 s (or 126 s), so the scale can only move by rounding
    keep = s2 == s
    assert keep.mean() > 0.5
    np.testing.assert_array_equal(q[keep], q2[keep])


def test_w4_packing_bit_positions_and_round_trip():
    codes = np.zeros((2, 16), dtype=np.uint8)
    codes[0, 3] = 0xA
    codes[1, 15] = 0xF
    words = quant.pack_w4(codes)
    assert words.dtype == np.int32 and words.shape == (2, 2)
    assert words.view(np.uint32)[0, 0] == 0xA << 12
    assert words.view(np.uint32)[1, 1] == 0xF0000000
    r = np.random.default_rng(24).integers(0, 16, size=(8, 256)).astype(np.uint8)
    np.testing.assert_array_equal(quant.unpack_w4(quant.pack_w4(r)), r)


# --------------------------------------------------------------------------- sampler
def test_sampler_golden():
    cases = _golden("sampler_examples.json")["cases"]
    for c in cases:
        if "logits_log_probs" in c:
            lg = np.log(np.array(c["logits_log_probs"], dtype=np.float64)) * c.get("logit_scale", 1.0)
        else:
            lg = np.array(c["logits"])
        lg = lg.astype(np.float32)
        for u, want in c["draws"]:
            tok, _ = sample.sample(lg, c["temperature"], c["top_k"], c["top_p"], np.float32(u))
            assert tok == want, (c, u)


def test_greedy_equals_argmax_with_lowest_index_ties():
    lg = np.array([1.0, 3.0, -2.0, 3.0], dtype=np.float32)
    assert sample.greedy(lg) == 1
    rng = np.random.default_rng(30)
    for _ in range(20):
        lg = rng.standard_normal(500).astype(np.float32)
        assert sample.sample(lg, 0.7, 1, 0.9, 0.3)[0] == int(torch.argmax(torch.from_numpy(lg)))


def test_full_top_k_and_p1_is_inverse_cdf():
    """k = V, p = 1 reduces to a plain categorical draw by inverse CDF."""
    rng = np.random.default_rng(31)
    V = 40
    for trial in range(30):
        lg = rng.standard_normal(V).astype(np.float32) * 2
        T = 0.8
        p = torch.softmax(torch.from_numpy(lg.astype(np.float64) / T), 0).numpy()
        order = np.lexsort((np.arange(V), -lg))
        cdf = np.cumsum(p[order])
        for u in rng.random(20):
            tok, det = sample.sample(lg, T, V, 1.0, np.float32(u))
            ref = order[min(np.searchsorted(cdf, np.float32(u), side="right"), V - 1)]
            if sample.near_boundary(det, rel=1e-5):
                continue
            assert tok == ref


def test_sampler_distribution_chi2():
    """Empirical frequencies over many uniforms match the renormalised top-k/top-p law."""
    from scipy import stats
    rng = np.random.default_rng(32)
    V, k, p, T = 16, 8, 0.9, 0.7
    lg = rng.standard_normal(V).astype(np.float32)
    # expected law, computed independently with torch: sort, keep k, softmax, nucleus cut
    z = torch.from_numpy(lg.astype(np.float64) / T)
    vals, idx = torch.sort(z, descending=True, stable=True)
    pk = torch.softmax(vals[:k], 0)
    c = torch.cumsum(pk, 0)
    n = int(torch.nonzero(c >= p * c[-1])[0]) + 1
    law = np.zeros(V)
    law[idx[:n].numpy()] = (pk[:n] / pk[:n].sum()).numpy()
    draws = 100000
    us = rng.random(draws, dtype=np.float32)
    counts = np.zeros(V)
    for u in us:
        counts[sample.sample(lg, T, k, p, u)[0]] += 1
    keep = law > 0
    assert counts[~keep].sum() == 0
    chi2, pval = stats.chisquare(counts[keep], law[keep] * draws)
    assert pval > 1e-3, (chi2, pval)


# --------------------------------------------------------------------------- quantised tensors
def test_dequantized_model_touches_exactly_the_four_linears():
    """Weight-only quantisation applies to the GPT's linear layers (Table I caption,
    Sec. III-B) and the reading is: the four per-layer matrices, nothing else.  Every
    other tensor (embeddings, LayerNorm, biases, LM head) must come back bit for bit;
    each of the 4 x L matrices must change and lie on the code grid of its mode:
    W8 rows are integer multiples in [-127, 127] of one bf16 scale per row (the largest
    |code| is 127), W4 groups of 128 are (q - z) * s with integer q, z in 0..15."""
    shape = workload.ModelShape(n_layer=3, d_model=128, n_head=2, d_head=64, d_ff=256, vocab=64, n_pos=32)
    w = workload.master_weights(shape, seed=3, threads=2)
    mats = ("w_qkv", "w_out", "w_fc1", "w_fc2")

    def bits(a):
        return np.ascontiguousarray(a, np.float32).view(np.uint32)

    for mode in ("w8", "w4"):
        dq = quant.dequantized_model(w, mode)
        assert set(dq) == set(w)
        for k in w:
            if k != "layers":
                np.testing.assert_array_equal(bits(dq[k]), bits(w[k]), err_msg=(mode, k))
        assert len(dq["layers"]) == shape.n_layer
        for l, (a, b) in enumerate(zip(w["layers"], dq["layers"])):
            assert set(a) == set(b)
            for k in a:
                if k in mats:
                    continue
                np.testing.assert_array_equal(bits(b[k]), bits(a[k]), err_msg=(mode, l, k))
            for k in mats:
                m = np.asarray(b[k], np.float64)
                assert m.shape == a[k].shape and not np.array_equal(bits(b[k]), bits(a[k])), (mode, l, k)
                if mode == "w8":
                    amax = np.max(np.abs(m), axis=1, keepdims=True)
                    s = amax / 127.0  # the row's largest code is +-127, so this is its scale
                    assert np.all(bits(s.astype(np.float32)) & 0xFFFF == 0), "scale is not a bf16"
                    c = m / s
                    np.testing.assert_array_equal(c, np.rint(c))
                    assert np.max(np.abs(c)) <= 127
                else:
                    N, K = m.shape
                    g = m.reshape(N, K // 128, 128)
                    # within a group the values are (q - z) s: their differences are multiples
                    # of s, and the 16 levels span at most 15 s around zero
                    lo, hi = g.min(axis=2), g.max(axis=2)
                    step = np.where(hi > lo, (hi - lo), 1.0)
                    for n in range(0, N, max(1, N // 7)):
                        for j in range(K // 128):
                            v = np.unique(g[n, j])
                            d = np.diff(v)
                            s = d.min() if d.size else 1.0
                            r = (v - v[0]) / s
                            np.testing.assert_allclose(r, np.rint(r), atol=1e-6)
                            assert np.rint(r[-1]) <= 15 and step[n, j] > 0
                            assert np.any(np.abs(v / s - np.rint(v / s)) < 1e-6), "no level at a multiple of s"


def test_dequantized_model_pin_catches_a_quantised_head(monkeypatch):
    """The pin above fails when the LM head or a bias is quantised too, or when a
    matrix is skipped (planted in a copy of the oracle, on the CPU)."""
    real = quant.dequantized_model

    def with_head(weights, mode, group=128):
        out = real(weights, mode, group)
        out["w_head"] = quant.dequantize_w8(*quant.quantize_w8(weights["w_head"]))
        return out

    def skip_out(weights, mode, group=128):
        out = real(weights, mode, group)
        for a, b in zip(weights["layers"], out["layers"]):
            b["w_out"] = a["w_out"]
        return out

    for planted in (with_head, skip_out):
        monkeypatch.setattr(quant, "dequantized_model", planted)
        with pytest.raises(AssertionError):
            test_dequantized_model_touches_exactly_the_four_linears()
    monkeypatch.setattr(quant, "dequantized_model", real)


def test_near_boundary_band():
    """The excuse band of the sampler parity check: a draw is 'near' exactly when
    r = u * c_n, or the top-p threshold p * c_k, lies within rel * c_k of a
    cumulative sum.  Built by hand: three kept weights with known partial sums."""
    lg = np.log(np.array([0.5, 0.3, 0.2], dtype=np.float64)).astype(np.float32)
    # cum = e / e_1 summed: [1, 1.6, 2.0] (to fp32 rounding); p = 1 so the threshold is c_3
    _, det = sample.sample(lg, 1.0, 3, 1.0, np.float32(0.25))
    cum = det["cum"].astype(np.float64)
    np.testing.assert_allclose(cum, [1.0, 1.6, 2.0], rtol=1e-6)
    c_k = cum[-1]
    # the threshold equals c_3 itself, so every draw of a p = 1 cut is within the band
    assert sample.near_boundary(det)
    # with p = 0.9 the threshold 1.8 sits 0.2 from every sum: only r decides
    for u, near in ((0.25, False), (0.5, True), (0.8, True), (0.3, False), (0.999, False)):
        _, d = sample.sample(lg, 1.0, 3, 0.9, np.float32(u))
        assert abs(float(d["thresh"]) - 1.8) < 1e-6
        r = float(d["r"])
        want = bool(np.any(np.abs(np.array(d["cum"], np.float64) - r) <= 1e-5 * c_k))
        assert want == near, (u, r)
        assert sample.near_boundary(d) == near, (u, r)
    # just inside and just outside the band around c_1 = 1 (n = 3, so r = u * c_3 = 2 u)
    for off, near in ((0.5e-5, True), (3e-5, False)):
        u = np.float32((1.0 + off * c_k) / c_k)
        _, d = sample.sample(lg, 1.0, 3, 0.9, u)
        assert sample.near_boundary(d) == near, (off, float(d["r"]))
    # greedy has no band
    _, d = sample.sample(lg, 1.0, 1, 0.9, np.float32(0.5))
    assert not sample.near_boundary(d)
