"""Oracle: weight-only quantisation of the GPT linears (W8A16 and W4A16).

TEST INFRASTRUCTURE ONLY -- see the package docstring.

The paper quantises only the GPT's weights, to 8 or 4 bits, keeping
activations in 16-bit floating point (Table I caption; Sec. III-B).  It does not
say how the codes are chosen, so this module fixes one reading, bit for bit:

W8A16, symmetric, one scale per output row n:
    amax = max_k |W[n,k]|
    s    = bf16(amax / 127)            (IEEE fp32 division, then round to nearest
                                         bf16, ties to even; s = 1 if that is 0)
    q    = clamp(rint(W[n,k] / s), -127, 127)      as int8
    dequantised weight = q * s          (exact in fp32)

W4A16, asymmetric, one (scale, zero) per output row n and group g of G
consecutive k (G = 128):
    mn = min(0, min of the group),  mx = max(0, max of the group)
         (the range always holds zero, so the zero-point lies in 0..15)
    s    = bf16((mx - mn) / 15)         (s = 1 if that is 0)
    z    = clamp(rint(-mn / s), 0, 15)  stored as a bf16 (an integer, exact;
                                         zero is +0, never the negative zero
                                         that rint(-0 / s) yields)
    q    = clamp(rint(W[n,k] / s) + z, 0, 15)
    dequantised weight = (q - z) * s    (exact in fp32)
    packing: word[n][k // 8] holds q of column k in bits 4*(k%8) .. 4*(k%8)+3.

``rint`` rounds half to even; every division is one IEEE fp32 division.
"""
from __future__ import annotations

import numpy as np


def bf16_rne(x):
    """Round fp32 values to the nearest bfloat16, ties to even (finite inputs), as fp32."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    u = (u + 0x7FFF + lsb) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32).reshape(x.shape)


def to_bits(x):
    """bf16 bit patterns (uint16) of fp32 values that are bf16-representable."""
    bits = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    assert not np.any(bits & 0xFFFF), "not bf16-representable"
    return (bits >> 16).astype(np.uint16)


def from_bits(b):
    """fp32 values of bf16 bit patterns."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def quantize_w8(w):
    """Per-row symmetric int8 codes and bf16 scales: returns (codes int8 [N,K], scales fp32 [N])."""
    w = np.asarray(w, dtype=np.float32)
    amax = np.max(np.abs(w), axis=1)
    s = bf16_rne(amax / np.float32(127.0))
    s = np.where(s == 0, np.float32(1.0), s).astype(np.float32)
    q = np.rint(w / s[:, None])
    q = np.clip(q, -127, 127).astype(np.int8)
    return q, s


def dequantize_w8(codes, scales):
    return codes.astype(np.float32) * np.asarray(scales, np.float32)[:, None]


def quantize_w4(w, group=128):
    """Group-wise asymmetric 4-bit codes.

    Returns (codes uint8 [N,K] in 0..15, scales fp32 [N,K/G], zeros fp32 [N,K/G]).
    """
    w = np.asarray(w, dtype=np.float32)
    N, K = w.shape
    if K % group:
        raise ValueError("K must be a multiple of the group size")
    g = w.reshape(N, K // group, group)
    mn = np.minimum(g.min(axis=2), np.float32(0.0))
    mx = np.maximum(g.max(axis=2), np.float32(0.0))
    s = bf16_rne((mx - mn) / np.float32(15.0))
    s = np.where(s == 0, np.float32(1.0), s).astype(np.float32)
    z = np.clip(np.rint(-mn / s), 0, 15).astype(np.float32) + np.float32(0.0)  # -0 -> +0
    q = np.rint(g / s[:, :, None]) + z[:, :, None]
    q = np.clip(q, 0, 15).astype(np.uint8).reshape(N, K)
    return q, s, z


def dequantize_w4(codes, scales, zeros, group=128):
    N, K = codes.shape
    q = codes.astype(np.float32).reshape(N, K // group, group)
    return ((q - zeros[:, :, None]) * scales[:, :, None]).reshape(N, K)


def pack_w4(codes):
    """Pack 4-bit codes [N,K] into int32 words [N,K/8], column k at bits 4*(k%8)."""
    N, K = codes.shape
    c = codes.astype(np.uint32).reshape(N, K // 8, 8)
    word = np.zeros((N, K // 8), dtype=np.uint32)
    for j in range(8):
        word |= c[:, :, j] << np.uint32(4 * j)
    return word.view(np.int32)


def unpack_w4(words):
    """Inverse of pack_w4."""
    N, W = words.shape
    u = np.asarray(words).view(np.uint32)
    out = np.empty((N, W, 8), dtype=np.uint8)
    for j in range(8):
        out[:, :, j] = (u >> np.uint32(4 * j)) & 0xF
    return out.reshape(N, W * 8)


def dequantized_model(weights, mode, group=128):
    """Copy of a weights dict whose four per-layer matrices are replaced by their
    quantise-then-dequantise values (mode 'w8' or 'w4'); other tensors unchanged."""
    out = {k: v for k, v in weights.items() if k != "layers"}
    out["layers"] = []
    for lw in weights["layers"]:
        nl = dict(lw)
        for name in ("w_qkv", "w_out", "w_fc1", "w_fc2"):
            if mode == "w8":
                nl[name] = dequantize_w8(*quantize_w8(lw[name]))
            elif mode == "w4":
                nl[name] = dequantize_w4(*quantize_w4(lw[name], group), group)
            else:
                raise ValueError(mode)
        out["layers"].append(nl)
    return out
