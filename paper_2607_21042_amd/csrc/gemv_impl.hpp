// Decode-time linear layers: y[b] = act[b] . W^T (+ bias, epilogue) for a small batch
// of rows, streaming each weight byte from HBM once per call.
//
// A 256-thread workgroup owns 4 * (64 / LPR) consecutive output rows; LPR lanes
// share a row and each lane owns NCH 16-byte chunks of it per pass over K
// (K = passes * LPR * NCH * elements-per-chunk).  Every global load a workgroup
// needs -- its weight chunks, their quantisation parameters and the activations
// -- is issued at the top, unrolled and branch-free, before the first barrier, so
// the kernel's latency is one memory round trip plus the streaming time.
// Activations are staged in LDS as fp32 (LayerNorm applied in place when the
// layer is preceded by one), every weight chunk is dequantised in registers and
// multiplied against all batch rows, and the LPR partial sums of a row are
// reduced with cross-lane shuffles.
//
// Weight storage (elements per 16-byte chunk):
//   FTTS_F32 4 fp32 | FTTS_BF16 8 bf16 | FTTS_W8A16 16 int8 codes, one bf16 scale
//   per row applied once at the end | FTTS_W4A16 32 4-bit codes of one 128-column
//   group; a chunk contributes s * (sum q x - z * sum x), the per-chunk sums of x
//   being formed while staging.
#pragma once
#include "ftts_internal.hpp"

namespace ftts {

template <int WT> struct WInfo;
template <> struct WInfo<FTTS_F32> { static constexpr int EPC = 4; };
template <> struct WInfo<FTTS_BF16> { static constexpr int EPC = 8; };
template <> struct WInfo<FTTS_W8A16> { static constexpr int EPC = 16; };
template <> struct WInfo<FTTS_W4A16> { static constexpr int EPC = 32; };

constexpr int kGemvLdsFloats = 24576;  // 96 KB of staged fp32 activations per workgroup

template <int WT, int BMAX>
__device__ __forceinline__ void dot_chunk(const uint4 wv, const float* __restrict__ xs, int stride, int B,
                                          float (&acc)[BMAX], float s4, float z4, const float* xsum,
                                          int xsum_stride) {
    const uint32_t wd[4] = {wv.x, wv.y, wv.z, wv.w};
    if constexpr (WT == FTTS_F32) {
#pragma unroll
        for (int b = 0; b < BMAX; ++b) {
            if (b < B) {
                const float4 x = *reinterpret_cast<const float4*>(xs + b * stride);
                float t = acc[b];
                t = fmaf(__uint_as_float(wd[0]), x.x, t);
                t = fmaf(__uint_as_float(wd[1]), x.y, t);
                t = fmaf(__uint_as_float(wd[2]), x.z, t);
                t = fmaf(__uint_as_float(wd[3]), x.w, t);
                acc[b] = t;
            }
        }
    } else if constexpr (WT == FTTS_BF16) {
        float wf[8];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            wf[2 * j] = bf16lo(wd[j]);
            wf[2 * j + 1] = bf16hi(wd[j]);
        }
#pragma unroll
        for (int b = 0; b < BMAX; ++b) {
            if (b < B) {
                const float4 x0 = *reinterpret_cast<const float4*>(xs + b * stride);
                const float4 x1 = *reinterpret_cast<const float4*>(xs + b * stride + 4);
                float t = acc[b];
                t = fmaf(wf[0], x0.x, t);
                t = fmaf(wf[1], x0.y, t);
                t = fmaf(wf[2], x0.z, t);
                t = fmaf(wf[3], x0.w, t);
                t = fmaf(wf[4], x1.x, t);
                t = fmaf(wf[5], x1.y, t);
                t = fmaf(wf[6], x1.z, t);
                t = fmaf(wf[7], x1.w, t);
                acc[b] = t;
            }
        }
    } else if constexpr (WT == FTTS_W8A16) {
        float wf[16];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
#pragma unroll
            for (int i = 0; i < 4; ++i) wf[4 * j + i] = (float)(int32_t)((int32_t)(wd[j] << (24 - 8 * i)) >> 24);
        }
#pragma unroll
        for (int b = 0; b < BMAX; ++b) {
            if (b < B) {
                float t = acc[b];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const float4 x = *reinterpret_cast<const float4*>(xs + b * stride + 4 * q);
                    t = fmaf(wf[4 * q + 0], x.x, t);
                    t = fmaf(wf[4 * q + 1], x.y, t);
                    t = fmaf(wf[4 * q + 2], x.z, t);
                    t = fmaf(wf[4 * q + 3], x.w, t);
                }
                acc[b] = t;
            }
        }
    } else {  // FTTS_W4A16
        float wf[32];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
#pragma unroll
            for (int i = 0; i < 8; ++i) wf[8 * j + i] = (float)((wd[j] >> (4 * i)) & 0xFu);
        }
#pragma unroll
        for (int b = 0; b < BMAX; ++b) {
            if (b < B) {
                float t = 0.f;
#pragma unroll
                for (int q = 0; q < 8; ++q) {
                    const float4 x = *reinterpret_cast<const float4*>(xs + b * stride + 4 * q);
                    t = fmaf(wf[4 * q + 0], x.x, t);
                    t = fmaf(wf[4 * q + 1], x.y, t);
                    t = fmaf(wf[4 * q + 2], x.z, t);
                    t = fmaf(wf[4 * q + 3], x.w, t);
                }
                t = fmaf(-z4, xsum[b * xsum_stride], t);
                acc[b] = fmaf(s4, t, acc[b]);
            }
        }
    }
}

// LPR lanes per row, NCH 16-byte chunks per lane per pass, up to BMAX batch rows.
template <int WT, int BMAX, int EPI, bool LN, int LPR, int NCH>
__global__ __launch_bounds__(256) void gemv_kernel(const GemvArgs a) {
    constexpr bool F32 = (WT == FTTS_F32);
    constexpr int EPC = WInfo<WT>::EPC;
    constexpr int RPW = kWave / LPR;
    constexpr int PK = LPR * NCH * EPC;          // K columns per pass
    extern __shared__ float s_act[];              // [BMAX][PK] (+ W4 chunk sums [BMAX][PK/32])
    __shared__ float s_mean[BMAX], s_rstd[BMAX];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int li = lane & (LPR - 1);
    const int row = blockIdx.x * (4 * RPW) + wave * RPW + lane / LPR;
    const bool row_ok = row < a.N;
    const int rr = row_ok ? row : a.N - 1;        // loads stay in bounds; results discarded
    const int B = a.B, K = a.K;
    const int n_groups = K / 128;
    float* s_xsum = s_act + BMAX * PK;

    size_t row_bytes;
    if constexpr (WT == FTTS_W4A16) row_bytes = (size_t)K / 2;
    else if constexpr (WT == FTTS_W8A16) row_bytes = (size_t)K;
    else row_bytes = (size_t)K * (F32 ? 4 : 2);
    const uint4* wrow = reinterpret_cast<const uint4*>(reinterpret_cast<const char*>(a.w) + row_bytes * rr);

    float acc[BMAX];
#pragma unroll
    for (int b = 0; b < BMAX; ++b) acc[b] = 0.f;

    constexpr int PK4 = PK / 4;                   // float4s of one staged batch row
    constexpr int NV = (BMAX * PK4 + 255) / 256;  // staged float4s per thread (<= 24 by the LDS budget)
    constexpr int NLN = LN ? (PK + 255) / 256 : 1;
    const float4* act4 = reinterpret_cast<const float4*>(a.act);
    float4* dst4 = reinterpret_cast<float4*>(s_act);
    const int total = B * PK4;

    for (int k0 = 0; k0 < K; k0 += PK) {
        // The vector-memory counter retires loads in issue order, so everything
        // the prologue waits for (activations, LayerNorm and quantisation
        // parameters) is issued before the weight stream, which then stays in
        // flight while the activations are staged and normalised (the barriers
        // below wait for LDS traffic only).
        if (k0 > 0) lds_barrier();
        float4 v[NV];
#pragma unroll
        for (int i = 0; i < NV; ++i) {
            const int j = min(tid + 256 * i, total - 1);
            const int b = j / PK4;
            v[i] = act4[((size_t)b * K + k0) / 4 + (j - b * PK4)];
        }
        float lg[NLN], lb[NLN];
        if constexpr (LN) {
#pragma unroll
            for (int i = 0; i < NLN; ++i) {
                const int k = min(tid + 256 * i, PK - 1);
                lg[i] = ld_act<F32>(a.ln_g, k);
                lb[i] = ld_act<F32>(a.ln_b, k);
            }
        }
        float s4[NCH], z4[NCH];
        if constexpr (WT == FTTS_W4A16) {
#pragma unroll
            for (int i = 0; i < NCH; ++i) {
                const int g = (k0 + (li + i * LPR) * 32) >> 7;
                s4[i] = bf16_to_f32(a.scale[(size_t)rr * n_groups + g]);
                z4[i] = bf16_to_f32(a.zero[(size_t)rr * n_groups + g]);
            }
        }
        // the weight stream of this pass
        uint4 wv[NCH];
#pragma unroll
        for (int i = 0; i < NCH; ++i) wv[i] = ld_stream(wrow + k0 / EPC + li + i * LPR);
        // Unconditional stores (clamped lanes rewrite the last element with its own
        // value) so the compiler keeps the loads above the weight stream.
#pragma unroll
        for (int i = 0; i < NV; ++i) dst4[min(tid + 256 * i, total - 1)] = v[i];
        lds_barrier();
        if constexpr (LN) {  // LN rows are single-pass (PK == K): stats from LDS, then normalise
            for (int b = wave; b < B; b += 4) {
                const float* xr = s_act + b * PK;
                float s = 0.f;
#pragma unroll
                for (int i = 0; i < PK / kWave; ++i) s += xr[lane + kWave * i];
                const float mean = wave_sum(s) / (float)PK;
                float var = 0.f;
#pragma unroll
                for (int i = 0; i < PK / kWave; ++i) {
                    const float d = xr[lane + kWave * i] - mean;
                    var = fmaf(d, d, var);
                }
                var = wave_sum(var) / (float)PK;
                if (lane == 0) {
                    s_mean[b] = mean;
                    s_rstd[b] = 1.0f / sqrtf(var + a.eps);
                }
            }
            lds_barrier();
#pragma unroll
            for (int i = 0; i < NLN; ++i) {
                const int k = tid + 256 * i;
                if (k < PK) {
#pragma unroll
                    for (int b = 0; b < BMAX; ++b)
                        if (b < B) {
                            const float y = (s_act[b * PK + k] - s_mean[b]) * s_rstd[b] * lg[i] + lb[i];
                            s_act[b * PK + k] = y;
                            if (a.hidden && blockIdx.x == 0) a.hidden[(size_t)b * PK + k] = y;
                        }
                }
            }
            lds_barrier();
        }
        if constexpr (WT == FTTS_W4A16) {
            constexpr int NC = PK / 32;
            for (int i = tid; i < B * NC; i += 256) {
                const int b = i / NC, c = i - b * NC;
                const float* p = s_act + b * PK + c * 32;
                float s = 0.f;
#pragma unroll
                for (int j = 0; j < 32; ++j) s += p[j];
                s_xsum[b * NC + c] = s;
            }
            lds_barrier();
        }
        // multiply
#pragma unroll
        for (int i = 0; i < NCH; ++i) {
            const int c = li + i * LPR;
            float sv = 0.f, zv = 0.f;
            if constexpr (WT == FTTS_W4A16) { sv = s4[i]; zv = z4[i]; }
            dot_chunk<WT, BMAX>(wv[i], s_act + c * EPC, PK, B, acc, sv, zv, s_xsum + c, PK / 32);
        }
    }

    // Reduce over the LPR lanes of a row; every lane ends with the full sums.
#pragma unroll
    for (int b = 0; b < BMAX; ++b) {
        if (b < B) {
            acc[b] = group_sum<LPR>(acc[b]);
        }
    }
    if (!row_ok) return;

    float rs = 1.f;
    if constexpr (WT == FTTS_W8A16) rs = bf16_to_f32(a.scale[row]);
    const float bias = ld_act<F32>(a.bias, row);
#pragma unroll
    for (int b = 0; b < BMAX; ++b) {
        if (b < B && (b & (LPR - 1)) == li) {
            const float v = fmaf(acc[b], rs, bias);
            float* o = a.out + (size_t)b * a.out_stride + row;
            if constexpr (EPI == EPI_STORE) {
                *o = v;
            } else if constexpr (EPI == EPI_GELU) {
                *o = gelu_tanh(v);
            } else if constexpr (EPI == EPI_RESID) {
                *o += v;
            } else {  // EPI_QKV: keep q/k/v in fp32 and append k, v to the paged cache
                *o = v;
                const int d = a.kv.d_model;
                if (row >= d && a.kv.active[b]) {
                    const int kvsel = row >= 2 * d;
                    const int r = row - d - kvsel * d;
                    const int slot = a.kv.seq_lens[b];
                    const int phys = a.kv.block_table[(size_t)b * a.kv.max_pages + slot / kPage];
                    const size_t off = kv_offset(a.kv.layer, a.kv.n_pages, phys, kvsel, a.kv.n_head,
                                                 r / kHeadDim, slot % kPage) + (r % kHeadDim);
                    st_act<F32>(a.kv.base, off, v);
                }
            }
        }
    }
}

// (LPR, NCH) tilings of one pass over K that the launchers instantiate.
struct Tiling {
    int lpr, nch;
};

template <int WT, int BMAX, int EPI, bool LN, int LPR, int NCH>
static hipError_t launch_tiled(const GemvArgs& a, hipStream_t st) {
    constexpr int RPB = 4 * (kWave / LPR);
    constexpr int PK = LPR * NCH * WInfo<WT>::EPC;
    const int blocks = (a.N + RPB - 1) / RPB;
    const size_t lds = (size_t)BMAX * PK * sizeof(float) + (WT == FTTS_W4A16 ? (size_t)BMAX * (PK / 32) * 4 : 0);
    if (lds > 65536) {
        static bool raised = false;  // once per instantiation
        if (!raised) {
            const hipError_t e = hipFuncSetAttribute(
                reinterpret_cast<const void*>(&gemv_kernel<WT, BMAX, EPI, LN, LPR, NCH>),
                hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
            if (e != hipSuccess) return e;
            raised = true;
        }
    }
    hipLaunchKernelGGL((gemv_kernel<WT, BMAX, EPI, LN, LPR, NCH>), dim3(blocks), dim3(256), lds, st, a);
    return hipGetLastError();
}

#define FTTS_TILE_CASE(L, C) \
    if (t.lpr == L && t.nch == C) return launch_tiled<WT, BMAX, EPI, LN, L, C>(a, st);

template <int WT, int BMAX, int EPI, bool LN>
static hipError_t by_tiling(const GemvArgs& a, Tiling t, hipStream_t st) {
    FTTS_TILE_CASE(64, 10) FTTS_TILE_CASE(64, 5) FTTS_TILE_CASE(64, 4) FTTS_TILE_CASE(32, 5)
    FTTS_TILE_CASE(32, 4) FTTS_TILE_CASE(16, 5) FTTS_TILE_CASE(16, 4) FTTS_TILE_CASE(16, 2)
    FTTS_TILE_CASE(8, 5) FTTS_TILE_CASE(8, 4) FTTS_TILE_CASE(8, 2) FTTS_TILE_CASE(8, 1)
    return hipErrorInvalidValue;
}
#undef FTTS_TILE_CASE

template <int WT, int EPI, bool LN>
static hipError_t by_batch(const GemvArgs& a, Tiling t, hipStream_t st) {
    if (a.B <= 1) return by_tiling<WT, 1, EPI, LN>(a, t, st);
    if (a.B <= 4) return by_tiling<WT, 4, EPI, LN>(a, t, st);
    return by_tiling<WT, 16, EPI, LN>(a, t, st);
}

// LayerNorm-fused layers (q/k/v, FC1 + GELU, LM head) and residual layers (out-proj,
// FC2) are instantiated in separate translation units per weight type.
template <int WT>
static hipError_t gemv_dispatch_ln(int epi, const GemvArgs& a, Tiling t, hipStream_t st) {
    if (epi == EPI_QKV) return by_batch<WT, EPI_QKV, true>(a, t, st);
    if (epi == EPI_GELU) return by_batch<WT, EPI_GELU, true>(a, t, st);
    if constexpr (WT == FTTS_F32 || WT == FTTS_BF16)
        if (epi == EPI_STORE) return by_batch<WT, EPI_STORE, true>(a, t, st);
    return hipErrorInvalidValue;
}

template <int WT>
static hipError_t gemv_dispatch_res(int epi, const GemvArgs& a, Tiling t, hipStream_t st) {
    if (epi == EPI_RESID) return by_batch<WT, EPI_RESID, false>(a, t, st);
    return hipErrorInvalidValue;
}

hipError_t gemv_ln_f32(int epi, const GemvArgs& a, Tiling t, hipStream_t st);
hipError_t gemv_ln_bf16(int epi, const GemvArgs& a, Tiling t, hipStream_t st);
hipError_t gemv_ln_w8(int epi, const GemvArgs& a, Tiling t, hipStream_t st);
hipError_t gemv_ln_w4(int epi, const GemvArgs& a, Tiling t, hipStream_t st);
hipError_t gemv_res_f32(int epi, const GemvArgs& a, Tiling t, hipStream_t st);
hipError_t gemv_res_bf16(int epi, const GemvArgs& a, Tiling t, hipStream_t st);
hipError_t gemv_res_w8(int epi, const GemvArgs& a, Tiling t, hipStream_t st);
hipError_t gemv_res_w4(int epi, const GemvArgs& a, Tiling t, hipStream_t st);

}  // namespace ftts
