// Decode-time linear layers: y[b] = act[b] . W^T (+ bias, epilogue) for a small
// batch of rows, streaming each weight byte from HBM exactly once per call.
//
// One 256-thread workgroup owns 4 * (64 / lpr) consecutive output rows; `lpr`
// lanes share a row and walk its K dimension in 16-byte chunks, so each group
// of lanes issues fully coalesced 16-byte loads.  The fp32 activations of all
// batch rows are staged in LDS (LayerNorm applied while staging when the
// layer is preceded by one), and every weight chunk is dequantised in
// registers and multiplied against all batch rows before the next chunk.
//
// Weight storage (element size per 16-byte chunk):
//   FTTS_F32   4 fp32      FTTS_BF16  8 bf16
//   FTTS_W8A16 16 int8 codes, one bf16 scale per row (applied once at the end)
//   FTTS_W4A16 32 4-bit codes (one group of 128 spans 4 chunks); each chunk
//              contributes s * (sum q x - z * sum x), the per-chunk sums of x
//              being precomputed in LDS.
#pragma once
#include "ftts_internal.hpp"

namespace ftts {

template <int WT> struct WInfo;
template <> struct WInfo<FTTS_F32> { static constexpr int EPC = 4; };
template <> struct WInfo<FTTS_BF16> { static constexpr int EPC = 8; };
template <> struct WInfo<FTTS_W8A16> { static constexpr int EPC = 16; };
template <> struct WInfo<FTTS_W4A16> { static constexpr int EPC = 32; };

constexpr int kActFloats = 12288;  // LDS budget for staged activations (48 KB); a multiple of 128 per batch row
constexpr int kUnroll = 5;         // weight chunks in flight per lane

__host__ __device__ constexpr int k_chunk(int bmax) { return kActFloats / bmax; }

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

template <int WT, int BMAX, int EPI, bool LN>
__global__ __launch_bounds__(256) void gemv_kernel(const GemvArgs a) {
    constexpr bool F32 = (WT == FTTS_F32);
    constexpr int EPC = WInfo<WT>::EPC;
    constexpr int KC = k_chunk(BMAX);
    extern __shared__ float s_act[];              // [BMAX][min(KC, K)]
    __shared__ float s_xsum[kActFloats / 32];     // W4: per-32-column sums of the activations
    __shared__ float s_mean[BMAX], s_rstd[BMAX];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int lpr = a.lpr;
    const int li = lane & (lpr - 1);
    const int rpw = kWave / lpr;
    const int row = blockIdx.x * (4 * rpw) + wave * rpw + lane / lpr;
    const bool row_ok = row < a.N;
    const int B = a.B, K = a.K;
    const int kcs = K < KC ? K : KC;              // LDS row stride of the staged activations

    if constexpr (LN) {
        for (int b = wave; b < B; b += 4) {
            const float* xr = a.act + (size_t)b * K;
            float s = 0.f;
            for (int k = lane; k < K; k += kWave) s += xr[k];
            const float mean = wave_sum(s) / (float)K;
            float v = 0.f;
            for (int k = lane; k < K; k += kWave) {
                const float d = xr[k] - mean;
                v = fmaf(d, d, v);
            }
            v = wave_sum(v) / (float)K;
            if (lane == 0) {
                s_mean[b] = mean;
                s_rstd[b] = 1.0f / sqrtf(v + a.eps);
            }
        }
    }

    float acc[BMAX];
#pragma unroll
    for (int b = 0; b < BMAX; ++b) acc[b] = 0.f;

    size_t row_bytes;
    if constexpr (WT == FTTS_W4A16) row_bytes = (size_t)K / 2;
    else if constexpr (WT == FTTS_W8A16) row_bytes = (size_t)K;
    else row_bytes = (size_t)K * (F32 ? 4 : 2);
    const uint4* wrow = reinterpret_cast<const uint4*>(reinterpret_cast<const char*>(a.w) +
                                                       row_bytes * (size_t)(row_ok ? row : 0));
    const int n_groups = K / 128;

    for (int kc = 0; kc < K; kc += KC) {
        const int kn = (K - kc) < KC ? (K - kc) : KC;
        __syncthreads();
        for (int i = tid; i < B * kn; i += 256) {
            const int b = i / kn, k = i - b * kn;
            float v = a.act[(size_t)b * K + kc + k];
            if constexpr (LN)
                v = (v - s_mean[b]) * s_rstd[b] * ld_act<F32>(a.ln_g, kc + k) + ld_act<F32>(a.ln_b, kc + k);
            s_act[b * kcs + k] = v;
        }
        if constexpr (WT == FTTS_W4A16) {
            __syncthreads();
            const int nc = kn / 32;
            for (int i = tid; i < B * nc; i += 256) {
                const int b = i / nc, c = i - b * nc;
                const float* p = s_act + b * kcs + c * 32;
                float s = 0.f;
#pragma unroll
                for (int j = 0; j < 32; ++j) s += p[j];
                s_xsum[b * (kcs / 32) + c] = s;
            }
        }
        __syncthreads();
        if (row_ok) {
            const int nch = kn / EPC;
            const uint4* wp = wrow + kc / EPC;
            for (int c0 = li; c0 < nch; c0 += lpr * kUnroll) {
                uint4 wv[kUnroll];
#pragma unroll
                for (int u = 0; u < kUnroll; ++u) {
                    const int c = c0 + u * lpr;
                    if (c < nch) wv[u] = wp[c];
                }
#pragma unroll
                for (int u = 0; u < kUnroll; ++u) {
                    const int c = c0 + u * lpr;
                    if (c < nch) {
                        float s4 = 0.f, z4 = 0.f;
                        if constexpr (WT == FTTS_W4A16) {
                            const int g = (kc + c * 32) >> 7;
                            s4 = bf16_to_f32(a.scale[(size_t)row * n_groups + g]);
                            z4 = bf16_to_f32(a.zero[(size_t)row * n_groups + g]);
                        }
                        dot_chunk<WT, BMAX>(wv[u], s_act + c * EPC, kcs, B, acc, s4, z4, s_xsum + c,
                                            kcs / 32);
                    }
                }
            }
        }
    }

    // Reduce over the lanes of a row; every lane ends with the full sums.
#pragma unroll
    for (int b = 0; b < BMAX; ++b) {
        if (b < B) {
            float v = acc[b];
            for (int o = lpr >> 1; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
            acc[b] = v;
        }
    }
    if (!row_ok) return;

    float rs = 1.f;
    if constexpr (WT == FTTS_W8A16) rs = bf16_to_f32(a.scale[row]);
    const float bias = ld_act<F32>(a.bias, row);
#pragma unroll
    for (int b = 0; b < BMAX; ++b) {
        if (b < B && (b & (lpr - 1)) == li) {
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

template <int WT, int BMAX, int EPI, bool LN>
static hipError_t launch_one(const GemvArgs& a, hipStream_t st) {
    const int rows_per_block = 4 * (kWave / a.lpr);
    const int blocks = (a.N + rows_per_block - 1) / rows_per_block;
    const int kcs = a.K < k_chunk(BMAX) ? a.K : k_chunk(BMAX);
    const size_t lds = (size_t)BMAX * kcs * sizeof(float);
    hipLaunchKernelGGL((gemv_kernel<WT, BMAX, EPI, LN>), dim3(blocks), dim3(256), lds, st, a);
    return hipGetLastError();
}

template <int WT, int EPI, bool LN>
static hipError_t by_batch(const GemvArgs& a, hipStream_t st) {
    if (a.B <= 1) return launch_one<WT, 1, EPI, LN>(a, st);
    if (a.B <= 2) return launch_one<WT, 2, EPI, LN>(a, st);
    if (a.B <= 4) return launch_one<WT, 4, EPI, LN>(a, st);
    if (a.B <= 8) return launch_one<WT, 8, EPI, LN>(a, st);
    return launch_one<WT, 16, EPI, LN>(a, st);
}

// Instantiates the launchers of one weight type (one translation unit each).
#define FTTS_GEMV_INSTANCE(WT, NAME)                                                        \
    hipError_t NAME(int epi, bool ln, const GemvArgs& a, hipStream_t st) {                   \
        if (epi == EPI_QKV && ln) return by_batch<WT, EPI_QKV, true>(a, st);                 \
        if (epi == EPI_GELU && ln) return by_batch<WT, EPI_GELU, true>(a, st);               \
        if (epi == EPI_RESID && !ln) return by_batch<WT, EPI_RESID, false>(a, st);           \
        if (epi == EPI_STORE && ln && (WT == FTTS_F32 || WT == FTTS_BF16))                   \
            return by_batch<WT, EPI_STORE, true>(a, st);                                     \
        return hipErrorInvalidValue;                                                         \
    }

hipError_t gemv_f32(int epi, bool ln, const GemvArgs& a, hipStream_t st);
hipError_t gemv_bf16(int epi, bool ln, const GemvArgs& a, hipStream_t st);
hipError_t gemv_w8(int epi, bool ln, const GemvArgs& a, hipStream_t st);
hipError_t gemv_w4(int epi, bool ln, const GemvArgs& a, hipStream_t st);

}  // namespace ftts
