// Dense contractions of the prefill: C[M][N] = A[M][K] . W[N][K]^T with fused
// epilogues (bias, q/k/v store + paged KV scatter, GELU, residual add).
//
// 16-bit modes: bf16 MFMA (v_mfma_f32_32x32x16_bf16, gfx950).  A 256-thread
// block computes a 64x64 tile as a 2x2 grid of waves, each wave one 32x32
// accumulator; 64x32 tiles of A and W go through double-buffered LDS.
// Quantised weights are expanded to bf16 exactly while staging (an int8 code,
// or a 4-bit code minus its zero-point, is an integer below 2^8), and their
// scales are applied to fp32 accumulators: once per row for W8A16, once per
// 128-column group for W4A16.  So the product is exact up to fp32 accumulation
// against the same dequantised weights the decode path uses.
//
// FTTS_F32 mode: a plain fp32 FMA tile kernel (4x4 outputs per thread).
#include "ftts_internal.hpp"

namespace ftts {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int GBM = 64, GBN = 64, GBK = 32, GLDK = GBK + 8;

// Epilogue of one output element.
template <bool F32, int EPI>
__device__ __forceinline__ void gemm_epilogue(const GemmArgs& a, int m, int n, float v) {
    v += ld_act<F32>(a.bias, n);
    if constexpr (EPI == EPI_RESID) {
        float* o = reinterpret_cast<float*>(a.out) + (size_t)m * a.N + n;
        *o += v;
    } else if constexpr (EPI == EPI_GELU) {
        st_act<F32>(a.out, (size_t)m * a.N + n, gelu_tanh(v));
    } else {
        st_act<F32>(a.out, (size_t)m * a.N + n, v);
        if constexpr (EPI == EPI_QKV) {
            const int d = a.kv.d_model;
            if (n >= d) {
                int sq = 0;
                while (sq + 1 < a.seqs.n && a.seqs.cu[sq + 1] <= m) ++sq;
                const int t = m - a.seqs.cu[sq];
                const int page = t / kPage;
                if (page < a.kv.max_pages) {
                    const int phys = a.kv.block_table[(size_t)sq * a.kv.max_pages + page];
                    if (phys >= 0 && phys < a.kv.n_pages) {
                        const int kvsel = n >= 2 * d;
                        const int r = n - d - kvsel * d;
                        const size_t off = kv_offset(a.kv.layer, a.kv.n_pages, phys, kvsel, a.kv.n_head,
                                                     r / kHeadDim, t % kPage) + (r % kHeadDim);
                        st_act<F32>(a.kv.base, off, v);
                    }
                }
            }
        }
    }
}

// Stage 8 consecutive k of one W row as bf16 (exact expansion of quantised codes).
template <int WT>
__device__ __forceinline__ uint4 load_w8elems(const GemmArgs& a, int n, int k) {
    if (n >= a.N) return make_uint4(0, 0, 0, 0);
    if constexpr (WT == FTTS_BF16) {
        return *reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(a.w) + (size_t)n * a.K + k);
    } else if constexpr (WT == FTTS_W8A16) {
        const uint2 q = *reinterpret_cast<const uint2*>(reinterpret_cast<const int8_t*>(a.w) + (size_t)n * a.K + k);
        uint32_t h[8];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            h[i] = (uint32_t)f32_to_bf16((float)(int32_t)((int32_t)(q.x << (24 - 8 * i)) >> 24));
            h[4 + i] = (uint32_t)f32_to_bf16((float)(int32_t)((int32_t)(q.y << (24 - 8 * i)) >> 24));
        }
        return make_uint4(h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16));
    } else {  // W4A16: (code - zero) for the 8 codes of one packed word
        const uint32_t word = reinterpret_cast<const uint32_t*>(a.w)[(size_t)n * (a.K / 8) + k / 8];
        const float z = bf16_to_f32(a.zero[(size_t)n * (a.K / 128) + k / 128]);
        uint32_t h[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) h[i] = (uint32_t)f32_to_bf16((float)((word >> (4 * i)) & 0xFu) - z);
        return make_uint4(h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16));
    }
}

template <int WT, int EPI>
__global__ __launch_bounds__(256) void gemm_mfma_kernel(const GemmArgs a) {
    __shared__ __attribute__((aligned(16))) uint16_t sA[2][GBM * GLDK];
    __shared__ __attribute__((aligned(16))) uint16_t sB[2][GBN * GLDK];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int m0 = blockIdx.y * GBM, n0 = blockIdx.x * GBN;
    const int lr = tid >> 2, lk = (tid & 3) * 8;   // staging: row, first k of this thread
    const int am = m0 + lr, bn = n0 + lr;
    const uint16_t* A = reinterpret_cast<const uint16_t*>(a.a);

    f32x16_t acc, accg;
#pragma unroll
    for (int i = 0; i < 16; ++i) { acc[i] = 0.f; accg[i] = 0.f; }

    const int nk = a.K / GBK;
    uint4 ra = am < a.M ? *reinterpret_cast<const uint4*>(A + (size_t)am * a.K + lk) : make_uint4(0, 0, 0, 0);
    uint4 rb = load_w8elems<WT>(a, bn, lk);
    *reinterpret_cast<uint4*>(&sA[0][lr * GLDK + lk]) = ra;
    *reinterpret_cast<uint4*>(&sB[0][lr * GLDK + lk]) = rb;
    __syncthreads();

    const int fr = lane & 31, fk = (lane >> 5) * 8;  // MFMA operand row and k offset of this lane
    const int my_n = n0 + wn * 32 + fr;              // output column of every accumulator of this lane
    for (int kt = 0; kt < nk; ++kt) {
        const int buf = kt & 1;
        if (kt + 1 < nk) {
            const int k1 = (kt + 1) * GBK + lk;
            ra = am < a.M ? *reinterpret_cast<const uint4*>(A + (size_t)am * a.K + k1) : make_uint4(0, 0, 0, 0);
            rb = load_w8elems<WT>(a, bn, k1);
        }
#pragma unroll
        for (int kk = 0; kk < GBK; kk += 16) {
            const bf16x8_t av = *reinterpret_cast<const bf16x8_t*>(&sA[buf][(wm * 32 + fr) * GLDK + kk + fk]);
            const bf16x8_t bv = *reinterpret_cast<const bf16x8_t*>(&sB[buf][(wn * 32 + fr) * GLDK + kk + fk]);
            if constexpr (WT == FTTS_W4A16) accg = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, bv, accg, 0, 0, 0);
            else acc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, bv, acc, 0, 0, 0);
        }
        if constexpr (WT == FTTS_W4A16) {
            if (((kt + 1) * GBK) % 128 == 0) {  // end of a quantisation group: apply its scale
                const int g = (kt * GBK) / 128;
                const float s = my_n < a.N ? bf16_to_f32(a.scale[(size_t)my_n * (a.K / 128) + g]) : 0.f;
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    acc[i] = fmaf(s, accg[i], acc[i]);
                    accg[i] = 0.f;
                }
            }
        }
        if (kt + 1 < nk) {
            *reinterpret_cast<uint4*>(&sA[buf ^ 1][lr * GLDK + lk]) = ra;
            *reinterpret_cast<uint4*>(&sB[buf ^ 1][lr * GLDK + lk]) = rb;
        }
        __syncthreads();
    }

    constexpr bool F32 = false;
    if (my_n >= a.N) return;
    float rs = 1.f;
    if constexpr (WT == FTTS_W8A16) rs = bf16_to_f32(a.scale[my_n]);
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        const int m = m0 + wm * 32 + (i >> 2) * 8 + (lane >> 5) * 4 + (i & 3);
        if (m < a.M) gemm_epilogue<F32, EPI>(a, m, my_n, acc[i] * rs);
    }
}

// fp32 tile GEMM: 64x64 outputs per 256-thread block, 4x4 per thread, k-tiles of 16.
template <int EPI>
__global__ __launch_bounds__(256) void gemm_f32_kernel(const GemmArgs a) {
    __shared__ float sA[16][64 + 4];
    __shared__ float sB[16][64 + 4];
    const int tid = threadIdx.x, ty = tid >> 4, tx = tid & 15;
    const int m0 = blockIdx.y * 64, n0 = blockIdx.x * 64;
    const float* A = reinterpret_cast<const float*>(a.a);
    const float* W = reinterpret_cast<const float*>(a.w);
    float acc[4][4] = {};
    const int lr = tid >> 2, lk = (tid & 3) * 4;
    for (int k0 = 0; k0 < a.K; k0 += 16) {
        const int am = m0 + lr, bn = n0 + lr;
        float4 va = am < a.M ? *reinterpret_cast<const float4*>(A + (size_t)am * a.K + k0 + lk) : make_float4(0, 0, 0, 0);
        float4 vb = bn < a.N ? *reinterpret_cast<const float4*>(W + (size_t)bn * a.K + k0 + lk) : make_float4(0, 0, 0, 0);
        __syncthreads();
        sA[lk + 0][lr] = va.x; sA[lk + 1][lr] = va.y; sA[lk + 2][lr] = va.z; sA[lk + 3][lr] = va.w;
        sB[lk + 0][lr] = vb.x; sB[lk + 1][lr] = vb.y; sB[lk + 2][lr] = vb.z; sB[lk + 3][lr] = vb.w;
        __syncthreads();
#pragma unroll
        for (int k = 0; k < 16; ++k) {
            float av[4], bv[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) { av[i] = sA[k][ty * 4 + i]; bv[i] = sB[k][tx * 4 + i]; }
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(av[i], bv[j], acc[i][j]);
        }
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int m = m0 + ty * 4 + i, n = n0 + tx * 4 + j;
            if (m < a.M && n < a.N) gemm_epilogue<true, EPI>(a, m, n, acc[i][j]);
        }
}

template <int WT>
static hipError_t mfma_by_epi(int epi, const GemmArgs& a, dim3 g, hipStream_t st) {
    switch (epi) {
        case EPI_STORE: hipLaunchKernelGGL((gemm_mfma_kernel<WT, EPI_STORE>), g, dim3(256), 0, st, a); break;
        case EPI_QKV: hipLaunchKernelGGL((gemm_mfma_kernel<WT, EPI_QKV>), g, dim3(256), 0, st, a); break;
        case EPI_GELU: hipLaunchKernelGGL((gemm_mfma_kernel<WT, EPI_GELU>), g, dim3(256), 0, st, a); break;
        case EPI_RESID: hipLaunchKernelGGL((gemm_mfma_kernel<WT, EPI_RESID>), g, dim3(256), 0, st, a); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_gemm(int wdtype, int epi, const GemmArgs& a, hipStream_t st) {
    const dim3 g((a.N + 63) / 64, (a.M + 63) / 64);
    switch (wdtype) {
        case FTTS_F32:
            switch (epi) {
                case EPI_STORE: hipLaunchKernelGGL(gemm_f32_kernel<EPI_STORE>, g, dim3(256), 0, st, a); break;
                case EPI_QKV: hipLaunchKernelGGL(gemm_f32_kernel<EPI_QKV>, g, dim3(256), 0, st, a); break;
                case EPI_GELU: hipLaunchKernelGGL(gemm_f32_kernel<EPI_GELU>, g, dim3(256), 0, st, a); break;
                case EPI_RESID: hipLaunchKernelGGL(gemm_f32_kernel<EPI_RESID>, g, dim3(256), 0, st, a); break;
                default: return hipErrorInvalidValue;
            }
            return hipGetLastError();
        case FTTS_BF16: return mfma_by_epi<FTTS_BF16>(epi, a, g, st);
        case FTTS_W8A16: return mfma_by_epi<FTTS_W8A16>(epi, a, g, st);
        case FTTS_W4A16: return mfma_by_epi<FTTS_W4A16>(epi, a, g, st);
    }
    return hipErrorInvalidValue;
}

}  // namespace ftts
