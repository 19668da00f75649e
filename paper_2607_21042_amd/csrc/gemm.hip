// Dense contractions of the prefill: C[M][N] = A[M][K] . W[N][K]^T with fused
// epilogues (bias, q/k/v store + paged KV scatter, GELU, residual add).
//
// 16-bit modes: bf16 MFMA (v_mfma_f32_32x32x16_bf16, gfx950).  A 256-thread
// block computes a (64*MT) x 128 tile as a 2x2 grid of waves, each wave MT x 2
// accumulators of 32x32, over 64-column K steps: 16*MT matrix instructions per
// wave between barriers, while the next step's tiles of A and W are in flight
// into registers (raw codes for quantised weights) and then stored to the other
// LDS buffer.  Quantised weights are expanded to bf16 exactly at that store (an
// int8 code, or a 4-bit code minus its zero-point, is an integer below 2^8), and
// their scales are applied to fp32 accumulators: once per row for W8A16, once
// per 128-column group for W4A16.  So the product is exact up to fp32
// accumulation against the same dequantised weights the decode path uses.
//
// Small M (short prefixes) leaves too few tiles for 256 CUs, so K is split into
// S slices of whole 128-column blocks; every slice stores its fp32 partial tile
// and the last of a tile's S workgroups to arrive (a per-tile counter) adds the
// partials in slice order -- reproducible whatever the arrival order -- and
// runs the epilogue.
//
// FTTS_F32 mode: a plain fp32 FMA tile kernel (4x4 outputs per thread).
#include <algorithm>

#include "ftts_internal.hpp"

namespace ftts {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int GBM = 64, GBN = 64, GBK = 32, GLDK = GBK + 8;

// Where row m of a packed prefill batch lands in the KV pool: its physical
// page (-1 if the page table does not cover it) and slot within the page.
struct RowSlot { int phys, slot; };
__device__ __forceinline__ RowSlot row_slot(const GemmArgs& a, int m) {
    int lo = 0, hi = a.seqs.n - 1;  // the sequence holding row m: cu[sq] <= m < cu[sq + 1]
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (a.seqs.cu[mid] <= m) lo = mid;
        else hi = mid - 1;
    }
    const int t = m - a.seqs.cu[lo], page = t / kPage;
    int phys = -1;
    if (page < a.kv.max_pages) {
        phys = a.kv.block_table[(size_t)lo * a.kv.max_pages + page];
        if (phys < 0 || phys >= a.kv.n_pages) phys = -1;
    }
    return RowSlot{phys, t % kPage};
}

// Epilogue of one output element (rs: the row's KV destination, EPI_QKV only).
template <bool F32, int EPI>
__device__ __forceinline__ void gemm_epilogue(const GemmArgs& a, int m, int n, float v, RowSlot rs) {
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
            if (n >= d && rs.phys >= 0) {
                const int kvsel = n >= 2 * d;
                const int r = n - d - kvsel * d;
                const size_t off = kv_offset(a.kv.layer, a.kv.n_pages, rs.phys, kvsel, a.kv.n_head, r / kHeadDim,
                                             rs.slot) + (r % kHeadDim);
                st_act<F32>(a.kv.base, off, v);
            }
        }
    }
}

// Raw staging of one thread's share of a 128 x 64 W tile: 4 chunks of 8 k.
template <int WT> struct WStage;
template <> struct WStage<FTTS_BF16> { uint4 v[4]; };
template <> struct WStage<FTTS_W8A16> { uint2 v[4]; };
template <> struct WStage<FTTS_W4A16> { uint32_t v[4]; uint16_t z[4]; };

constexpr int G2N = 128, G2K = 64, G2LD = G2K + 8;  // tile columns, K step, LDS row pitch (bf16)
constexpr int kGemmMaxSplits = 8;

template <int WT>
__device__ __forceinline__ WStage<WT> stage_w(const GemmArgs& a, int n0, int k0) {
    WStage<WT> ws;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int idx = threadIdx.x + 256 * i, n = min(n0 + (idx >> 3), a.N - 1), k = k0 + (idx & 7) * 8;
        if constexpr (WT == FTTS_BF16) {
            ws.v[i] = *reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(a.w) + (size_t)n * a.K + k);
        } else if constexpr (WT == FTTS_W8A16) {
            ws.v[i] = *reinterpret_cast<const uint2*>(reinterpret_cast<const int8_t*>(a.w) + (size_t)n * a.K + k);
        } else {
            ws.v[i] = reinterpret_cast<const uint32_t*>(a.w)[(size_t)n * (a.K / 8) + k / 8];
            ws.z[i] = a.zero[(size_t)n * (a.K / 128) + k / 128];
        }
    }
    return ws;
}

template <int WT>
__device__ __forceinline__ uint4 expand_w(const WStage<WT>& ws, int i) {
    if constexpr (WT == FTTS_BF16) {
        return ws.v[i];
    } else if constexpr (WT == FTTS_W8A16) {
        const uint2 q = ws.v[i];
        uint32_t h[8];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            h[j] = (uint32_t)f32_to_bf16((float)(int32_t)((int32_t)(q.x << (24 - 8 * j)) >> 24));
            h[4 + j] = (uint32_t)f32_to_bf16((float)(int32_t)((int32_t)(q.y << (24 - 8 * j)) >> 24));
        }
        return make_uint4(h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16));
    } else {
        const uint32_t word = ws.v[i];
        const float z = bf16_to_f32(ws.z[i]);
        uint32_t h[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) h[j] = (uint32_t)f32_to_bf16((float)((word >> (4 * j)) & 0xFu) - z);
        return make_uint4(h[0] | (h[1] << 16), h[2] | (h[3] << 16), h[4] | (h[5] << 16), h[6] | (h[7] << 16));
    }
}

template <int AV> struct AStage { uint4 v[AV]; };
template <int AV>
__device__ __forceinline__ AStage<AV> stage_a(const uint16_t* A, const GemmArgs& a, int m0, int k0) {
    AStage<AV> r;
#pragma unroll
    for (int i = 0; i < AV; ++i) {
        const int idx = threadIdx.x + 256 * i, m = min(m0 + (idx >> 3), a.M - 1);
        r.v[i] = *reinterpret_cast<const uint4*>(A + (size_t)m * a.K + k0 + (idx & 7) * 8);
    }
    return r;
}

// Registers -> LDS buffer (quantised codes expanded here, after their loads are in).
template <int WT, int AV>
__device__ __forceinline__ void store_stage(const AStage<AV>& ra, const WStage<WT>& rw, uint16_t* sA, uint16_t* sB) {
#pragma unroll
    for (int i = 0; i < AV; ++i) {
        const int idx = threadIdx.x + 256 * i;
        *reinterpret_cast<uint4*>(&sA[(idx >> 3) * G2LD + (idx & 7) * 8]) = ra.v[i];
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int idx = threadIdx.x + 256 * i;
        *reinterpret_cast<uint4*>(&sB[(idx >> 3) * G2LD + (idx & 7) * 8]) = expand_w<WT>(rw, i);
    }
}

template <int WT, int EPI, int MT>
__global__ __launch_bounds__(256, 2) void gemm_mfma_kernel(const GemmArgs a) {
    constexpr int BM = 64 * MT, AV = BM * G2K / 8 / 256;  // A uint4 per thread per step
    __shared__ __attribute__((aligned(16))) uint16_t sA[2][BM * G2LD];
    __shared__ __attribute__((aligned(16))) uint16_t sB[2][G2N * G2LD];
    __shared__ int s_last;
    __shared__ RowSlot s_rows[EPI == EPI_QKV ? BM : 1];  // KV destination of each row of the tile
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int m0 = blockIdx.y * BM, n0 = blockIdx.x * G2N;
    if constexpr (EPI == EPI_QKV) {
        if (tid < BM) s_rows[tid] = row_slot(a, min(m0 + tid, a.M - 1));  // read after the first barrier
    }
    const int S = gridDim.z, sl = blockIdx.z;
    const int nb = a.K / G2K;  // K steps
    // this slice's K steps: whole 128-column blocks when split
    const int kb0 = S > 1 ? 2 * (sl * (nb / 2) / S) : 0, kb1 = S > 1 ? 2 * ((sl + 1) * (nb / 2) / S) : nb;
    const uint16_t* A = reinterpret_cast<const uint16_t*>(a.a);
    const int fr = lane & 31, fh = lane >> 5;


    f32x16_t acc[MT][2], accg[WT == FTTS_W4A16 ? MT : 1][2];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int nt = 0; nt < 2; ++nt)
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                acc[mt][nt][i] = 0.f;
                if constexpr (WT == FTTS_W4A16) accg[mt][nt][i] = 0.f;
            }
    // the output columns of this lane's accumulators
    const int nl0 = n0 + wn * 64 + fr, nl1 = nl0 + 32;

    AStage<AV> ra = stage_a<AV>(A, a, m0, kb0 * G2K);
    WStage<WT> rw = stage_w<WT>(a, n0, kb0 * G2K);
    store_stage<WT, AV>(ra, rw, sA[0], sB[0]);
    __syncthreads();
    float sc[2] = {0.f, 0.f};
    for (int kt = kb0; kt < kb1; ++kt) {
        const int buf = (kt - kb0) & 1;
        if (kt + 1 < kb1) {
            ra = stage_a<AV>(A, a, m0, (kt + 1) * G2K);
            rw = stage_w<WT>(a, n0, (kt + 1) * G2K);
        }
        if constexpr (WT == FTTS_W4A16) {
            if ((kt & 1) == 0) {  // this 128-column group's scales, used when it ends
                const int g = kt / 2;
                sc[0] = bf16_to_f32(a.scale[(size_t)min(nl0, a.N - 1) * (a.K / 128) + g]);
                sc[1] = bf16_to_f32(a.scale[(size_t)min(nl1, a.N - 1) * (a.K / 128) + g]);
            }
        }
#pragma unroll
        for (int kk = 0; kk < G2K; kk += 16) {
            bf16x8_t av[MT], bv[2];
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
                av[mt] = *reinterpret_cast<const bf16x8_t*>(&sA[buf][(wm * 32 * MT + mt * 32 + fr) * G2LD + kk + fh * 8]);
#pragma unroll
            for (int nt = 0; nt < 2; ++nt)
                bv[nt] = *reinterpret_cast<const bf16x8_t*>(&sB[buf][(wn * 64 + nt * 32 + fr) * G2LD + kk + fh * 8]);
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int nt = 0; nt < 2; ++nt) {
                    if constexpr (WT == FTTS_W4A16)
                        accg[mt][nt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[mt], bv[nt], accg[mt][nt], 0, 0, 0);
                    else
                        acc[mt][nt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[mt], bv[nt], acc[mt][nt], 0, 0, 0);
                }
        }
        if constexpr (WT == FTTS_W4A16) {
            if (kt & 1) {  // end of a quantisation group: apply its scale
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                    for (int nt = 0; nt < 2; ++nt)
#pragma unroll
                        for (int i = 0; i < 16; ++i) {
                            acc[mt][nt][i] = fmaf(sc[nt], accg[mt][nt][i], acc[mt][nt][i]);
                            accg[mt][nt][i] = 0.f;
                        }
            }
        }
        if (kt + 1 < kb1) store_stage<WT, AV>(ra, rw, sA[buf ^ 1], sB[buf ^ 1]);  // last read before the previous barrier
        __syncthreads();
    }

    auto row_of = [&](int mt, int i) { return m0 + wm * 32 * MT + mt * 32 + (i >> 2) * 8 + fh * 4 + (i & 3); };
    if (MT == 1 && S > 1) {  // the plan splits K only with 64-row tiles
        // partial tiles go out with device-coherent stores, waited for before the
        // arrival count, so the last workgroup reads them without a cache flush
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int nt = 0; nt < 2; ++nt) {
                const int n = nt ? nl1 : nl0;
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const int m = row_of(mt, i);
                    if (m < a.M && n < a.N)
                        __hip_atomic_store(a.part + ((size_t)sl * a.M + m) * a.N + n, acc[mt][nt][i], __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_AGENT);
                }
            }
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
        const int tile = blockIdx.y * gridDim.x + blockIdx.x;
        if (tid == 0)
            s_last = __hip_atomic_fetch_add(a.count + tile, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
                     (unsigned)(S - 1);
        __syncthreads();
        if (!s_last) return;
        // sum the S partials in slice order, RJ slices' loads in flight at a time
        constexpr int RJ = 2;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int nt = 0; nt < 2; ++nt)
#pragma unroll
                for (int i = 0; i < 16; ++i) acc[mt][nt][i] = 0.f;
        for (int s0 = 0; s0 < S; s0 += RJ) {
            float pv[RJ][MT][2][16];
#pragma unroll
            for (int j = 0; j < RJ; ++j) {
                const int ss = min(s0 + j, S - 1);
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                    for (int nt = 0; nt < 2; ++nt) {
                        const int n = min(nt ? nl1 : nl0, a.N - 1);
#pragma unroll
                        for (int i = 0; i < 16; ++i)
                            pv[j][mt][nt][i] = __hip_atomic_load(
                                a.part + ((size_t)ss * a.M + min(row_of(mt, i), a.M - 1)) * a.N + n, __ATOMIC_RELAXED,
                                __HIP_MEMORY_SCOPE_AGENT);
                    }
            }
#pragma unroll
            for (int j = 0; j < RJ; ++j)
                if (s0 + j < S) {
#pragma unroll
                    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                        for (int nt = 0; nt < 2; ++nt)
#pragma unroll
                            for (int i = 0; i < 16; ++i) acc[mt][nt][i] += pv[j][mt][nt][i];
                }
        }
        if (tid == 0) __hip_atomic_store(a.count + tile, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }

    constexpr bool F32 = false;
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) {
        const int n = nt ? nl1 : nl0;
        if (n >= a.N) continue;
        float rs = 1.f;
        if constexpr (WT == FTTS_W8A16) rs = bf16_to_f32(a.scale[n]);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int m = row_of(mt, i);
                if (m < a.M)
                    gemm_epilogue<F32, EPI>(a, m, n, acc[mt][nt][i] * rs,
                                            EPI == EPI_QKV ? s_rows[EPI == EPI_QKV ? m - m0 : 0] : RowSlot{-1, 0});
            }
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
            if (m < a.M && n < a.N)
                gemm_epilogue<true, EPI>(a, m, n, acc[i][j], EPI == EPI_QKV ? row_slot(a, m) : RowSlot{-1, 0});
        }
}

template <int WT, int MT>
static hipError_t mfma_by_epi(int epi, const GemmArgs& a, dim3 g, hipStream_t st) {
    switch (epi) {
        case EPI_STORE: hipLaunchKernelGGL((gemm_mfma_kernel<WT, EPI_STORE, MT>), g, dim3(256), 0, st, a); break;
        case EPI_QKV: hipLaunchKernelGGL((gemm_mfma_kernel<WT, EPI_QKV, MT>), g, dim3(256), 0, st, a); break;
        case EPI_GELU: hipLaunchKernelGGL((gemm_mfma_kernel<WT, EPI_GELU, MT>), g, dim3(256), 0, st, a); break;
        case EPI_RESID: hipLaunchKernelGGL((gemm_mfma_kernel<WT, EPI_RESID, MT>), g, dim3(256), 0, st, a); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

// Tile shape and K split of a 16-bit-mode prefill GEMM: 128-row tiles when
// there are enough of them, else 64-row tiles and, if still short of about
// two tiles per CU, K slices of whole 128-column blocks (at least two each).
GemmPlan gemm_plan(int M, int N, int K) {
    GemmPlan p{};
    const int tn = (N + G2N - 1) / G2N;
    p.mt = (M + 127) / 128 * tn >= 512 ? 2 : 1;
    const int bm = 64 * p.mt;
    p.tiles_m = (M + bm - 1) / bm;
    p.tiles_n = tn;
    const int tiles = p.tiles_m * p.tiles_n;
    p.splits = 1;
    if (p.mt == 1 && K % 128 == 0 && tiles > 0 && tiles < 256) {
        const int want = (320 + tiles - 1) / tiles, most = K / 256;
        p.splits = std::max(1, std::min(std::min(want, most), kGemmMaxSplits));
    }
    return p;
}

bool gemm_mfma_supported(int K) { return K % G2K == 0; }

hipError_t launch_gemm(int wdtype, int epi, const GemmArgs& a, hipStream_t st) {
    if (wdtype == FTTS_F32) {
        const dim3 g((a.N + 63) / 64, (a.M + 63) / 64);
        switch (epi) {
            case EPI_STORE: hipLaunchKernelGGL(gemm_f32_kernel<EPI_STORE>, g, dim3(256), 0, st, a); break;
            case EPI_QKV: hipLaunchKernelGGL(gemm_f32_kernel<EPI_QKV>, g, dim3(256), 0, st, a); break;
            case EPI_GELU: hipLaunchKernelGGL(gemm_f32_kernel<EPI_GELU>, g, dim3(256), 0, st, a); break;
            case EPI_RESID: hipLaunchKernelGGL(gemm_f32_kernel<EPI_RESID>, g, dim3(256), 0, st, a); break;
            default: return hipErrorInvalidValue;
        }
        return hipGetLastError();
    }
    if (!gemm_mfma_supported(a.K)) return hipErrorInvalidValue;
    const GemmPlan p = gemm_plan(a.M, a.N, a.K);
    if (p.splits > 1 && (!a.part || !a.count)) return hipErrorInvalidValue;
    const dim3 g(p.tiles_n, p.tiles_m, p.splits);
    switch (wdtype) {
        case FTTS_BF16: return p.mt == 2 ? mfma_by_epi<FTTS_BF16, 2>(epi, a, g, st) : mfma_by_epi<FTTS_BF16, 1>(epi, a, g, st);
        case FTTS_W8A16: return p.mt == 2 ? mfma_by_epi<FTTS_W8A16, 2>(epi, a, g, st) : mfma_by_epi<FTTS_W8A16, 1>(epi, a, g, st);
        case FTTS_W4A16: return p.mt == 2 ? mfma_by_epi<FTTS_W4A16, 2>(epi, a, g, st) : mfma_by_epi<FTTS_W4A16, 1>(epi, a, g, st);
    }
    return hipErrorInvalidValue;
}

}  // namespace ftts
