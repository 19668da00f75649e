// Dense contractions of the prefill: C[M][N] = A[M][K] . W[N][K]^T with fused
// epilogues (bias, q/k/v store + paged KV scatter, GELU, residual add).
//
// 16-bit modes: bf16 MFMA (v_mfma_f32_32x32x16_bf16, gfx950).  Large GEMMs with
// bf16 weights take gemm_big_kernel (256 x 256 tiles, below).  Otherwise a 256-thread
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

// Store of one biased output element for the non-residual epilogues (rs: the
// row's KV destination, EPI_QKV only).
template <bool F32, int EPI>
__device__ __forceinline__ void gemm_store(const GemmArgs& a, int m, int n, float v, RowSlot rs) {
    if constexpr (EPI == EPI_GELU) {
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

// Epilogue of one output element.
template <bool F32, int EPI>
__device__ __forceinline__ void gemm_epilogue(const GemmArgs& a, int m, int n, float v, RowSlot rs) {
    v += ld_act<F32>(a.bias, n);
    if constexpr (EPI == EPI_RESID) {
        float* o = reinterpret_cast<float*>(a.out) + (size_t)m * a.N + n;
        *o += v;
    } else {
        gemm_store<F32, EPI>(a, m, n, v, rs);
    }
}

// The tanh GELU written as u * sigmoid(2 c (u + 0.044715 u^3)) -- the same
// function, since 0.5 (1 + tanh z) = 1 / (1 + exp(-2 z)) -- on one exponential
// and one hardware reciprocal (the result is rounded to bf16).
__device__ __forceinline__ float gelu_one_exp(float u) {
    const float c2 = 2.0f * 0.7978845608028654f;
    return u * __builtin_amdgcn_rcpf(1.0f + __expf(-c2 * (u + 0.044715f * u * u * u)));
}

// Raw staging of one thread's share of a 128 x 64 W tile: 4 chunks of 8 k.
template <int WT> struct WStage;
template <> struct WStage<FTTS_BF16> { uint4 v[4]; };
template <> struct WStage<FTTS_W8A16> { uint2 v[4]; };
template <> struct WStage<FTTS_W4A16> { uint32_t v[4]; uint16_t z[4]; };

constexpr int G2N = 128, G2K = 64, G2LD = G2K + 8;  // tile columns, K step, LDS row pitch (bf16)
constexpr int kGemmMaxSplits = 8;
constexpr int kGemmEpiBytes = 8192;  // a wave's epilogue staging: 32 rows x 64 columns of fp32

// Device-coherent 8-byte store / load (two fp32) for the split-K partials.
__device__ __forceinline__ void st_dev2(float* p, float x, float y) {
    const uint64_t v = (uint64_t)__float_as_uint(x) | ((uint64_t)__float_as_uint(y) << 32);
    __hip_atomic_store(reinterpret_cast<uint64_t*>(p), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ uint64_t ld_dev2(const float* p) {
    return __hip_atomic_load(reinterpret_cast<const uint64_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

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
    constexpr int SA = BM * G2LD, SB = G2N * G2LD;          // bf16 elements of one A / W buffer
    // both operand buffers in one array: the epilogue reuses it, 8 KB per wave
    __shared__ __attribute__((aligned(16))) uint16_t s_ab[2 * SA + 2 * SB];
    static_assert((2 * SA + 2 * SB) * 2 >= 4 * kGemmEpiBytes, "epilogue staging fits the operand buffers");
    auto sA = [&](int b) { return s_ab + b * SA; };
    auto sB = [&](int b) { return s_ab + 2 * SA + b * SB; };
    __shared__ int s_last;
    __shared__ RowSlot s_rows[EPI == EPI_QKV ? BM : 1];  // KV destination of each row of the tile
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    // Workgroups are dealt to the 8 XCDs round-robin by linear id: give each XCD a
    // contiguous run of tiles in row-major order, so the column tiles of one row
    // block share an XCD's L2 and the activation block is fetched there once
    // (column-major with at most 8 row blocks, where the weights are the bulk).
    // Every K slice of a tile maps alike, so the split-K pairing is unchanged.
    int m0, n0;
    {
        const int T = gridDim.x * gridDim.y, b = blockIdx.y * gridDim.x + blockIdx.x;
        const int x = b & 7, l = b >> 3, q = T >> 3, r = T & 7;
        const int t = (x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q) + l;
        if (gridDim.y <= 8) {  // few row blocks: a weight tile's row blocks share an XCD instead
            m0 = (t % gridDim.y) * BM;
            n0 = (t / gridDim.y) * G2N;
        } else {
            m0 = (t / gridDim.x) * BM;
            n0 = (t % gridDim.x) * G2N;
        }
    }
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
    store_stage<WT, AV>(ra, rw, sA(0), sB(0));
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
                av[mt] = *reinterpret_cast<const bf16x8_t*>(&sA(buf)[(wm * 32 * MT + mt * 32 + fr) * G2LD + kk + fh * 8]);
#pragma unroll
            for (int nt = 0; nt < 2; ++nt)
                bv[nt] = *reinterpret_cast<const bf16x8_t*>(&sB(buf)[(wn * 64 + nt * 32 + fr) * G2LD + kk + fh * 8]);
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
        if (kt + 1 < kb1) store_stage<WT, AV>(ra, rw, sA(buf ^ 1), sB(buf ^ 1));  // last read before the previous barrier
        __syncthreads();
    }

    if (MT == 1 && S > 1) {  // the plan splits K only with 64-row tiles
        // The accumulators go out in fragment order -- pair e of thread t at
        // (e * 256 + t) * 2, so each store instruction covers 512 contiguous bytes
        // and the thread in the same position of the tile's last workgroup reads
        // them back -- with device-coherent 8-byte stores waited for before the
        // arrival count, so the last workgroup reads them without a cache flush.
        constexpr int NV = MT * 2 * 16;
        const int T = gridDim.x * gridDim.y, tile = blockIdx.y * gridDim.x + blockIdx.x;
        auto slot = [&](int ss) { return a.part + ((size_t)ss * T + tile) * 256 * NV + 2 * tid; };
        {
            float* pp = slot(sl);
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int nt = 0; nt < 2; ++nt)
#pragma unroll
                    for (int i = 0; i < 16; i += 2)
                        st_dev2(pp + ((mt * 2 + nt) * 8 + i / 2) * 512, acc[mt][nt][i], acc[mt][nt][i + 1]);
        }
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
        if (tid == 0)
            s_last = __hip_atomic_fetch_add(a.count + tile, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
                     (unsigned)(S - 1);
        __syncthreads();
        if (!s_last) return;
        // sum the S partials in slice order, RJ slices' loads in flight at a time
        constexpr int RJ = 4;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int nt = 0; nt < 2; ++nt)
#pragma unroll
                for (int i = 0; i < 16; ++i) acc[mt][nt][i] = 0.f;
        for (int s0 = 0; s0 < S; s0 += RJ) {
            uint64_t pv[RJ][NV / 2];
#pragma unroll
            for (int j = 0; j < RJ; ++j) {
                const float* pp = slot(min(s0 + j, S - 1));
#pragma unroll
                for (int e = 0; e < NV / 2; ++e) pv[j][e] = ld_dev2(pp + e * 512);
            }
#pragma unroll
            for (int j = 0; j < RJ; ++j)
                if (s0 + j < S) {
#pragma unroll
                    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                        for (int nt = 0; nt < 2; ++nt)
#pragma unroll
                            for (int i = 0; i < 16; i += 2) {
                                const uint64_t v = pv[j][((mt * 2 + nt) * 16 + i) / 2];
                                acc[mt][nt][i] += __uint_as_float((uint32_t)v);
                                acc[mt][nt][i + 1] += __uint_as_float((uint32_t)(v >> 32));
                            }
                }
        }
        if (tid == 0) __hip_atomic_store(a.count + tile, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }

    {
        // Epilogue through LDS (N is a multiple of 8: the launcher checks it) (the operand buffers are free: every wave passed the
        // loop's last barrier): each wave writes its (32 MT) x 64 sub-tile in
        // row-major order and reads it back as 16-byte row pieces for coalesced
        // stores -- output rows and, for q/k/v, the new keys and values into their
        // KV pages (64 columns are one head); for the residual update x += y, 32
        // rows at a time, all old values loaded before the stores.  Pieces are
        // XOR-swizzled by row so that the column-wise writes of the MFMA layout do
        // not collide in banks.
        char* eb = reinterpret_cast<char*>(s_ab) + wave * kGemmEpiBytes;
        const int rw0 = m0 + wm * 32 * MT, cw0 = n0 + wn * 64;
        float bias[2], rs[2] = {1.f, 1.f};
#pragma unroll
        for (int nt = 0; nt < 2; ++nt) {
            const int n = min(cw0 + nt * 32 + fr, a.N - 1);
            bias[nt] = ld_act<false>(a.bias, n);
            if constexpr (WT == FTTS_W8A16) rs[nt] = bf16_to_f32(a.scale[n]);
        }
        if constexpr (EPI != EPI_RESID) {
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int nt = 0; nt < 2; ++nt)
#pragma unroll
                    for (int i = 0; i < 16; ++i) {
                        float y = acc[mt][nt][i] * rs[nt] + bias[nt];
                        if constexpr (EPI == EPI_GELU) y = gelu_one_exp(y);
                        const int rl = mt * 32 + (i >> 2) * 8 + fh * 4 + (i & 3), cl = nt * 32 + fr;
                        *reinterpret_cast<uint16_t*>(eb + rl * 128 + (((cl >> 3) ^ (rl & 7)) << 4) + (cl & 7) * 2) =
                            f32_to_bf16(y);
                    }
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
            uint16_t* out = reinterpret_cast<uint16_t*>(a.out);
#pragma unroll
            for (int it = 0; it < 4 * MT; ++it) {
                const int j = lane + 64 * it, rl = j >> 3, q = j & 7;
                const uint4 v = *reinterpret_cast<const uint4*>(eb + rl * 128 + ((q ^ (rl & 7)) << 4));
                const int m = rw0 + rl, n = cw0 + q * 8;
                if (m < a.M && n < a.N) {
                    *reinterpret_cast<uint4*>(out + (size_t)m * a.N + n) = v;
                    if constexpr (EPI == EPI_QKV) {
                        const int d = a.kv.d_model;
                        const RowSlot r_s = s_rows[m - m0];
                        if (n >= d && r_s.phys >= 0) {
                            const int kvsel = n >= 2 * d, r = n - d - kvsel * d;
                            const size_t off = kv_offset(a.kv.layer, a.kv.n_pages, r_s.phys, kvsel, a.kv.n_head,
                                                         r / kHeadDim, r_s.slot) + (r % kHeadDim);
                            *reinterpret_cast<uint4*>(reinterpret_cast<uint16_t*>(a.kv.base) + off) = v;
                        }
                    }
                }
            }
        } else {
            float* x = reinterpret_cast<float*>(a.out);
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
                for (int nt = 0; nt < 2; ++nt)
#pragma unroll
                    for (int i = 0; i < 16; ++i) {
                        const int rl = (i >> 2) * 8 + fh * 4 + (i & 3), cl = nt * 32 + fr;
                        const int sl4 = (cl >> 2) ^ (((rl >> 2) & 1) << 3);
                        *reinterpret_cast<float*>(eb + rl * 256 + sl4 * 16 + (cl & 3) * 4) =
                            acc[mt][nt][i] * rs[nt] + bias[nt];
                    }
                asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
                float4 y[8], old[8];
#pragma unroll
                for (int it = 0; it < 8; ++it) {
                    const int j = lane + 64 * it, rl = j >> 4, q = j & 15;
                    y[it] = *reinterpret_cast<const float4*>(eb + rl * 256 + ((q ^ (((rl >> 2) & 1) << 3)) << 4));
                    const int m = min(rw0 + mt * 32 + rl, a.M - 1), n = min(cw0 + q * 4, a.N - 4);
                    old[it] = *reinterpret_cast<const float4*>(x + (size_t)m * a.N + n);
                }
#pragma unroll
                for (int it = 0; it < 8; ++it) {
                    const int j = lane + 64 * it, rl = j >> 4, q = j & 15;
                    const int m = rw0 + mt * 32 + rl, n = cw0 + q * 4;
                    if (m < a.M && n < a.N)
                        *reinterpret_cast<float4*>(x + (size_t)m * a.N + n) = make_float4(
                            old[it].x + y[it].x, old[it].y + y[it].y, old[it].z + y[it].z, old[it].w + y[it].w);
                }
                asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // this pass's reads done before the next writes
            }
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

// Large 16-bit prefill GEMMs (bf16 weights, enough 256 x 256 tiles to fill the
// chip): a 512-thread block computes a 256 x 256 tile as a 2 x 4 grid of waves,
// each wave 4 x 2 accumulators of 32x32, over 32-column K steps.  Both operand
// tiles come in through 1 KB direct-to-LDS loads (16 rows of 64 bytes per
// instruction, 16-byte pieces XOR-swizzled by row / 4 so that an MFMA operand
// read touches every bank once) into a ring of four stages, three steps ahead of
// the products: a step waits for its own stage's loads (the two later steps'
// stay in flight), passes one barrier, reads the operands of its first 16
// columns, issues the reads of the second 16 and the refill of the stage the
// previous step used, and runs the first 8 matrix instructions while those reads
// return, then the other 8.  The
// stages are separate LDS objects and the loop is unrolled over them, so the
// compiler sees that a read of one stage does not wait for loads into another.
// Twice the tile edge of the 128 x 128 kernel halves the operand bytes per
// product.  Tiles are ordered for the per-XCD L2s: workgroups are spread over the
// 8 XCDs round-robin, so block b takes tile t from the contiguous run of tiles
// given to XCD b % 8, and consecutive tiles form groups of 4 row blocks that
// walk the columns -- the 32 tiles an XCD runs at once share 4 row blocks of the
// activations and about 8 column blocks of the weights.  (The mapping is a
// bijection whatever the placement; only the cache reuse depends on it.)
constexpr int GB = 256, GBKB = 32, GSTAGE = GB * GBKB * 2;  // tile edge, K step, bytes per operand stage
__shared__ __attribute__((aligned(1024))) char g_sa0[GSTAGE], g_sa1[GSTAGE], g_sa2[GSTAGE], g_sa3[GSTAGE];
__shared__ __attribute__((aligned(1024))) char g_sb0[GSTAGE], g_sb1[GSTAGE], g_sb2[GSTAGE], g_sb3[GSTAGE];
template <int S> __device__ __forceinline__ char* big_a() {
    return S == 0 ? g_sa0 : S == 1 ? g_sa1 : S == 2 ? g_sa2 : g_sa3;
}
template <int S> __device__ __forceinline__ char* big_b() {
    return S == 0 ? g_sb0 : S == 1 ? g_sb1 : S == 2 ? g_sb2 : g_sb3;
}

typedef __attribute__((address_space(3))) char gemm_lds_char;
// Wave w's 16 KB epilogue buffer: one of the eight operand stages.
__device__ __forceinline__ char* big_epi_buf(int w) {
    switch (w) {
        case 0: return g_sa0; case 1: return g_sa1; case 2: return g_sa2; case 3: return g_sa3;
        case 4: return g_sb0; case 5: return g_sb1; case 6: return g_sb2; default: return g_sb3;
    }
}

// The GELU of the large-tile epilogue (gelu_one_exp, above).
__device__ __forceinline__ float gelu_sigmoid_form(float u) { return gelu_one_exp(u); }

// Two fp32 values to packed bf16 (round to nearest even) in one gfx950 instruction.
__device__ __forceinline__ uint32_t bf16x2_rne(float lo, float hi) {
    typedef __bf16 bf16x2_v __attribute__((ext_vector_type(2)));
    typedef float f32x2_v __attribute__((ext_vector_type(2)));
    const f32x2_v v = {lo, hi};
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_v));
}
__device__ __forceinline__ void gemm_dma16(const void* src, char* dst) {
    __builtin_amdgcn_global_load_lds(src, (gemm_lds_char*)dst, 16, 0, 0);
}

// This wave's share (2 of 16 instructions) of one 256 x 32 bf16 operand tile:
// rows r0 .. r0 + 255 (clamped to rows - 1), columns k0 .. k0 + 31.
__device__ __forceinline__ int big_slot(int row, int piece) { return piece ^ ((row >> 2) & 3); }
__device__ __forceinline__ void big_stage(const uint16_t* X, int rows, int K, int r0, int k0, char* dst) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
        const int o = wave * 2 + i, r = o * 16 + (lane >> 2), pc = big_slot(r, lane & 3);
        gemm_dma16(X + (size_t)min(r0 + r, rows - 1) * K + k0 + pc * 8, dst + o * 1024);
    }
}

// Operand reads are issued as ds_read_b128 in inline assembly and waited for by
// big_wait: the compiler cannot tell which stage a direct-to-LDS load writes, and
// would otherwise wait for every load in flight before the first read of a step.
__device__ __forceinline__ bf16x8_t big_read(const char* tile, int row, int piece) {
    const uint32_t addr = (uint32_t)(uintptr_t)(gemm_lds_char*)(tile + row * 64 + (big_slot(row, piece) << 4));
    bf16x8_t r;
    asm volatile("ds_read_b128 %0, %1" : "=v"(r) : "v"(addr) : "memory");
    return r;
}

struct BigCtx {
    const uint16_t *A, *W;
    int M, N, K, m0, n0, wm, wn, fr, fh, nk;
};

// Operand reads of one K half (16 columns) of a stage, and the wait for them.
template <int S>
__device__ __forceinline__ void big_read_half(const BigCtx& c, int half, bf16x8_t (&av)[4], bf16x8_t (&bv)[2]) {
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) av[mt] = big_read(big_a<S>(), c.wm * 128 + mt * 32 + c.fr, 2 * half + c.fh);
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) bv[nt] = big_read(big_b<S>(), c.wn * 64 + nt * 32 + c.fr, 2 * half + c.fh);
}
__device__ __forceinline__ void big_wait_half(bf16x8_t (&av)[4], bf16x8_t (&bv)[2]) {
    asm volatile("s_waitcnt lgkmcnt(0)"
                 : "+v"(av[0]), "+v"(av[1]), "+v"(av[2]), "+v"(av[3]), "+v"(bv[0]), "+v"(bv[1])
                 :
                 : "memory");
}
__device__ __forceinline__ void big_mfma_half(f32x16_t (&acc)[4][2], const bf16x8_t (&av)[4], const bf16x8_t (&bv)[2]) {
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int nt = 0; nt < 2; ++nt)
            acc[mt][nt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[mt], bv[nt], acc[mt][nt], 0, 0, 0);
}

// Stage s's loads have landed in every wave: wait until only the later steps'
// loads (4 per step, steps up to kt + 3 issued) are in flight, then a bare
// barrier.  A fenced __syncthreads would also wait for those later loads.
__device__ __forceinline__ void big_stage_ready(const BigCtx& c, int s) {
    __builtin_amdgcn_sched_barrier(0);
    const int later = (s + 1 < c.nk) + (s + 2 < c.nk);  // steps after s whose loads are out
    if (later == 2) asm volatile("s_waitcnt vmcnt(8)" ::: "memory");
    else if (later == 1) asm volatile("s_waitcnt vmcnt(4)" ::: "memory");
    else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
}

// One K step on stage S, software-pipelined by halves: on entry (a0, b0) hold
// step kt's first half, read and waited for.  The second half's reads go out
// with the refill of the stage step kt - 1 used (loads for step kt + 3), then the
// first half's products; after the next stage is ready its first half is read
// into (a0, b0) while the second half's products run.
template <int S>
__device__ __forceinline__ void big_step(const BigCtx& c, int kt, f32x16_t (&acc)[4][2], bf16x8_t (&a0)[4],
                                         bf16x8_t (&b0)[2]) {
    bf16x8_t a1[4], b1[2];
    big_read_half<S>(c, 1, a1, b1);
    if (kt + 3 < c.nk) {  // stage (S + 3) % 4: every wave finished reading it before the last barrier
        big_stage(c.A, c.M, c.K, c.m0, (kt + 3) * GBKB, big_a<(S + 3) % 4>());
        big_stage(c.W, c.N, c.K, c.n0, (kt + 3) * GBKB, big_b<(S + 3) % 4>());
    }
    __builtin_amdgcn_sched_barrier(0);
    big_mfma_half(acc, a0, b0);
    __builtin_amdgcn_sched_barrier(0);
    big_wait_half(a1, b1);
    if (kt + 1 < c.nk) {
        // (the step's reads of stage S are complete, so this barrier also frees it)
        big_stage_ready(c, kt + 1);
        big_read_half<(S + 1) % 4>(c, 0, a0, b0);
    }
    __builtin_amdgcn_sched_barrier(0);
    big_mfma_half(acc, a1, b1);
    __builtin_amdgcn_sched_barrier(0);
    if (kt + 1 < c.nk) big_wait_half(a0, b0);
}

template <int EPI>
__global__ __launch_bounds__(512) void gemm_big_kernel(const GemmArgs a) {
    __shared__ RowSlot s_rows[EPI == EPI_QKV ? GB : 1];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    BigCtx c;
    c.A = reinterpret_cast<const uint16_t*>(a.a);
    c.W = reinterpret_cast<const uint16_t*>(a.w);
    c.M = a.M, c.N = a.N, c.K = a.K;
    {
        const int tn = (a.N + GB - 1) / GB, tm = (a.M + GB - 1) / GB, T = tm * tn;
        const int b = blockIdx.x, x = b & 7, l = b >> 3, q = T >> 3, r = T & 7;
        const int t = (x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q) + l;
        constexpr int GM = 8;  // row blocks per group
        const int g = t / (GM * tn), gm = min(GM, tm - g * GM), w = t - g * GM * tn;
        c.m0 = (g * GM + w % gm) * GB;
        c.n0 = (w / gm) * GB;
    }
    c.wm = wave >> 2, c.wn = wave & 3;  // rows wm*128 .., columns wn*64 ..
    c.fr = lane & 31, c.fh = lane >> 5;
    c.nk = a.K / GBKB;
    const int m0 = c.m0, n0 = c.n0, wm = c.wm, wn = c.wn, fr = c.fr, fh = c.fh;
    if constexpr (EPI == EPI_QKV) {
        if (tid < GB) s_rows[tid] = row_slot(a, min(m0 + tid, a.M - 1));  // read after the first barrier
    }
    f32x16_t acc[4][2];
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int nt = 0; nt < 2; ++nt)
#pragma unroll
            for (int i = 0; i < 16; ++i) acc[mt][nt][i] = 0.f;
    // prologue: steps 0, 1, 2 into stages 0, 1, 2
    big_stage(c.A, c.M, c.K, m0, 0, g_sa0);
    big_stage(c.W, c.N, c.K, n0, 0, g_sb0);
    if (c.nk > 1) {
        big_stage(c.A, c.M, c.K, m0, GBKB, g_sa1);
        big_stage(c.W, c.N, c.K, n0, GBKB, g_sb1);
    }
    if (c.nk > 2) {
        big_stage(c.A, c.M, c.K, m0, 2 * GBKB, g_sa2);
        big_stage(c.W, c.N, c.K, n0, 2 * GBKB, g_sb2);
    }
    bf16x8_t a0[4], b0[2];
    big_stage_ready(c, 0);
    big_read_half<0>(c, 0, a0, b0);
    big_wait_half(a0, b0);
    for (int kt = 0; kt < c.nk; kt += 4) {
        big_step<0>(c, kt, acc, a0, b0);
        if (kt + 1 < c.nk) big_step<1>(c, kt + 1, acc, a0, b0);
        if (kt + 2 < c.nk) big_step<2>(c, kt + 2, acc, a0, b0);
        if (kt + 3 < c.nk) big_step<3>(c, kt + 3, acc, a0, b0);
    }
    __syncthreads();  // s_rows written before the loop is read below
    // Epilogue through LDS (the operand stages are free now: one 16 KB stage per
    // wave): each wave writes its biased (and activated) 128 x 64 sub-tile in
    // row-major order, then reads it back as 16-byte row pieces for coalesced
    // stores -- the output rows, the new keys and values into their KV pages, or
    // for the residual update x += y in two 64-row halves, all old values of a
    // half loaded before its stores.  Pieces are XOR-swizzled by row so that the
    // column-wise writes of the MFMA layout do not collide in banks.
    char* eb = big_epi_buf(wave);
    float bias[2];
#pragma unroll
    for (int nt = 0; nt < 2; ++nt) bias[nt] = ld_act<false>(a.bias, min(n0 + wn * 64 + nt * 32 + fr, a.N - 1));
    const int rw0 = m0 + wm * 128, cw0 = n0 + wn * 64;  // this wave's first row and column
    if constexpr (EPI != EPI_RESID) {
#pragma unroll
        for (int mt = 0; mt < 4; ++mt)
#pragma unroll
            for (int nt = 0; nt < 2; ++nt)
#pragma unroll
                for (int i = 0; i < 16; i += 2) {
                    float2 y = make_float2(acc[mt][nt][i] + bias[nt], acc[mt][nt][i + 1] + bias[nt]);
                    if constexpr (EPI == EPI_GELU) y = make_float2(gelu_sigmoid_form(y.x), gelu_sigmoid_form(y.y));
                    const uint32_t pk = bf16x2_rne(y.x, y.y);  // rows i and i + 1 of the same column
#pragma unroll
                    for (int e = 0; e < 2; ++e) {
                        const int rl = mt * 32 + ((i + e) >> 2) * 8 + fh * 4 + ((i + e) & 3), cl = nt * 32 + fr;
                        *reinterpret_cast<uint16_t*>(eb + rl * 128 + (((cl >> 3) ^ (rl & 7)) << 4) + (cl & 7) * 2) =
                            (uint16_t)(pk >> (16 * e));
                    }
                }
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        uint16_t* out = reinterpret_cast<uint16_t*>(a.out);
#pragma unroll
        for (int it = 0; it < 16; ++it) {
            const int j = lane + 64 * it, rl = j >> 3, q = j & 7;
            const uint4 v = *reinterpret_cast<const uint4*>(eb + rl * 128 + ((q ^ (rl & 7)) << 4));
            const int m = rw0 + rl, n = cw0 + q * 8;
            if (m < a.M && n < a.N) {
                *reinterpret_cast<uint4*>(out + (size_t)m * a.N + n) = v;
                if constexpr (EPI == EPI_QKV) {
                    const int d = a.kv.d_model;
                    const RowSlot rs = s_rows[wm * 128 + rl];
                    if (n >= d && rs.phys >= 0) {
                        const int kvsel = n >= 2 * d, r = n - d - kvsel * d;
                        const size_t off = kv_offset(a.kv.layer, a.kv.n_pages, rs.phys, kvsel, a.kv.n_head,
                                                     r / kHeadDim, rs.slot) + (r % kHeadDim);
                        *reinterpret_cast<uint4*>(reinterpret_cast<uint16_t*>(a.kv.base) + off) = v;
                    }
                }
            }
        }
    } else {
        float* x = reinterpret_cast<float*>(a.out);
#pragma unroll
        for (int half = 0; half < 2; ++half) {
#pragma unroll
            for (int mh = 0; mh < 2; ++mh)
#pragma unroll
                for (int nt = 0; nt < 2; ++nt)
#pragma unroll
                    for (int i = 0; i < 16; ++i) {
                        const int rl = mh * 32 + (i >> 2) * 8 + fh * 4 + (i & 3), cl = nt * 32 + fr;
                        const int slot = (cl >> 2) ^ (((rl >> 2) & 1) << 3);
                        *reinterpret_cast<float*>(eb + rl * 256 + slot * 16 + (cl & 3) * 4) =
                            acc[half * 2 + mh][nt][i] + bias[nt];
                    }
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
            float4 y[16], old[16];
#pragma unroll
            for (int it = 0; it < 16; ++it) {
                const int j = lane + 64 * it, rl = j >> 4, q = j & 15;
                y[it] = *reinterpret_cast<const float4*>(eb + rl * 256 + ((q ^ (((rl >> 2) & 1) << 3)) << 4));
                const int m = min(rw0 + half * 64 + rl, a.M - 1), n = min(cw0 + q * 4, a.N - 4);
                old[it] = *reinterpret_cast<const float4*>(x + (size_t)m * a.N + n);
            }
#pragma unroll
            for (int it = 0; it < 16; ++it) {
                const int j = lane + 64 * it, rl = j >> 4, q = j & 15;
                const int m = rw0 + half * 64 + rl, n = cw0 + q * 4;
                if (m < a.M && n < a.N)
                    *reinterpret_cast<float4*>(x + (size_t)m * a.N + n) =
                        make_float4(old[it].x + y[it].x, old[it].y + y[it].y, old[it].z + y[it].z, old[it].w + y[it].w);
            }
            asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // this half's reads done before the next half's writes
        }
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
    p.mt = (M + 127) / 128 * tn >= 256 ? 2 : 1;
    const int bm = 64 * p.mt;
    p.tiles_m = (M + bm - 1) / bm;
    p.tiles_n = tn;
    const int tiles = p.tiles_m * p.tiles_n;
    p.splits = 1;
    // split K only where each slice keeps enough K steps: below K = 1024 the
    // partial-tile round trip costs more than the shorter K loop saves
    if (p.mt == 1 && K % 128 == 0 && K >= 1024 && tiles > 0 && tiles < 256) {
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
    if (!gemm_mfma_supported(a.K) || a.N % 8) return hipErrorInvalidValue;  // 16-byte epilogue stores
    // bf16 weights with at least 128 tiles of 256 x 256: the large-tile kernel
    const long big_tiles = (long)((a.M + GB - 1) / GB) * ((a.N + GB - 1) / GB);
    if (wdtype == FTTS_BF16 && big_tiles >= 128 && a.N % 8 == 0) {
        const dim3 g((unsigned)big_tiles);
        switch (epi) {
            case EPI_STORE: hipLaunchKernelGGL(gemm_big_kernel<EPI_STORE>, g, dim3(512), 0, st, a); break;
            case EPI_QKV: hipLaunchKernelGGL(gemm_big_kernel<EPI_QKV>, g, dim3(512), 0, st, a); break;
            case EPI_GELU: hipLaunchKernelGGL(gemm_big_kernel<EPI_GELU>, g, dim3(512), 0, st, a); break;
            case EPI_RESID: hipLaunchKernelGGL(gemm_big_kernel<EPI_RESID>, g, dim3(512), 0, st, a); break;
            default: return hipErrorInvalidValue;
        }
        return hipGetLastError();
    }
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
