// Batched decode linears on the matrix cores: out[b][n] = act[b] . W[n]^T + bias
// (+ epilogue) for up to 32 sequences per launch, bf16 / W8A16 / W4A16 weights.
//
// At 8-32 sequences a decode linear still moves every weight byte once per step
// and is bound by HBM, but the per-row dot products of the GEMV family would
// re-stage all activations in every workgroup and run 8-32 FMAs per weight on
// the VALU.  Here each wave computes a 32 (sequences) x 32 (features) tile with
// v_mfma_f32_32x32x16_bf16 over a range of K, reading its weight rows straight
// from HBM into registers (no reuse, so no LDS staging) and the bf16 activations
// (a few tens of KB, L2-resident) alongside.
//
// Work split: a workgroup (4 waves) owns 32 features and one of S slices of K;
// its waves take the slice's 32-column chunks (128 for W4A16, one quantisation
// group) round robin, issue every load of their share at once (S is chosen so
// that a share fits the registers), and add their tiles in LDS.  With S > 1 every workgroup
// stores its partial tile, and the last of the S to arrive (a per-tile counter)
// adds the S partials in slice order -- the same order whatever the arrival
// order, so results are reproducible -- and applies the epilogue; it also
// resets the counter, which is zero between calls.
//
// K order inside a chunk: lane (row, h) feeds the MFMA k-slots h*8..h*8+7 of
// step st from contiguous memory (bf16: k = h*16 + st*8 + i; W4A16: word h*8+st),
// and the activation operand uses the same map, so each lane's loads are
// contiguous and the dot product is unchanged.
#include "ftts_internal.hpp"

namespace ftts {

typedef __bf16 bgemm_bf16x8 __attribute__((ext_vector_type(8)));
typedef float bgemm_f32x16 __attribute__((ext_vector_type(16)));

constexpr int kBgemmRows = 32;  // sequences per launch
constexpr int kBgemmFeat = 32;  // features per workgroup
constexpr int kBgemmMaxSplits = 12;  // K slices per feature tile (K <= 6144 for bf16 / W8A16)

template <int WT> struct BChunk;  // one lane's share of one chunk
template <> struct BChunk<FTTS_BF16> {
    static constexpr int KC = 32, STEPS = 2;
    uint4 w[2];
    uint4 a[2];
};
template <> struct BChunk<FTTS_W8A16> {
    static constexpr int KC = 32, STEPS = 2;
    uint4 w[1];
    uint4 a[2];
};
template <> struct BChunk<FTTS_W4A16> {
    static constexpr int KC = 128, STEPS = 8;
    uint4 w[2];
    uint4 a[8];
    float s, z;
};

// Chunks a wave holds in registers at once (its whole share of a K slice).
template <int WT> struct ChunksPerWave { static constexpr int value = 4; };
template <> struct ChunksPerWave<FTTS_W4A16> { static constexpr int value = 2; };

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    return (uint32_t)f32_to_bf16(lo) | ((uint32_t)f32_to_bf16(hi) << 16);
}

template <int WT>
__device__ __forceinline__ void load_chunk(const BgemmArgs& p, int n, int m, int h, int c, BChunk<WT>& ch) {
    using C = BChunk<WT>;
    const int nn = min(n, p.N - 1);
    const uint16_t* act = reinterpret_cast<const uint16_t*>(p.act);
    // activation row m (zeros past the batch): 8 x 16 bytes for W4A16, 2 otherwise
    const int ka = c * C::KC + h * (C::KC / 2);
#pragma unroll
    for (int i = 0; i < (int)(sizeof(ch.a) / 16); ++i)
        ch.a[i] = m < p.B ? *reinterpret_cast<const uint4*>(act + (size_t)m * p.K + ka + i * 8) : make_uint4(0, 0, 0, 0);
    if constexpr (WT == FTTS_BF16) {
        const uint4* w = reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(p.w) + (size_t)nn * p.K + ka);
        ch.w[0] = ld_stream(w);
        ch.w[1] = ld_stream(w + 1);
    } else if constexpr (WT == FTTS_W8A16) {
        ch.w[0] = ld_stream(reinterpret_cast<const uint4*>(reinterpret_cast<const int8_t*>(p.w) + (size_t)nn * p.K + ka));
    } else {
        const uint4* w = reinterpret_cast<const uint4*>(reinterpret_cast<const uint32_t*>(p.w) + (size_t)nn * (p.K / 8) +
                                                        c * 16 + h * 8);
        ch.w[0] = ld_stream(w);
        ch.w[1] = ld_stream(w + 1);
        ch.s = bf16_to_f32(p.scale[(size_t)nn * (p.K / 128) + c]);
        ch.z = bf16_to_f32(p.zero[(size_t)nn * (p.K / 128) + c]);
    }
}

// The weight operand of MFMA step st (8 bf16; quantised codes expanded exactly).
template <int WT>
__device__ __forceinline__ bgemm_bf16x8 w_operand(const BChunk<WT>& ch, int st) {
    uint4 r;
    if constexpr (WT == FTTS_BF16) {
        r = ch.w[st];
    } else if constexpr (WT == FTTS_W8A16) {
        const uint32_t lo = st == 0 ? ch.w[0].x : ch.w[0].z, hi = st == 0 ? ch.w[0].y : ch.w[0].w;
        auto q = [](uint32_t word, int i) { return (float)(int32_t)((int32_t)(word << (24 - 8 * i)) >> 24); };
        r = make_uint4(pack_bf16x2(q(lo, 0), q(lo, 1)), pack_bf16x2(q(lo, 2), q(lo, 3)), pack_bf16x2(q(hi, 0), q(hi, 1)),
                       pack_bf16x2(q(hi, 2), q(hi, 3)));
    } else {
        const uint4 v = st < 4 ? ch.w[0] : ch.w[1];
        const uint32_t word = (st & 3) == 0 ? v.x : (st & 3) == 1 ? v.y : (st & 3) == 2 ? v.z : v.w;
        auto q = [&](int i) { return (float)((word >> (4 * i)) & 0xFu) - ch.z; };
        r = make_uint4(pack_bf16x2(q(0), q(1)), pack_bf16x2(q(2), q(3)), pack_bf16x2(q(4), q(5)), pack_bf16x2(q(6), q(7)));
    }
    return __builtin_bit_cast(bgemm_bf16x8, r);
}

template <int EPI>
__device__ __forceinline__ void bgemm_epilogue(const BgemmArgs& p, int m, int n, float v) {
    v += bf16_to_f32(reinterpret_cast<const uint16_t*>(p.bias)[n]);
    if constexpr (EPI == EPI_RESID) {
        p.out[(size_t)m * p.out_stride + n] += v;
    } else if constexpr (EPI == EPI_GELU) {
        reinterpret_cast<uint16_t*>(p.out_bf16)[(size_t)m * p.out_stride + n] = f32_to_bf16(gelu_tanh(v));
    } else {
        p.out[(size_t)m * p.out_stride + n] = v;
        if constexpr (EPI == EPI_QKV) {
            const int d = p.kv.d_model;
            if (n >= d && p.kv.active[m]) {
                const int kvsel = n >= 2 * d;
                const int r = n - d - kvsel * d;
                const int slot = p.kv.seq_lens[m];
                const int phys = p.kv.block_table[(size_t)m * p.kv.max_pages + slot / kPage];
                st_act<false>(p.kv.base,
                              kv_offset(p.kv.layer, p.kv.n_pages, phys, kvsel, p.kv.n_head, r / kHeadDim, slot % kPage) +
                                  r % kHeadDim,
                              v);
            }
        }
    }
}

template <int WT, int EPI>
__global__ __launch_bounds__(256) void bgemm_kernel(const BgemmArgs p) {
    using C = BChunk<WT>;
    constexpr int CPW = ChunksPerWave<WT>::value;
    __shared__ float s_red[4][kBgemmRows * kBgemmFeat];
    __shared__ int s_last;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int f = blockIdx.x, s = blockIdx.y, S = gridDim.y;
    const int n0 = f * kBgemmFeat;
    const int fr = lane & 31, h = lane >> 5;
    const int nchunks = p.K / C::KC;
    const int c0 = s * nchunks / S, c1 = (s + 1) * nchunks / S;

    // Every load of this wave goes out first (chunks c0 + wave + 4j; indices past
    // the slice repeat its last chunk and are not used), then the products.
    C ch[CPW];
#pragma unroll
    for (int j = 0; j < CPW; ++j) load_chunk<WT>(p, n0 + fr, fr, h, min(c0 + wave + 4 * j, c1 - 1), ch[j]);
    bgemm_f32x16 acc;
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[i] = 0.f;
#pragma unroll
    for (int j = 0; j < CPW; ++j) {
        if (c0 + wave + 4 * j < c1) {
            bgemm_f32x16 part;
#pragma unroll
            for (int i = 0; i < 16; ++i) part[i] = 0.f;
#pragma unroll
            for (int st = 0; st < C::STEPS; ++st) {
                const bgemm_bf16x8 av = __builtin_bit_cast(bgemm_bf16x8, ch[j].a[st]);
                part = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, w_operand<WT>(ch[j], st), part, 0, 0, 0);
            }
            if constexpr (WT == FTTS_W4A16) {
#pragma unroll
                for (int i = 0; i < 16; ++i) acc[i] = fmaf(ch[j].s, part[i], acc[i]);
            } else {
#pragma unroll
                for (int i = 0; i < 16; ++i) acc[i] += part[i];
            }
        }
    }
    // acc[i] holds (sequence m, feature n0 + fr): m = (i / 4) * 8 + h * 4 + i % 4
#pragma unroll
    for (int i = 0; i < 16; ++i) s_red[wave][((i >> 2) * 8 + h * 4 + (i & 3)) * kBgemmFeat + fr] = acc[i];
    __syncthreads();
    float v[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int e = tid + 256 * i;
        v[i] = (s_red[0][e] + s_red[1][e]) + (s_red[2][e] + s_red[3][e]);
    }
    if (S > 1) {
        // Partials go out with device-coherent stores and are waited for before the
        // arrival count, so the last group reads them (device-coherent loads) without
        // any cache flush.
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int e = tid + 256 * i, m = e / kBgemmFeat, n = n0 + e % kBgemmFeat;
            if (m < p.B && n < p.N)
                __hip_atomic_store(p.part + ((size_t)s * p.B + m) * p.N + n, v[i], __ATOMIC_RELAXED,
                                   __HIP_MEMORY_SCOPE_AGENT);
        }
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
        if (tid == 0)
            s_last = __hip_atomic_fetch_add(p.count + f, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
                     (unsigned)(S - 1);
        __syncthreads();
        if (!s_last) return;
        // all S x 4 loads go out before the first add (indices clamped, extras unused)
        float pv[4][kBgemmMaxSplits];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int e = tid + 256 * i, m = min(e / kBgemmFeat, p.B - 1), n = min(n0 + e % kBgemmFeat, p.N - 1);
#pragma unroll
            for (int k = 0; k < kBgemmMaxSplits; ++k)
                pv[i][k] = __hip_atomic_load(p.part + ((size_t)min(k, S - 1) * p.B + m) * p.N + n, __ATOMIC_RELAXED,
                                             __HIP_MEMORY_SCOPE_AGENT);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            float t = 0.f;
#pragma unroll
            for (int k = 0; k < kBgemmMaxSplits; ++k)
                if (k < S) t += pv[i][k];
            v[i] = t;
        }
        if (tid == 0) __hip_atomic_store(p.count + f, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    float rs = 1.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int e = tid + 256 * i, m = e / kBgemmFeat, n = n0 + e % kBgemmFeat;
        if (m < p.B && n < p.N) {
            if constexpr (WT == FTTS_W8A16) rs = bf16_to_f32(p.scale[n]);
            bgemm_epilogue<EPI>(p, m, n, v[i] * rs);
        }
    }
}

template <int WT>
static hipError_t bgemm_by_epi(int epi, const BgemmArgs& a, dim3 g, hipStream_t st) {
    switch (epi) {
        case EPI_STORE: hipLaunchKernelGGL((bgemm_kernel<WT, EPI_STORE>), g, dim3(256), 0, st, a); break;
        case EPI_QKV: hipLaunchKernelGGL((bgemm_kernel<WT, EPI_QKV>), g, dim3(256), 0, st, a); break;
        case EPI_GELU: hipLaunchKernelGGL((bgemm_kernel<WT, EPI_GELU>), g, dim3(256), 0, st, a); break;
        case EPI_RESID: hipLaunchKernelGGL((bgemm_kernel<WT, EPI_RESID>), g, dim3(256), 0, st, a); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

// K slices per feature tile: enough that each wave's share fits its registers.
int bgemm_splits(int wdtype, int N, int K) {
    (void)N;
    const int kc = wdtype == FTTS_W4A16 ? 128 : 32;
    const int per_group = 4 * (wdtype == FTTS_W4A16 ? ChunksPerWave<FTTS_W4A16>::value : ChunksPerWave<FTTS_BF16>::value);
    const int chunks = K / kc;
    return (chunks + per_group - 1) / per_group;
}

bool bgemm_supported(int wdtype, int K) {
    if (wdtype == FTTS_F32) return false;
    return K % (wdtype == FTTS_W4A16 ? 128 : 32) == 0 && bgemm_splits(wdtype, 0, K) <= kBgemmMaxSplits;
}

hipError_t launch_bgemm(int wdtype, int epi, const BgemmArgs& in, hipStream_t st) {
    // The LM head is never quantised.
    const int wt = epi == EPI_STORE ? FTTS_BF16 : wdtype;
    if (!bgemm_supported(wt, in.K)) return hipErrorInvalidValue;
    const int S = bgemm_splits(wt, in.N, in.K);
    const dim3 g((in.N + kBgemmFeat - 1) / kBgemmFeat, S);
    for (int b0 = 0; b0 < in.B; b0 += kBgemmRows) {
        BgemmArgs a = in;
        a.B = in.B - b0 < kBgemmRows ? in.B - b0 : kBgemmRows;
        a.act = reinterpret_cast<const uint16_t*>(in.act) + (size_t)b0 * in.K;
        if (in.out) a.out = in.out + (size_t)b0 * in.out_stride;
        if (in.out_bf16) a.out_bf16 = reinterpret_cast<uint16_t*>(in.out_bf16) + (size_t)b0 * in.out_stride;
        if (epi == EPI_QKV) {
            a.kv.seq_lens = in.kv.seq_lens + b0;
            a.kv.active = in.kv.active + b0;
            a.kv.block_table = in.kv.block_table + (size_t)b0 * in.kv.max_pages;
        }
        hipError_t e;
        switch (wt) {
            case FTTS_BF16: e = bgemm_by_epi<FTTS_BF16>(epi, a, g, st); break;
            case FTTS_W8A16: e = bgemm_by_epi<FTTS_W8A16>(epi, a, g, st); break;
            case FTTS_W4A16: e = bgemm_by_epi<FTTS_W4A16>(epi, a, g, st); break;
            default: return hipErrorInvalidValue;
        }
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace ftts
