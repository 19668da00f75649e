// Batched decode linears on the matrix cores: out[b][n] = act[b] . W[n]^T + bias
// (+ epilogue) for up to 32 sequences per launch, bf16 / W8A16 / W4A16 weights.
//
// At 8-32 sequences a decode linear still moves every weight byte once per step
// and is bound by HBM, but the per-row dot products of the GEMV family would
// re-stage all activations in every workgroup and run 8-32 FMAs per weight on
// the VALU.  Here each wave computes a 32 (sequences) x 32 (features) tile with
// v_mfma_f32_32x32x16_bf16 over a range of K: its weight rows and its input rows
// (bf16 activations, or the fp32 residual stream when a LayerNorm is fused) come
// in through coalesced direct-to-LDS loads (whole row runs per instruction; an
// operand read in MFMA layout touches 32 rows, which as a global load would cost
// the address units far more than the bytes) and are read back in MFMA layout.
//
// Work split: a workgroup (4 waves) owns 32 features (or 64, two MFMA tiles per
// wave, when the 32-feature grid of a LayerNorm-fused linear would not be
// resident at once) and one of S slices of K; each wave takes a run of
// consecutive 32-column chunks (128 for W4A16, one quantisation group) of the
// slice, issues every load of its share at once (S is chosen so that a share
// fits), and the waves add their tiles in LDS.  With S > 1 every workgroup
// stores its partial tile, and the last of the S to arrive (a per-tile counter)
// adds the S partials in slice order -- the same order whatever the arrival
// order, so results are reproducible -- and applies the epilogue; it also
// resets the counter, which is zero between calls.
//
// K order inside a chunk: lane (row, h) feeds the MFMA k-slots h*8..h*8+7 of
// step st from contiguous columns (bf16: k = h*16 + st*8 + i; W4A16: word
// h*8+st), and the input operand uses the same map, so the dot product is
// unchanged.
#include "ftts_internal.hpp"

namespace ftts {

typedef __bf16 bgemm_bf16x8 __attribute__((ext_vector_type(8)));
typedef float bgemm_f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bgemm_bf16x2 __attribute__((ext_vector_type(2)));

constexpr int kBgemmRows = 32;  // sequences per launch
constexpr int kBgemmFeat = 32;  // features per MFMA tile (a workgroup owns FT tiles)
constexpr int kBgemmMaxSplits = 12;  // K slices per feature tile (K <= 6144 for bf16 / W8A16)

template <int WT> struct BChunk;  // one lane's share of one chunk
template <> struct BChunk<FTTS_BF16> {
    static constexpr int KC = 32, STEPS = 2, CB = 64;  // CB: bytes of one weight row per chunk
    uint4 w[2];
    uint4 a[2];
};
template <> struct BChunk<FTTS_W8A16> {
    static constexpr int KC = 32, STEPS = 2, CB = 32;
    uint4 w[1];
    uint4 a[2];
};
template <> struct BChunk<FTTS_W4A16> {
    static constexpr int KC = 128, STEPS = 8, CB = 64;
    uint4 w[2];
    uint4 a[8];
    float s, z;
};

// Chunks per wave (its whole share of a K slice).  A LayerNorm input is staged as
// fp32 rows in LDS (32 rows x 64 columns per wave, 128 for W4A16), which keeps
// three workgroups per CU.
constexpr int kBgemmWaves = 4, kBgemmThreads = kBgemmWaves * 64;
template <int WT, bool LN> struct ChunksPerWave { static constexpr int value = LN ? 2 : 4; };
template <> struct ChunksPerWave<FTTS_W4A16, false> { static constexpr int value = 2; };
template <> struct ChunksPerWave<FTTS_W4A16, true> { static constexpr int value = 1; };

// The LayerNorm input: 256 threads = 8 tile groups x 32 rows merge the tile
// statistics; a slice's gains and biases sit in LDS.
constexpr int kLnGroups = kBgemmThreads / kBgemmRows;
constexpr int kLnMaxTP = 8;                                  // tiles per group: K <= 2048
constexpr int kLnMaxK = kLnGroups * kLnMaxTP * kStatTile;


__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {  // one packed conversion
    const bgemm_bf16x2 v = {(__bf16)lo, (__bf16)hi};
    return __builtin_bit_cast(uint32_t, v);
}

template <int WT, bool LN>
__device__ __forceinline__ void load_chunk(const BgemmArgs& p, int n, int m, int h, int c, BChunk<WT>& ch) {
    using C = BChunk<WT>;
    const int nn = min(n, p.N - 1);
    const int ka = c * C::KC + h * (C::KC / 2);
    // Every load is unconditional (rows past the batch read the last row and are
    // zeroed afterwards), so the loads of all chunks stay in flight together.
    const int mr = min(m, p.B - 1);
    (void)mr;
    (void)ka;
    if constexpr (WT == FTTS_W4A16) {
        ch.s = bf16_to_f32(p.scale[(size_t)nn * (p.K / 128) + c]);
        ch.z = bf16_to_f32(p.zero[(size_t)nn * (p.K / 128) + c]);
    }
}

// Weight staging.  A wave's chunks are consecutive, so each of its 32 rows is
// one run of RB = CPW * CB bytes; direct-to-LDS loads bring the runs in with
// 16 lanes (or fewer) per run and several whole runs per 1 KB instruction, and
// the products read their operands from LDS.  The 16-byte pieces of row r are
// stored XOR-swizzled by r (piece p at slot p ^ (r % pieces)) so that the 32
// rows of one operand read fall into different banks.
typedef __attribute__((address_space(3))) char bgemm_lds_char;
__device__ __forceinline__ void lds_dma16(const char* src, char* dst) {
    __builtin_amdgcn_global_load_lds(src, (bgemm_lds_char*)dst, 16, 0, 0);
}
template <int WT, bool LN, int FT> struct WStageShape {
    static constexpr int RB = ChunksPerWave<WT, LN>::value * BChunk<WT>::CB;  // bytes per row
    static constexpr int PIECES = RB / 16, BYTES = FT * kBgemmFeat * RB, OPS = BYTES / 1024;
    static_assert(BYTES % 1024 == 0 && (PIECES & (PIECES - 1)) == 0, "staging shape");
};

template <int WT, bool LN, int FT>
__device__ __forceinline__ void stage_weights(const BgemmArgs& p, int n0, int cw0, int c1, char* dst) {
    using C = BChunk<WT>;
    using SH = WStageShape<WT, LN, FT>;
    constexpr int PPC = C::CB / 16;  // pieces per chunk
    const int lane = threadIdx.x & 63;
    const size_t row_bytes = WT == FTTS_W4A16 ? (size_t)p.K / 2 : WT == FTTS_W8A16 ? (size_t)p.K : (size_t)p.K * 2;
    const char* wb = reinterpret_cast<const char*>(p.w);
#pragma unroll
    for (int i = 0; i < SH::OPS; ++i) {
        const int off = i * 1024 + lane * 16, r = off / SH::RB, q = (off % SH::RB) / 16;
        const int pc = q ^ (r & (SH::PIECES - 1));                // the piece that lands in slot q
        const int c = min(cw0 + pc / PPC, c1 - 1);                 // its chunk (past the slice: a repeat)
        const int n = min(n0 + r, p.N - 1);
        lds_dma16(wb + (size_t)n * row_bytes + (size_t)c * C::CB + (pc % PPC) * 16, dst + i * 1024);
    }
}

// This lane's weight operands of local chunk j (row fr, k half h) from the staged rows.
template <int WT, bool LN, int FT>
__device__ __forceinline__ void read_weights(const char* src, int fr, int h, int j, BChunk<WT>& ch) {
    using SH = WStageShape<WT, LN, FT>;
    constexpr int NW = (int)(sizeof(ch.w) / 16), PPC = BChunk<WT>::CB / 16;
#pragma unroll
    for (int i = 0; i < NW; ++i) {
        const int pc = j * PPC + h * NW + i, q = pc ^ (fr & (SH::PIECES - 1));
        ch.w[i] = *reinterpret_cast<const uint4*>(src + fr * SH::RB + q * 16);
    }
}

// LayerNorm input staging: this wave's 32 fp32 rows over its CPW chunks, RBX bytes
// a row, by the same 1 KB direct-to-LDS loads and the same XOR swizzle of 16-byte
// pieces.  Rows past the batch repeat the last row (their outputs are zeroed).
template <int WT> struct XStageShape {
    static constexpr int RBX = ChunksPerWave<WT, true>::value * BChunk<WT>::KC * 4;
    static constexpr int PIECES = RBX / 16, BYTES = kBgemmRows * RBX, OPS = BYTES / 1024;
    static_assert(BYTES % 1024 == 0 && (PIECES & (PIECES - 1)) == 0, "input staging shape");
};

template <int WT>
__device__ __forceinline__ void stage_x(const BgemmArgs& p, int cw0, int c1, char* dst) {
    using SH = XStageShape<WT>;
    constexpr int KC = BChunk<WT>::KC;
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int i = 0; i < SH::OPS; ++i) {
        const int off = i * 1024 + lane * 16, r = off / SH::RBX, q = (off % SH::RBX) / 16;
        const int pc = q ^ (r & (SH::PIECES - 1));  // the piece that lands in slot q: columns pc*4 .. +3
        const int c = min(cw0 + pc * 4 / KC, c1 - 1);
        const float* src = p.ln_x + (size_t)min(r, p.B - 1) * p.K + (size_t)c * KC + (pc * 4) % KC;
        lds_dma16(reinterpret_cast<const char*>(src), dst + i * 1024);
    }
}

// A 16-bit input is staged the same way: this wave's 32 bf16 rows over its CPW
// chunks, RBA bytes a row.
template <int WT> struct AStageShape {
    static constexpr int RBA = ChunksPerWave<WT, false>::value * BChunk<WT>::KC * 2;
    static constexpr int PIECES = RBA / 16, BYTES = kBgemmRows * RBA, OPS = BYTES / 1024;
    static_assert(BYTES % 1024 == 0 && (PIECES & (PIECES - 1)) == 0, "input staging shape");
};

template <int WT>
__device__ __forceinline__ void stage_act(const BgemmArgs& p, int cw0, int c1, char* dst) {
    using SH = AStageShape<WT>;
    constexpr int KC = BChunk<WT>::KC;
    const int lane = threadIdx.x & 63;
    const uint16_t* act = reinterpret_cast<const uint16_t*>(p.act);
#pragma unroll
    for (int i = 0; i < SH::OPS; ++i) {
        const int off = i * 1024 + lane * 16, r = off / SH::RBA, q = (off % SH::RBA) / 16;
        const int pc = q ^ (r & (SH::PIECES - 1));  // columns pc*8 .. +7
        const int c = min(cw0 + pc * 8 / KC, c1 - 1);
        const uint16_t* src = act + (size_t)min(r, p.B - 1) * p.K + (size_t)c * KC + (pc * 8) % KC;
        lds_dma16(reinterpret_cast<const char*>(src), dst + i * 1024);
    }
}

// Eight consecutive bf16 inputs of row fr at column kl of this wave's staged run.
template <int WT>
__device__ __forceinline__ uint4 read_a8(const char* src, int fr, int kl) {
    using SH = AStageShape<WT>;
    const int q = (kl >> 3) ^ (fr & (SH::PIECES - 1));
    return *reinterpret_cast<const uint4*>(src + fr * SH::RBA + q * 16);
}

// Four consecutive fp32 inputs of row fr at column kl of this wave's staged run.
template <int WT>
__device__ __forceinline__ float4 read_x4(const char* src, int fr, int kl) {
    using SH = XStageShape<WT>;
    const int q = (kl >> 2) ^ (fr & (SH::PIECES - 1));
    return *reinterpret_cast<const float4*>(src + fr * SH::RBX + q * 16);
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

// Everything the epilogue reads that does not depend on the products, loaded at
// the start so that it arrives while the weights stream in.
template <int EPT> struct EpiPre {
    float bias, scale;
    float xold[EPT];   // EPI_RESID
    int on[EPT];       // EPI_QKV: the row is active (appends its key and value)
    int slot[EPT];     //          at this KV slot
    int phys[EPT];     //          in this physical page
};

// FT = 2: the workgroup owns 64 features (each wave two MFMA tiles over its chunks),
// which halves the input rows staged per weight byte; used for the wide
// LayerNorm-fused linears.
template <int WT, int EPI, bool LN, int FT>
__global__ __launch_bounds__(kBgemmThreads) void bgemm_kernel(const BgemmArgs p) {
    using C = BChunk<WT>;
    constexpr int FEAT = FT * kBgemmFeat, EPT = kBgemmRows * FEAT / kBgemmThreads;
    constexpr int CPW = ChunksPerWave<WT, LN>::value, NT = kBgemmThreads;
    constexpr int MAXS = FT == 1 ? kBgemmMaxSplits : 8;
    static_assert(FT == 1 || (WT != FTTS_W4A16 && EPI != EPI_RESID), "two tiles per wave: 16-bit / int8 only, no stats");
    constexpr int SLICE = CPW * kBgemmWaves * C::KC, GBPER = (SLICE + NT - 1) / NT;  // columns of a K slice
    // staged input rows (fp32 for a LayerNorm input, else bf16); once consumed, the
    // wave's buffer takes its partial tile for the sum over waves
    constexpr int IN_BYTES = LN ? XStageShape<WT>::BYTES : AStageShape<WT>::BYTES;
    static_assert(IN_BYTES >= kBgemmRows * FEAT * 4, "wave tile must fit the staged inputs");
    __shared__ __attribute__((aligned(1024))) char s_xs[kBgemmWaves][IN_BYTES];
    __shared__ __attribute__((aligned(16))) float s_g[LN ? SLICE : 1];
    __shared__ __attribute__((aligned(16))) float s_b[LN ? SLICE : 1];
    __shared__ float2 s_gs[LN ? kLnGroups : 1][LN ? kBgemmRows : 1];
    __shared__ float s_mean[LN ? kBgemmRows : 1], s_rstd[LN ? kBgemmRows : 1];
    __shared__ __attribute__((aligned(1024))) char s_wt[kBgemmWaves][WStageShape<WT, LN, FT>::BYTES];
    int& s_last = *reinterpret_cast<int*>(s_wt[0]);  // used only after every product is formed
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int f = blockIdx.x, s = blockIdx.y, S = gridDim.y;
    const int n0 = f * FEAT;
    const int fr = lane & 31, h = lane >> 5;
    const int nchunks = p.K / C::KC;
    const int c0 = s * nchunks / S, c1 = (s + 1) * nchunks / S;
    // this thread's epilogue elements: feature ne, rows mrow(i)
    const int ne = min(n0 + (tid & (FEAT - 1)), p.N - 1);
    auto mrow = [&](int i) { return tid / FEAT + (NT / FEAT) * i; };

    // 1. LayerNorm inputs: this thread's (row, tile group) statistics, the slice's gains/biases.
    const int T = p.K / kStatTile, TP = (T + kLnGroups - 1) / kLnGroups;
    const int lr = tid & (kBgemmRows - 1), lq = tid >> 5;
    float2 st[LN ? kLnMaxTP : 1];
    uint16_t gr[LN ? GBPER : 1], br[LN ? GBPER : 1];
    const int k0 = c0 * C::KC, kn = (c1 - c0) * C::KC;
    if constexpr (LN) {
        const int m = min(lr, p.B - 1);
#pragma unroll
        for (int j = 0; j < kLnMaxTP; ++j) st[j] = p.ln_stats[(size_t)min(lq * TP + j, T - 1) * p.stats_ld + m];
#pragma unroll
        for (int j = 0; j < GBPER; ++j) {
            const int k = min(tid + NT * j, kn - 1);
            gr[j] = reinterpret_cast<const uint16_t*>(p.ln_g)[k0 + k];
            br[j] = reinterpret_cast<const uint16_t*>(p.ln_b)[k0 + k];
        }
    }
    // 2. epilogue operands
    EpiPre<EPT> pre;
    pre.bias = bf16_to_f32(reinterpret_cast<const uint16_t*>(p.bias)[ne]);
    pre.scale = WT == FTTS_W8A16 ? bf16_to_f32(p.scale[ne]) : 1.f;
    if constexpr (EPI == EPI_RESID) {
#pragma unroll
        for (int i = 0; i < EPT; ++i) pre.xold[i] = p.out[(size_t)min(mrow(i), p.B - 1) * p.out_stride + ne];
    }
    const bool kv_col = EPI == EPI_QKV && ne >= p.kv.d_model;
    if constexpr (EPI == EPI_QKV) {
#pragma unroll
        for (int i = 0; i < EPT; ++i) {
            const int m = min(mrow(i), p.B - 1);
            pre.on[i] = p.kv.active[m];
            pre.slot[i] = p.kv.seq_lens[m];
        }
    }
    // 3. every weight and input load of this wave: its chunks are c0 + wave * CPW + j
    // (indices past the slice repeat its last chunk and are not used)
    const int cw0 = c0 + wave * CPW;
    stage_weights<WT, LN, FT>(p, n0, cw0, c1, s_wt[wave]);
    if constexpr (LN) stage_x<WT>(p, cw0, c1, s_xs[wave]);
    else stage_act<WT>(p, cw0, c1, s_xs[wave]);
    C ch[CPW];
#pragma unroll
    for (int j = 0; j < CPW; ++j) load_chunk<WT, LN>(p, n0 + fr, fr, h, min(cw0 + j, c1 - 1), ch[j]);
    // Nothing that waits for a load may be scheduled above this point: every load
    // above is in flight before the first wait.
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (EPI == EPI_QKV) {
#pragma unroll
        for (int i = 0; i < EPT; ++i) {
            const int m = min(mrow(i), p.B - 1);
            // (an inactive row's slot may be anything: the page index is clamped and unused)
            const int pg = min(max(pre.slot[i], 0) / kPage, p.kv.max_pages - 1);
            pre.phys[i] = p.kv.block_table[(size_t)m * p.kv.max_pages + pg];
        }
    }
    __builtin_amdgcn_sched_barrier(0);
    // 4. LayerNorm: merge the statistics (law of total variance, fixed order), then
    // normalise the inputs into bf16 operands.
    if constexpr (LN) {
        // this group's tiles: lq * TP + j for j < cnt
        const int cnt = min(max(T - lq * TP, 0), TP);
        float sum = 0.f;
#pragma unroll
        for (int j = 0; j < kLnMaxTP; ++j) sum += j < cnt ? st[j].x : 0.f;
        const float mean_q = sum / (float)(max(cnt, 1) * kStatTile);
        float m2 = 0.f;
#pragma unroll
        for (int j = 0; j < kLnMaxTP; ++j) {
            const float dm = st[j].x * (1.0f / kStatTile) - mean_q;
            m2 += j < cnt ? st[j].y + (float)kStatTile * dm * dm : 0.f;
        }
        s_gs[lq][lr] = make_float2(sum, m2);
#pragma unroll
        for (int j = 0; j < GBPER; ++j)
            if (tid + NT * j < kn) {
                s_g[tid + NT * j] = bf16_to_f32(gr[j]);
                s_b[tid + NT * j] = bf16_to_f32(br[j]);
            }
        __syncthreads();
        if (tid < kBgemmRows) {
            // every group is read (empty ones hold zeros and weigh nothing): no branches
            float2 gs[kLnGroups];
#pragma unroll
            for (int q = 0; q < kLnGroups; ++q) gs[q] = s_gs[q][tid];
            float tot = 0.f;
#pragma unroll
            for (int q = 0; q < kLnGroups; ++q) tot += gs[q].x;
            const float mean = tot / (float)p.K;
            float M2 = 0.f;
#pragma unroll
            for (int q = 0; q < kLnGroups; ++q) {
                const int nq = min(max(T - q * TP, 0), TP) * kStatTile;
                const float dm = gs[q].x / (float)max(nq, 1) - mean;
                M2 += nq > 0 ? gs[q].y + (float)nq * dm * dm : 0.f;
            }
            s_mean[tid] = mean;
            s_rstd[tid] = tid < p.B ? 1.0f / sqrtf(M2 / (float)p.K + p.ln_eps) : 0.f;
        }
        __syncthreads();
        const float mean = s_mean[fr], rstd = s_rstd[fr];
        const bool live = fr < p.B;
#pragma unroll
        for (int j = 0; j < CPW; ++j) {
            // 16-value aligned offset into the slice's gains/biases
            const int kl = min(cw0 + j, c1 - 1) * C::KC + h * (C::KC / 2) - k0;
            const int kx = j * C::KC + h * (C::KC / 2);  // the same column in this wave's staged run
#pragma unroll
            for (int i = 0; i < C::KC / 16; ++i) {
                const float4 u = read_x4<WT>(s_xs[wave], fr, kx + 8 * i);
                const float4 v = read_x4<WT>(s_xs[wave], fr, kx + 8 * i + 4);
                const float4 g0 = *reinterpret_cast<const float4*>(s_g + kl + 8 * i);
                const float4 g1 = *reinterpret_cast<const float4*>(s_g + kl + 8 * i + 4);
                const float4 b0 = *reinterpret_cast<const float4*>(s_b + kl + 8 * i);
                const float4 b1 = *reinterpret_cast<const float4*>(s_b + kl + 8 * i + 4);
                const float xs[8] = {u.x, u.y, u.z, u.w, v.x, v.y, v.z, v.w};
                const float gs[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
                const float bs[8] = {b0.x, b0.y, b0.z, b0.w, b1.x, b1.y, b1.z, b1.w};
                float y[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const float t = (xs[e] - mean) * rstd * gs[e] + bs[e];
                    y[e] = live ? t : 0.f;
                }
                if (p.hidden && f == 0 && live) {  // feature tile 0 of each slice covers the slice's columns
                    float4* hd = reinterpret_cast<float4*>(p.hidden + (size_t)fr * p.K + k0 + kl + 8 * i);
                    hd[0] = make_float4(y[0], y[1], y[2], y[3]);
                    hd[1] = make_float4(y[4], y[5], y[6], y[7]);
                }
                ch[j].a[i] = make_uint4(pack_bf16x2(y[0], y[1]), pack_bf16x2(y[2], y[3]), pack_bf16x2(y[4], y[5]),
                                        pack_bf16x2(y[6], y[7]));
            }
        }
    }
    if constexpr (!LN) {
        // operand a[i] of chunk j: columns j*KC + h*KC/2 + 8i .. +7 of the staged run
        const bool live = fr < p.B;
#pragma unroll
        for (int j = 0; j < CPW; ++j)
#pragma unroll
            for (int i = 0; i < (int)(sizeof(ch[j].a) / 16); ++i) {
                const uint4 a = read_a8<WT>(s_xs[wave], fr, j * C::KC + h * (C::KC / 2) + 8 * i);
                ch[j].a[i] = live ? a : make_uint4(0, 0, 0, 0);
            }
    }
    // 5. products: tile t covers features n0 + 32 t ..
    bgemm_f32x16 acc[FT];
#pragma unroll
    for (int t = 0; t < FT; ++t)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[t][i] = 0.f;
#pragma unroll
    for (int j = 0; j < CPW; ++j) {
        if (cw0 + j < c1) {
#pragma unroll
            for (int t = 0; t < FT; ++t) {
                read_weights<WT, LN, FT>(s_wt[wave], fr + kBgemmFeat * t, h, j, ch[j]);
                bgemm_f32x16 part;
#pragma unroll
                for (int i = 0; i < 16; ++i) part[i] = 0.f;
#pragma unroll
                for (int st2 = 0; st2 < C::STEPS; ++st2) {
                    const bgemm_bf16x8 av = __builtin_bit_cast(bgemm_bf16x8, ch[j].a[st2]);
                    part = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, w_operand<WT>(ch[j], st2), part, 0, 0, 0);
                }
                if constexpr (WT == FTTS_W4A16) {
#pragma unroll
                    for (int i = 0; i < 16; ++i) acc[t][i] = fmaf(ch[j].s, part[i], acc[t][i]);
                } else {
#pragma unroll
                    for (int i = 0; i < 16; ++i) acc[t][i] += part[i];
                }
            }
        }
    }
    // acc[t][i] holds (sequence m, feature n0 + 32 t + fr): m = (i / 4) * 8 + h * 4 + i % 4
    auto red = [&](int w) { return reinterpret_cast<float*>(s_xs[w]); };
    {
        float* r = red(wave);
#pragma unroll
        for (int t = 0; t < FT; ++t)
#pragma unroll
            for (int i = 0; i < 16; ++i) r[((i >> 2) * 8 + h * 4 + (i & 3)) * FEAT + kBgemmFeat * t + fr] = acc[t][i];
    }
    __syncthreads();
    float v[EPT];
#pragma unroll
    for (int i = 0; i < EPT; ++i) {
        const int e = tid + NT * i;
        float t = 0.f;
#pragma unroll
        for (int w = 0; w < kBgemmWaves; ++w) t += red(w)[e];
        v[i] = t;
    }
    if (S > 1) {
        // Partials go out with device-coherent stores and are waited for before the
        // arrival count, so the last group reads them (device-coherent loads) without
        // any cache flush.
#pragma unroll
        for (int i = 0; i < EPT; ++i) {
            const int m = mrow(i), n = n0 + (tid & (FEAT - 1));
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
        // Every partial load goes out before the first add; only the S slices that
        // exist are read (uniform branches), the rest stay zero and add nothing.
        float pv[EPT][MAXS];
#pragma unroll
        for (int k = 0; k < MAXS; ++k) {
#pragma unroll
            for (int i = 0; i < EPT; ++i) pv[i][k] = 0.f;
            if (k < S) {
#pragma unroll
                for (int i = 0; i < EPT; ++i)
                    pv[i][k] = __hip_atomic_load(p.part + ((size_t)k * p.B + min(mrow(i), p.B - 1)) * p.N + ne,
                                                 __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
        }
#pragma unroll
        for (int i = 0; i < EPT; ++i) {
            float t = 0.f;
#pragma unroll
            for (int k = 0; k < MAXS; ++k) t += pv[i][k];
            v[i] = t;
        }
        if (tid == 0) __hip_atomic_store(p.count + f, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    // 6. epilogue
    const bool col_ok = n0 + (tid & (FEAT - 1)) < p.N;
    float xn[EPT];
#pragma unroll
    for (int i = 0; i < EPT; ++i) {
        const int m = mrow(i);
        const bool ok = m < p.B && col_ok;
        const float y = v[i] * pre.scale + pre.bias;
        xn[i] = 0.f;
        if (!ok) continue;
        const size_t o = (size_t)m * p.out_stride + ne;
        if constexpr (EPI == EPI_RESID) {
            xn[i] = pre.xold[i] + y;
            p.out[o] = xn[i];
        } else if constexpr (EPI == EPI_GELU) {
            reinterpret_cast<uint16_t*>(p.out_bf16)[o] = f32_to_bf16(gelu_tanh(y));
        } else {
            p.out[o] = y;
            if constexpr (EPI == EPI_QKV) {
                if (kv_col && pre.on[i]) {
                    const int d = p.kv.d_model, kvsel = ne >= 2 * d, r = ne - d - kvsel * d;
                    st_act<false>(p.kv.base,
                                  kv_offset(p.kv.layer, p.kv.n_pages, pre.phys[i], kvsel, p.kv.n_head, r / kHeadDim,
                                            pre.slot[i] % kPage) +
                                      r % kHeadDim,
                                  y);
                }
            }
        }
    }
    if constexpr (EPI == EPI_RESID) {
        if (p.stats_out) {
#pragma unroll
            for (int i = 0; i < EPT; ++i) {
                const float2 ts = tile_stats32(xn[i]);
                if ((tid & (FEAT - 1)) == 0 && mrow(i) < p.B) p.stats_out[(size_t)f * p.stats_ld + mrow(i)] = ts;
            }
        }
    }
}

template <int WT, bool LN>
static hipError_t bgemm_by_epi(int epi, int ft, const BgemmArgs& a, dim3 g, hipStream_t st) {
    const dim3 blk(kBgemmThreads);
    constexpr bool two = LN && WT != FTTS_W4A16;  // the only instantiations with FT = 2
    switch (epi) {
        case EPI_STORE:
            if (two && ft == 2) hipLaunchKernelGGL((bgemm_kernel<WT, EPI_STORE, LN, two ? 2 : 1>), g, blk, 0, st, a);
            else hipLaunchKernelGGL((bgemm_kernel<WT, EPI_STORE, LN, 1>), g, blk, 0, st, a);
            break;
        case EPI_QKV:
            if (two && ft == 2) hipLaunchKernelGGL((bgemm_kernel<WT, EPI_QKV, LN, two ? 2 : 1>), g, blk, 0, st, a);
            else hipLaunchKernelGGL((bgemm_kernel<WT, EPI_QKV, LN, 1>), g, blk, 0, st, a);
            break;
        case EPI_GELU:
            if (two && ft == 2) hipLaunchKernelGGL((bgemm_kernel<WT, EPI_GELU, LN, two ? 2 : 1>), g, blk, 0, st, a);
            else hipLaunchKernelGGL((bgemm_kernel<WT, EPI_GELU, LN, 1>), g, blk, 0, st, a);
            break;
        case EPI_RESID:
            if constexpr (LN) return hipErrorInvalidValue;  // the residual update never normalises its input
            else hipLaunchKernelGGL((bgemm_kernel<WT, EPI_RESID, false, 1>), g, blk, 0, st, a);
            break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

// K slices per feature tile: enough that each wave's share fits its registers.
int bgemm_splits(int wdtype, int N, int K, bool ln) {
    (void)N;
    const int kc = wdtype == FTTS_W4A16 ? 128 : 32;
    const int cpw = wdtype == FTTS_W4A16 ? (ln ? ChunksPerWave<FTTS_W4A16, true>::value
                                               : ChunksPerWave<FTTS_W4A16, false>::value)
                                         : (ln ? ChunksPerWave<FTTS_BF16, true>::value
                                               : ChunksPerWave<FTTS_BF16, false>::value);
    const int chunks = K / kc, per_group = kBgemmWaves * cpw;
    return (chunks + per_group - 1) / per_group;
}

bool bgemm_supported(int wdtype, int K, bool ln) {
    if (wdtype == FTTS_F32) return false;
    if (ln && (K % kStatTile != 0 || K > kLnMaxK)) return false;
    return K % (wdtype == FTTS_W4A16 ? 128 : 32) == 0 && bgemm_splits(wdtype, 0, K, ln) <= kBgemmMaxSplits;
}

hipError_t launch_bgemm(int wdtype, int epi, const BgemmArgs& in, hipStream_t st) {
    // The LM head is never quantised.
    const int wt = epi == EPI_STORE ? FTTS_BF16 : wdtype;
    const bool ln = in.ln_x != nullptr;
    if (!bgemm_supported(wt, in.K, ln)) return hipErrorInvalidValue;
    if (epi == EPI_RESID && in.stats_out && in.N % kStatTile != 0) return hipErrorInvalidValue;
    const int S = bgemm_splits(wt, in.N, in.K, ln);
    // 64 features per workgroup for a LayerNorm-fused linear whose 32-feature grid
    // would not be resident at once (three workgroups per CU): fewer, larger groups
    // beat a second round.
    static const int n_cu = [] {
        int dev = 0, n = 0;
        if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
            return 0;
        return n;
    }();
    const long tiles32 = (in.N + kBgemmFeat - 1) / kBgemmFeat;
    const int ft = ln && wt != FTTS_W4A16 && epi != EPI_RESID && S <= 8 && tiles32 * S > 3L * n_cu ? 2 : 1;
    const dim3 g((in.N + kBgemmFeat * ft - 1) / (kBgemmFeat * ft), S);
    for (int b0 = 0; b0 < in.B; b0 += kBgemmRows) {
        BgemmArgs a = in;
        a.B = in.B - b0 < kBgemmRows ? in.B - b0 : kBgemmRows;
        if (in.act) a.act = reinterpret_cast<const uint16_t*>(in.act) + (size_t)b0 * in.K;
        if (in.ln_x) a.ln_x = in.ln_x + (size_t)b0 * in.K;
        if (in.hidden) a.hidden = in.hidden + (size_t)b0 * in.K;
        if (in.ln_stats) a.ln_stats = in.ln_stats + b0;
        if (in.stats_out) a.stats_out = in.stats_out + b0;
        if (in.out) a.out = in.out + (size_t)b0 * in.out_stride;
        if (in.out_bf16) a.out_bf16 = reinterpret_cast<uint16_t*>(in.out_bf16) + (size_t)b0 * in.out_stride;
        if (epi == EPI_QKV) {
            a.kv.seq_lens = in.kv.seq_lens + b0;
            a.kv.active = in.kv.active + b0;
            a.kv.block_table = in.kv.block_table + (size_t)b0 * in.kv.max_pages;
        }
        hipError_t e;
        switch (wt) {
            case FTTS_BF16: e = ln ? bgemm_by_epi<FTTS_BF16, true>(epi, ft, a, g, st) : bgemm_by_epi<FTTS_BF16, false>(epi, ft, a, g, st); break;
            case FTTS_W8A16: e = ln ? bgemm_by_epi<FTTS_W8A16, true>(epi, ft, a, g, st) : bgemm_by_epi<FTTS_W8A16, false>(epi, ft, a, g, st); break;
            case FTTS_W4A16: e = ln ? bgemm_by_epi<FTTS_W4A16, true>(epi, ft, a, g, st) : bgemm_by_epi<FTTS_W4A16, false>(epi, ft, a, g, st); break;
            default: return hipErrorInvalidValue;
        }
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace ftts
