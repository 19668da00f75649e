// Persistent single-launch decode step for the IndexTTS-2 GPT shape
// (d_model 1280, 20 heads of 64, d_ff 5120), batch 1-2, bf16 / W8A16 / W4A16.
//
// Why: at batch 1 one step is about 121 dependent phases (5 per layer plus the
// head) over 0.97 GB of bf16 weights.  Separate kernels pay a launch gap and a
// cold memory ramp per phase; here one launch covers the whole step and each
// workgroup holds the next phase's weight share in registers before it waits
// for that phase's input, so the weight stream overlaps the synchronisation.
//
// Layout: one 512-thread workgroup per CU (256).  Before waiting for a phase's
// input every thread issues its share of the NEXT phase's weights; the wait
// (a poll of the exchange words) then overlaps that stream.  A wave's loads
// retire in issue order, so the poll also waits for the prefetch, which at
// <= 51 KB per CU lands well within the exchange latency.
//
// Exchange: every value crossing workgroups travels as one 64-bit word
// (fp32 value | epoch << 32) written and read with device-coherent (sc1)
// accesses.  A consumer knows its data has arrived when every word carries the
// epoch of the current (step, event); no flags, counters or fences are needed.
// Each phase depends on all workgroups of the previous one, so a single buffer
// per kind of data is never overwritten before every reader has consumed it.
// Waits are bounded: on timeout a workgroup raises the abort word and every
// workgroup leaves at its next wait (ftts_check_workspace reports it).
//
// Work split per layer (rows of a matrix split evenly over the 256 groups):
//   P0  LN1 + q/k/v rows (15 per group), k/v also appended to the KV pool
//   P1  attention, one group per (sequence, head); the new token's k/v come from
//       the exchange, older slots from the pool (written by earlier launches)
//   P2  out-proj rows (5 per group) + residual of the group's own x rows
//   P3  LN2 + FC1 rows (20 per group) + GELU
//   P4  FC2 rows (5 per group) + residual
// then LN_f + LM head rows (<= 64 per group) and, for greedy decoding, the
// argmax over all groups' candidates.
#include "gemv_impl.hpp"
#include "kv_page.hpp"

namespace ftts {
namespace mega {

constexpr int NT = 512;               // threads per workgroup (8 waves)
constexpr unsigned kSpinLimit = 1u << 19;  // about a second of polling

template <int WT> struct Tiles;  // (lanes per row, 16-byte chunks per lane) per phase
template <> struct Tiles<FTTS_BF16> {
    static constexpr int QL = 32, QC = 5, OL = 32, OC = 5, AL = 16, AC = 10, BL = 64, BC = 10;
};
template <> struct Tiles<FTTS_W8A16> {
    static constexpr int QL = 16, QC = 5, OL = 16, OC = 5, AL = 16, AC = 5, BL = 64, BC = 5;
};
template <> struct Tiles<FTTS_W4A16> {
    static constexpr int QL = 8, QC = 5, OL = 8, OC = 5, AL = 8, AC = 5, BL = 32, BC = 5;
};
constexpr int HL = 8, HC = 20;        // LM head (bf16): 64 rows per group

__device__ __forceinline__ uint32_t ld_agent(const uint32_t* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_agent(uint32_t* p, uint32_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void put(uint64_t* p, uint32_t epoch, float v) {
    __hip_atomic_store(p, ((uint64_t)epoch << 32) | __float_as_uint(v), __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
}

typedef __attribute__((address_space(3))) char lds_char;

// Copy `bytes` (a multiple of 16) from global memory to LDS with direct
// global->LDS loads: each wave moves 1 KB per instruction, no registers held.
// The LDS buffer must be a multiple of 1 KB long (the last wave instruction may
// write up to 1 KB - 16 bytes past `bytes`, with a repeat of the last chunk).
__device__ __forceinline__ void dma_to_lds(const void* src, int bytes, char* dst) {
    const int n = bytes >> 4;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const char* s = reinterpret_cast<const char*>(src);
    lds_char* d = (lds_char*)(dst);
    for (int c0 = wave * 64; c0 < n; c0 += NT) {
        const int c = min(c0 + lane, n - 1);
        __builtin_amdgcn_global_load_lds(s + (size_t)c * 16, d + c0 * 16, 16, 0, 0);
    }
}

// One phase's share of a weight matrix: rows [r0, r0 + R), contiguous in memory,
// copied into an LDS buffer ahead of use; per-row bias and quantisation
// parameters of this thread's row are kept in registers.
template <int WT, int LPR, int NCH, int K>
struct Share {
    static constexpr int ROW_BYTES = WT == FTTS_W4A16 ? K / 2 : WT == FTTS_W8A16 ? K : 2 * K;
    float s4[NCH], z4[NCH];
    float rs, bias;
    int R;
    char* buf;
    __device__ __forceinline__ void issue(const void* W, const void* S, const void* Z, const void* bias_p, int r0,
                                          int nrows, char* lds) {
        const int li = threadIdx.x & (LPR - 1);
        const int row = r0 + min((int)threadIdx.x / LPR, nrows - 1);
        R = nrows;
        buf = lds;
        bias = bf16_to_f32(reinterpret_cast<const uint16_t*>(bias_p)[row]);
        rs = 1.f;
        if constexpr (WT == FTTS_W8A16) rs = bf16_to_f32(reinterpret_cast<const uint16_t*>(S)[row]);
#pragma unroll
        for (int i = 0; i < NCH; ++i) {
            s4[i] = 0.f;
            z4[i] = 0.f;
            if constexpr (WT == FTTS_W4A16) {
                const int g = ((li + i * LPR) * 32) >> 7;
                s4[i] = bf16_to_f32(reinterpret_cast<const uint16_t*>(S)[(size_t)row * (K / 128) + g]);
                z4[i] = bf16_to_f32(reinterpret_cast<const uint16_t*>(Z)[(size_t)row * (K / 128) + g]);
            }
        }
        dma_to_lds(reinterpret_cast<const char*>(W) + (size_t)r0 * ROW_BYTES, nrows * ROW_BYTES, lds);
    }
    // acc[b] = dot product of this thread's row with s_in[b] (+ bias); every lane of the row gets it.
    template <int B_>
    __device__ __forceinline__ void dot(const float* s_in, const float* s_xs, int B, float (&acc)[B_]) const {
        constexpr int EPC = WInfo<WT>::EPC;
        const int li = threadIdx.x & (LPR - 1);
        const int slot = min((int)threadIdx.x / LPR, R - 1);
        const uint4* wrow = reinterpret_cast<const uint4*>(buf + slot * ROW_BYTES);
#pragma unroll
        for (int b = 0; b < B_; ++b) acc[b] = 0.f;
#pragma unroll
        for (int i = 0; i < NCH; ++i) {
            const int c = li + i * LPR;
            dot_chunk<WT, B_>(wrow[c], s_in + c * EPC, K, B, acc, s4[i], z4[i], s_xs + c, K / 32);
        }
#pragma unroll
        for (int b = 0; b < B_; ++b) {
            float v = acc[b];
#pragma unroll
            for (int o = LPR >> 1; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
            acc[b] = fmaf(v, rs, bias);
        }
    }
};

// The LM head (bf16), streamed straight into registers: 64 rows per group at most.
template <int LPR, int NCH, int K>
struct RegShare {
    uint4 w[NCH];
    float bias;
    __device__ __forceinline__ void issue(const void* W, const void* bias_p, int row) {
        const int li = threadIdx.x & (LPR - 1);
        bias = bf16_to_f32(reinterpret_cast<const uint16_t*>(bias_p)[row]);
        const uint4* wr = reinterpret_cast<const uint4*>(reinterpret_cast<const char*>(W) + (size_t)2 * K * row);
#pragma unroll
        for (int i = 0; i < NCH; ++i) w[i] = ld_stream(wr + li + i * LPR);
    }
    template <int B_>
    __device__ __forceinline__ void dot(const float* s_in, int B, float (&acc)[B_]) const {
        const int li = threadIdx.x & (LPR - 1);
#pragma unroll
        for (int b = 0; b < B_; ++b) acc[b] = 0.f;
#pragma unroll
        for (int i = 0; i < NCH; ++i) {
            const int c = li + i * LPR;
            dot_chunk<FTTS_BF16, B_>(w[i], s_in + c * 8, K, B, acc, 0.f, 0.f, nullptr, 0);
        }
#pragma unroll
        for (int b = 0; b < B_; ++b) {
            float v = acc[b];
#pragma unroll
            for (int o = LPR >> 1; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
            acc[b] = v + bias;
        }
    }
};

// Wait until the n words at src all carry `epoch`, then store their values to dst
// (LDS).  All threads of the workgroup take part and agree on the outcome.  The
// words are read with device-scope relaxed atomic loads (sc1), which the
// compiler waits for before their use.  Returns false when the wait ran out or
// another workgroup gave up.
__device__ __forceinline__ bool gather(const uint64_t* src, int n, uint32_t epoch, float* dst, uint32_t* ctl) {
    constexpr int U = 10;
    const int tid = threadIdx.x;
    for (int base = 0; base < n; base += NT * U) {
        uint64_t v[U];
        unsigned spins = 0;
        while (true) {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int j = min(base + tid + NT * u, n - 1);
                v[u] = __hip_atomic_load(src + j, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
            bool ok = true;
#pragma unroll
            for (int u = 0; u < U; ++u) ok = ok && (uint32_t)(v[u] >> 32) == epoch;
            if (__syncthreads_and(ok)) break;
            const bool give_up = ++spins > kSpinLimit || ld_agent(ctl + 1) != 0;
            if (__syncthreads_or(give_up)) {
                if (tid == 0) st_agent(ctl + 1, 1u);
                return false;
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int j = base + tid + NT * u;
            if (j < n) dst[j] = __uint_as_float((uint32_t)v[u]);
        }
    }
    __syncthreads();
    return true;
}

// Sum over the workgroup (every thread gets it).
__device__ __forceinline__ float block_sum(float v, float* red) {
    v = wave_sum(v);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
    __syncthreads();
    float t = 0.f;
#pragma unroll
    for (int i = 0; i < NT / 64; ++i) t += red[i];
    __syncthreads();
    return t;
}

// LayerNorm of the B rows of src (LDS, width D) into dst; g/b hold this thread's
// columns tid, tid + 512, ... (preloaded).
template <int NPER>
__device__ __forceinline__ void layer_norm_rows(const float* src, float* dst, const float (&g)[NPER],
                                                const float (&bb)[NPER], float eps, int B, float* red) {
    const int tid = threadIdx.x;
    for (int b = 0; b < B; ++b) {
        const float* x = src + b * D;
        float xv[NPER];
        float s = 0.f;
#pragma unroll
        for (int i = 0; i < NPER; ++i) {
            const int k = tid + NT * i;
            xv[i] = k < D ? x[k] : 0.f;
            s += xv[i];
        }
        const float mean = block_sum(s, red) / (float)D;
        float var = 0.f;
#pragma unroll
        for (int i = 0; i < NPER; ++i) {
            const int k = tid + NT * i;
            const float d = k < D ? xv[i] - mean : 0.f;
            var = fmaf(d, d, var);
        }
        var = block_sum(var, red) / (float)D;
        const float rstd = 1.0f / sqrtf(var + eps);
#pragma unroll
        for (int i = 0; i < NPER; ++i) {
            const int k = tid + NT * i;
            if (k < D) dst[b * D + k] = (xv[i] - mean) * rstd * g[i] + bb[i];
        }
    }
    __syncthreads();
}

template <int NPER>
__device__ __forceinline__ void load_ln(const void* g, const void* bb, float (&gv)[NPER], float (&bv)[NPER]) {
#pragma unroll
    for (int i = 0; i < NPER; ++i) {
        const int k = min((int)threadIdx.x + NT * i, D - 1);
        gv[i] = bf16_to_f32(reinterpret_cast<const uint16_t*>(g)[k]);
        bv[i] = bf16_to_f32(reinterpret_cast<const uint16_t*>(bb)[k]);
    }
}

// Per-32-column sums of the staged activations (W4A16 only).
__device__ __forceinline__ void chunk_sums(const float* src, float* xs, int K, int B) {
    const int nc = K / 32;
    for (int i = threadIdx.x; i < B * nc; i += NT) {
        const int b = i / nc, c = i - b * nc;
        const float* p = src + b * K + c * 32;
        float s = 0.f;
#pragma unroll
        for (int j = 0; j < 32; ++j) s += p[j];
        xs[b * nc + c] = s;
    }
    __syncthreads();
}

template <int WT, int BMAX>
__global__ __launch_bounds__(NT) void decode_mega_kernel(const Args a) {
    using T = Tiles<WT>;
    constexpr int NPER = (D + NT - 1) / NT;
    constexpr int kBuf = 51200;                                       // largest share: 20 x 1280 or 5 x 5120 bf16
    __shared__ __attribute__((aligned(1024))) char s_w[2][kBuf];     // weight shares, alternating by phase
    __shared__ __attribute__((aligned(16))) float s_in[BMAX * FF];    // phase input (normalised for LN phases)
    __shared__ __attribute__((aligned(16))) float s_x[BMAX * D];      // residual stream as last gathered
    __shared__ float s_xs[BMAX * FF / 32];                            // W4A16 chunk sums
    __shared__ float s_q[3 * 64];                                     // attention: q, k, v of the new token
    __shared__ float s_pm[8], s_pl[8], s_po[8][64];                   // attention wave partials
    __shared__ float s_cv[BMAX][64];                                  // head: per-slot best value
    __shared__ int s_ci[BMAX][64];                                    //       and its row
    __shared__ int s_active[BMAX];
    __shared__ float s_red[NT / 64];
    __shared__ int s_abort;

    const int wg = blockIdx.x, tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int B = a.B;
    const uint32_t step = ld_agent(a.ctl);
    auto E = [&](int ev) { return (step << 8) | (uint32_t)ev; };
    if (tid == 0) s_abort = ld_agent(a.ctl + 1) != 0;
    __syncthreads();
    if (s_abort) return;

    const int q0 = 3 * D * wg / G, q1 = 3 * D * (wg + 1) / G;
    const int d0 = D * wg / G, d1 = D * (wg + 1) / G;
    const int f0 = FF * wg / G, f1 = FF * (wg + 1) / G;
    const int v0 = a.V * wg / G, v1 = a.V * (wg + 1) / G;
    const bool is_att = wg < B * NH;
    const int att_b = wg / NH, att_h = wg % NH;

    Share<WT, T::QL, T::QC, D> pq;
    Share<WT, T::OL, T::OC, D> po;
    Share<WT, T::AL, T::AC, D> p1;
    Share<WT, T::BL, T::BC, FF> p2;
    const int sq = tid / T::QL, so = tid / T::OL, s1 = tid / T::AL, s2 = tid / T::BL, sh = tid / HL;
    float lg[NPER], lb[NPER];
    // Buffer use: q/k/v and FC1 in s_w[0], out-proj and FC2 in s_w[1]; each DMA
    // into a buffer is issued after a barrier that follows the buffer's last read.
    pq.issue(a.qkv_w.at(0), a.qkv_s.at(0), a.qkv_z.at(0), a.qkv_b.at(0), q0, q1 - q0, s_w[0]);

    for (int l = 0; l < a.n_layer; ++l) {
        // ---------------- P0: LN1 + q/k/v -------------------------------------------------
        load_ln<NPER>(a.ln1_g.at(l), a.ln1_b.at(l), lg, lb);
        po.issue(a.out_w.at(l), a.out_s.at(l), a.out_z.at(l), a.out_b.at(l), d0, d1 - d0, s_w[1]);
        if (l == 0) {  // the embedding, computed locally by every group
            for (int b = 0; b < B; ++b) {
                const int t = a.tokens[b], p = a.positions[b], s = a.seq_lens[b];
                bool act = t >= 0 && t < a.V && p >= 0 && p < a.n_pos && s >= 0 && s < a.max_pages * kPage;
                if (act) {
                    const int phys = a.block_table[(size_t)b * a.max_pages + s / kPage];
                    act = phys >= 0 && phys < a.n_pages;
                }
                for (int k = tid; k < D; k += NT)
                    s_x[b * D + k] = act ? ld_act<false>(a.tok_emb, (size_t)t * D + k) +
                                               ld_act<false>(a.pos_emb, (size_t)p * D + k)
                                         : 0.f;
                if (tid == 0) {
                    s_active[b] = act;
                    if (wg == 0) a.active_out[b] = act;
                }
            }
            __syncthreads();
        } else if (!gather(a.ex_x, B * D, E(5 * l), s_x, a.ctl)) {
            return;
        }
        layer_norm_rows<NPER>(s_x, s_in, lg, lb, a.eps, B, s_red);
        if constexpr (WT == FTTS_W4A16) chunk_sums(s_in, s_xs, D, B);
        {
            float acc[BMAX];
            pq.template dot<BMAX>(s_in, s_xs, B, acc);
            const int row = q0 + sq;
            const int li = tid & (T::QL - 1);
            if (sq < q1 - q0) {
#pragma unroll
                for (int b = 0; b < BMAX; ++b) {
                    if (b < B && li == b) {
                        put(a.ex_qkv + (size_t)b * 3 * D + row, E(5 * l + 1), acc[b]);
                        if (row >= D && s_active[b]) {
                            const int kvsel = row >= 2 * D;
                            const int r = row - D - kvsel * D;
                            const int slot = a.seq_lens[b];
                            const int phys = a.block_table[(size_t)b * a.max_pages + slot / kPage];
                            st_act<false>(a.kv,
                                          kv_offset(l, a.n_pages, phys, kvsel, NH, r / 64, slot % kPage) + r % 64,
                                          acc[b]);
                        }
                    }
                }
            }
        }
        // ---------------- P1: attention, one group per (sequence, head) ---------------------
        __syncthreads();  // P0's reads of s_w[0] are done
        p1.issue(a.fc1_w.at(l), a.fc1_s.at(l), a.fc1_z.at(l), a.fc1_b.at(l), f0, f1 - f0, s_w[0]);
        if (is_att) {
            const int b = att_b, h = att_h;
            const int ncache = a.seq_lens[b];                 // cached slots (new token excluded)
            const int npg = (ncache + kPage - 1) / kPage;
            const int grp = lane >> 3, sub = lane & 7;
            // this wave's first page goes out before the new token's q/k/v arrive
            const int lp = wave + 8 * lane;
            const int my_phys = (s_active[b] && lp < npg) ? a.block_table[(size_t)b * a.max_pages + lp] : -1;
            const int my_pages = (s_active[b] && npg > wave) ? (npg - wave + 7) / 8 : 0;
            PageRegs<false> cur;
            bool ok_cur = false;
            auto bases = [&](int j, size_t& kb, size_t& vb) {
                int phys = __shfl(my_phys, j, kWave);
                const bool ok = phys >= 0 && phys < a.n_pages;
                phys = ok ? phys : 0;
                kb = kv_offset(l, a.n_pages, phys, 0, NH, h, 0);
                vb = kv_offset(l, a.n_pages, phys, 1, NH, h, 0);
                return ok;
            };
            size_t kb, vb;
            if (my_pages > 0) {
                ok_cur = bases(0, kb, vb);
                load_page<false>(a.kv, kb, vb, lane, cur);
            }
            const uint64_t* src = a.ex_qkv + (size_t)b * 3 * D + h * 64;
            if (!gather(src, 64, E(5 * l + 1), s_q, a.ctl) || !gather(src + D, 64, E(5 * l + 1), s_q + 64, a.ctl) ||
                !gather(src + 2 * D, 64, E(5 * l + 1), s_q + 128, a.ctl))
                return;
            float q[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) q[j] = s_q[sub * 8 + j] * 0.125f;  // 1/sqrt(64), exact
            // The cache holds keys and values in bf16; attend to the new token as cached.
            auto cached = [](float v) { return bf16_to_f32(f32_to_bf16(v)); };
            float m = -INFINITY, lsum = 0.f, o[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) o[j] = 0.f;
            if (wave == 0) {  // the new token itself, straight from the exchange
                float t = 0.f;
#pragma unroll
                for (int j = 0; j < 8; ++j) t = fmaf(q[j], cached(s_q[64 + sub * 8 + j]), t);
                t += __shfl_xor(t, 1, kWave);
                t += __shfl_xor(t, 2, kWave);
                t += __shfl_xor(t, 4, kWave);
                m = t;
                if (grp == 0) {
                    lsum = 1.f;
#pragma unroll
                    for (int j = 0; j < 8; ++j) o[j] = cached(s_q[128 + sub * 8 + j]);
                }
            }
            for (int j = 0; j < my_pages; ++j) {
                const int p = wave + 8 * j;
                if (j > 0) {
                    ok_cur = bases(j, kb, vb);
                    load_page<false>(a.kv, kb, vb, lane, cur);
                }
                float sc[8];
                float pm = -INFINITY;
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    float kv[8];
                    unpack8<false>(cur, false, i, kv);
                    float t = 0.f;
#pragma unroll
                    for (int d = 0; d < 8; ++d) t = fmaf(q[d], kv[d], t);
                    t += __shfl_xor(t, 1, kWave);
                    t += __shfl_xor(t, 2, kWave);
                    t += __shfl_xor(t, 4, kWave);
                    const int tok = p * kPage + i * 8 + grp;
                    sc[i] = (ok_cur && tok < ncache) ? t : -INFINITY;
                    pm = fmaxf(pm, sc[i]);
                }
                pm = fmaxf(pm, __shfl_xor(pm, 8, kWave));
                pm = fmaxf(pm, __shfl_xor(pm, 16, kWave));
                pm = fmaxf(pm, __shfl_xor(pm, 32, kWave));
                if (pm > -INFINITY) {
                    const float mn = fmaxf(m, pm);
                    const float alpha = expf(m - mn);
                    m = mn;
                    lsum *= alpha;
#pragma unroll
                    for (int d = 0; d < 8; ++d) o[d] *= alpha;
#pragma unroll
                    for (int i = 0; i < 8; ++i) {
                        if (sc[i] > -INFINITY) {  // slots past the context never enter the sum
                            const float pr = expf(sc[i] - m);
                            float vv[8];
                            unpack8<false>(cur, true, i, vv);
                            lsum += pr;
#pragma unroll
                            for (int d = 0; d < 8; ++d) o[d] = fmaf(pr, vv[d], o[d]);
                        }
                    }
                }
            }
#pragma unroll
            for (int d = 0; d < 8; ++d) {
                float t = o[d];
                t += __shfl_xor(t, 8, kWave);
                t += __shfl_xor(t, 16, kWave);
                t += __shfl_xor(t, 32, kWave);
                o[d] = t;
            }
            lsum += __shfl_xor(lsum, 8, kWave);
            lsum += __shfl_xor(lsum, 16, kWave);
            lsum += __shfl_xor(lsum, 32, kWave);
            if (lane < 8) {
#pragma unroll
                for (int d = 0; d < 8; ++d) s_po[wave][lane * 8 + d] = o[d];
            }
            if (lane == 0) {
                s_pm[wave] = m;
                s_pl[wave] = lsum;
            }
            __syncthreads();
            if (tid < 64) {  // log-sum-exp merge of the 8 wave partials
                float M = -INFINITY;
#pragma unroll
                for (int i = 0; i < 8; ++i) M = fmaxf(M, s_pm[i]);
                float L = 0.f, acc = 0.f;
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    if (s_pm[i] > -INFINITY) {
                        const float wgt = expf(s_pm[i] - M);
                        L = fmaf(s_pl[i], wgt, L);
                        acc = fmaf(s_po[i][tid], wgt, acc);
                    }
                }
                put(a.ex_o + (size_t)b * D + h * 64 + tid, E(5 * l + 2), (s_active[b] && L > 0.f) ? acc / L : 0.f);
            }
        }
        // ---------------- P2: out-proj + residual --------------------------------------------
        __syncthreads();  // every wave is done reading s_in (P0) before it is overwritten
        if (!gather(a.ex_o, B * D, E(5 * l + 2), s_in, a.ctl)) return;
        if constexpr (WT == FTTS_W4A16) chunk_sums(s_in, s_xs, D, B);
        {
            float acc[BMAX];
            po.template dot<BMAX>(s_in, s_xs, B, acc);
            const int row = d0 + so;
            const int li = tid & (T::OL - 1);
            if (so < d1 - d0) {
#pragma unroll
                for (int b = 0; b < BMAX; ++b)
                    if (b < B && li == b) put(a.ex_x + (size_t)b * D + row, E(5 * l + 3), s_x[b * D + row] + acc[b]);
            }
        }
        // ---------------- P3: LN2 + FC1 + GELU -----------------------------------------------
        __syncthreads();  // every wave is done reading s_in / s_x / s_w[1] of P2
        load_ln<NPER>(a.ln2_g.at(l), a.ln2_b.at(l), lg, lb);
        p2.issue(a.fc2_w.at(l), a.fc2_s.at(l), a.fc2_z.at(l), a.fc2_b.at(l), d0, d1 - d0, s_w[1]);
        if (!gather(a.ex_x, B * D, E(5 * l + 3), s_x, a.ctl)) return;
        layer_norm_rows<NPER>(s_x, s_in, lg, lb, a.eps, B, s_red);
        if constexpr (WT == FTTS_W4A16) chunk_sums(s_in, s_xs, D, B);
        {
            float acc[BMAX];
            p1.template dot<BMAX>(s_in, s_xs, B, acc);
            const int row = f0 + s1;
            const int li = tid & (T::AL - 1);
            if (s1 < f1 - f0) {
#pragma unroll
                for (int b = 0; b < BMAX; ++b)
                    if (b < B && li == b) put(a.ex_h + (size_t)b * FF + row, E(5 * l + 4), gelu_tanh(acc[b]));
            }
        }
        // ---------------- P4: FC2 + residual -------------------------------------------------
        __syncthreads();  // every wave is done reading s_in / s_w[0] of P3
        if (l + 1 < a.n_layer)
            pq.issue(a.qkv_w.at(l + 1), a.qkv_s.at(l + 1), a.qkv_z.at(l + 1), a.qkv_b.at(l + 1), q0, q1 - q0, s_w[0]);
        if (!gather(a.ex_h, B * FF, E(5 * l + 4), s_in, a.ctl)) return;
        if constexpr (WT == FTTS_W4A16) chunk_sums(s_in, s_xs, FF, B);
        {
            float acc[BMAX];
            p2.template dot<BMAX>(s_in, s_xs, B, acc);
            const int row = d0 + s2;
            const int li = tid & (T::BL - 1);
            if (s2 < d1 - d0) {
#pragma unroll
                for (int b = 0; b < BMAX; ++b)
                    if (b < B && li == b) put(a.ex_x + (size_t)b * D + row, E(5 * l + 5), s_x[b * D + row] + acc[b]);
            }
        }
        __syncthreads();  // s_in / s_x free for the next layer
    }

    // ---------------- LN_f + LM head (+ greedy argmax) -------------------------------------
    // (the head's weights stream while the last FC2 outputs are gathered)
    RegShare<HL, HC, D> ph;
    ph.issue(a.head_w, a.head_b, v0 + min(sh, v1 - v0 - 1));
    load_ln<NPER>(a.lnf_g, a.lnf_b, lg, lb);
    if (!gather(a.ex_x, B * D, E(5 * a.n_layer), s_x, a.ctl)) return;
    layer_norm_rows<NPER>(s_x, s_in, lg, lb, a.eps, B, s_red);
    {
        float acc[BMAX];
        ph.template dot<BMAX>(s_in, B, acc);
        const int row = v0 + sh;
        const int li = tid & (HL - 1);
        const bool mine = sh < v1 - v0;
#pragma unroll
        for (int b = 0; b < BMAX; ++b) {
            if (b < B && li == b) {
                if (mine) a.logits[(size_t)b * a.V + row] = acc[b];
                s_cv[b][sh] = mine ? acc[b] : -INFINITY;
                s_ci[b][sh] = mine ? row : 0x7FFFFFFF;
            }
        }
    }
    if (!a.greedy) {
        if (wg == 0 && tid == 0) st_agent(a.ctl, step + 1);
        return;
    }
    __syncthreads();
    if (tid < B) {  // this group's best row for each sequence
        float bv = -INFINITY;
        int bi = 0x7FFFFFFF;
        for (int s = 0; s < NT / HL; ++s) {
            const float v = s_cv[tid][s];
            const int i = s_ci[tid][s];
            if (v > bv || (v == bv && i < bi)) {
                bv = v;
                bi = i;
            }
        }
        put(a.ex_arg + ((size_t)wg * B + tid) * 2, E(5 * a.n_layer + 1), bv);
        put(a.ex_arg + ((size_t)wg * B + tid) * 2 + 1, E(5 * a.n_layer + 1), __int_as_float(bi));
    }
    if (wg != 0) return;
    if (!gather(a.ex_arg, G * B * 2, E(5 * a.n_layer + 1), s_in, a.ctl)) return;
    if (wave < B) {
        const int b = wave;
        float bv = -INFINITY;
        int bi = 0x7FFFFFFF;
        for (int g = lane; g < G; g += 64) {
            const float v = s_in[(g * B + b) * 2];
            const int i = __float_as_int(s_in[(g * B + b) * 2 + 1]);
            if (v > bv || (v == bv && i < bi)) {
                bv = v;
                bi = i;
            }
        }
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) {
            const float ov = __shfl_xor(bv, o, kWave);
            const int oi = __shfl_xor(bi, o, kWave);
            if (ov > bv || (ov == bv && oi < bi)) {
                bv = ov;
                bi = oi;
            }
        }
        if (lane == 0) a.sampled[b] = s_active[b] ? (bi < a.V ? bi : 0) : -1;
    }
    if (tid == 0) st_agent(a.ctl, step + 1);
}

}  // namespace mega

hipError_t launch_decode_mega(int wdtype, const mega::Args& a, hipStream_t st) {
    using namespace mega;
    const dim3 g(G), blk(NT);
    switch (wdtype) {
        case FTTS_BF16:
            if (a.B <= 1) hipLaunchKernelGGL((decode_mega_kernel<FTTS_BF16, 1>), g, blk, 0, st, a);
            else hipLaunchKernelGGL((decode_mega_kernel<FTTS_BF16, BM>), g, blk, 0, st, a);
            break;
        case FTTS_W8A16:
            if (a.B <= 1) hipLaunchKernelGGL((decode_mega_kernel<FTTS_W8A16, 1>), g, blk, 0, st, a);
            else hipLaunchKernelGGL((decode_mega_kernel<FTTS_W8A16, BM>), g, blk, 0, st, a);
            break;
        case FTTS_W4A16:
            if (a.B <= 1) hipLaunchKernelGGL((decode_mega_kernel<FTTS_W4A16, 1>), g, blk, 0, st, a);
            else hipLaunchKernelGGL((decode_mega_kernel<FTTS_W4A16, BM>), g, blk, 0, st, a);
            break;
        default:
            return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace ftts
