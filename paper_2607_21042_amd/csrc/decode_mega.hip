// Persistent single-launch decode step for the IndexTTS-2 GPT shape
// (d_model 1280, 20 heads of 64, d_ff 5120), batch 1-2, bf16 / W8A16 / W4A16.
//
// Why: at batch 1 one step is about 121 dependent phases (5 per layer plus the
// head) over 0.97 GB of bf16 weights.  Separate kernels pay a launch gap and a
// cold memory ramp per phase; here one launch covers the whole step, and each
// workgroup's weight share for a phase is already in LDS when that phase's
// input arrives.
//
// Layout: one 512-thread workgroup per CU (256).  Waves 0-6 compute; wave 7 only
// moves weights: it copies each phase's share of a weight matrix into LDS with
// direct global->LDS loads one or two phases ahead (none while attention runs:
// the FC1 share goes out once every attention partial is done).  A wave's vector loads
// retire in issue order, so keeping the weight stream in a wave of its own is
// what lets the compute waves' polls, parameter loads and KV page loads return
// without waiting behind it.  The copy wave takes part in every workgroup
// barrier (it learns the outcome of each poll round from LDS) and, before the
// barrier that releases a phase's dot products, waits with an explicit vmcnt for
// the share that phase needs, leaving the next share in flight.
// Workgroup barriers are bare s_barrier (plus an LDS wait), never __syncthreads,
// whose memory fence would wait for every outstanding load of the wave.
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
// then LN_f + LM head rows (<= 40 per group) and, for greedy decoding, the
// argmax over all groups' candidates.
#include "gemv_impl.hpp"
#include "kv_page.hpp"

namespace ftts {
namespace mega {

constexpr int NT = 512;                    // threads per workgroup (8 waves)
constexpr int NC = 448;                    // compute threads (waves 0-6)
constexpr int NWC = NC / 64;               // compute waves
constexpr int DW = NWC;                    // the copy wave
constexpr unsigned kSpinLimit = 1u << 19;  // about a second of polling
constexpr int kBuf = 51200;                // one LDS weight buffer: 20 x 1280 or 5 x 5120 bf16
constexpr int kHeadRowsMax = 2 * kBuf / (2 * D);  // LM-head rows a group holds (both buffers)

template <int WT> struct Tiles;  // (lanes per row, 16-byte chunks per lane) per phase, <= NC threads
template <> struct Tiles<FTTS_BF16> {
    static constexpr int QL = 16, QC = 10, OL = 32, OC = 5, AL = 16, AC = 10, BL = 64, BC = 10;
};
template <> struct Tiles<FTTS_W8A16> {
    static constexpr int QL = 16, QC = 5, OL = 16, OC = 5, AL = 16, AC = 5, BL = 64, BC = 5;
};
template <> struct Tiles<FTTS_W4A16> {  // 4-byte chunks (8 codes): many more lanes per row than 16-byte ones
    static constexpr int QL = 16, QC = 10, OL = 32, OC = 5, AL = 16, AC = 10, BL = 64, BC = 10;
};
constexpr int HL = 8, HC = 20;  // LM head (bf16)

template <int WT, int K>
constexpr int row_bytes() { return WT == FTTS_W4A16 ? K / 2 : WT == FTTS_W8A16 ? K : 2 * K; }
// Direct-to-LDS instructions the copy wave issues for `bytes` (1 KB each).
constexpr int dma_ops(int bytes) { return (bytes + 1023) / 1024; }
template <int WT> struct Ops {  // per share, fixed by the shape: rows per group = 15, 5, 20, 5
    static constexpr int PQ = dma_ops(3 * D / G * row_bytes<WT, D>());
    static constexpr int PO = dma_ops(D / G * row_bytes<WT, D>());
    static constexpr int P1 = dma_ops(FF / G * row_bytes<WT, D>());
    static constexpr int P2 = dma_ops(D / G * row_bytes<WT, FF>());
    static_assert(PQ <= 63 && PO <= 63 && P1 <= 63 && P2 <= 63, "vmcnt holds 63");
    static_assert(3 * D / G * row_bytes<WT, D>() <= kBuf && FF / G * row_bytes<WT, D>() <= kBuf &&
                      D / G * row_bytes<WT, FF>() <= kBuf, "share exceeds an LDS buffer");
};
static_assert(3 * D % G == 0 && D % G == 0 && FF % G == 0, "rows split evenly over the groups");
static_assert(D + NH * kMaxSplit * kPartWords <= FF, "merged o and the attention partials share s_in");
static_assert(BM * NH * kMaxSplit <= G, "attention groups fit the grid");
static_assert(BM * NH * kMaxSplit <= kDoneStride && kDoneReplicas + 2 <= 64, "done-word layout");

// Optional phase timeline (built only with FTTS_MEGA_TRACE): thread 0 of each
// group stamps the 100 MHz wall clock at fixed points of every layer.
constexpr int kMarksPerLayer = 20, kMarkSlots = 1 + 50 * kMarksPerLayer + 8;
#ifdef FTTS_MEGA_TRACE
__device__ unsigned long long g_mega_marks[G][2][kMarkSlots];  // [group][compute wave 0 | copy wave]
#define MEGA_MARK(slot)                                                                                   \
    do {                                                                                                  \
        if ((threadIdx.x & 63) == 0 && threadIdx.x / 64 % 7 == 0)                                          \
            g_mega_marks[blockIdx.x][threadIdx.x / (64 * 7)][(slot)] = wall_clock64();                     \
    } while (0)
#else
#define MEGA_MARK(slot) ((void)0)
#endif
#define MEGA_LMARK(l, e) MEGA_MARK(1 + (l) * kMarksPerLayer + (e))

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

// threadIdx.x as a value the compiler cannot prove loop-invariant: addresses
// derived from it are formed where they are used instead of being hoisted out
// of the layer loop and held in registers for the whole step.
__device__ __forceinline__ int fresh_tid() {
    int t = threadIdx.x;
    asm volatile("" : "+v"(t));
    return t;
}

// Workgroup barrier that waits only for the wave's own LDS traffic.
__device__ __forceinline__ void bar() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }
// Wait until at most N of the wave's vector memory operations are outstanding.
template <int N>
__device__ __forceinline__ void wait_vm() {
    static_assert(N >= 0 && N <= 63, "vmcnt range");
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

typedef __attribute__((address_space(3))) char lds_char;

// Copy wave: rows [r0, r0 + nrows) of a row-major matrix (row_b bytes a row,
// 16-byte aligned) into LDS, 1 KB per instruction.  Lanes past the end repeat
// the last 16 bytes, so up to 1 KB - 16 bytes past the share are written.
__device__ __forceinline__ void dma_rows(const void* W, int row_b, int r0, int nrows, char* dst) {
    const int lane = threadIdx.x & 63;
    const int n = nrows * row_b >> 4;
    const char* s = reinterpret_cast<const char*>(W) + (size_t)r0 * row_b;
    lds_char* d = (lds_char*)(dst);
    for (int c0 = 0; c0 < n; c0 += 64) {
        const int c = min(c0 + lane, n - 1);
        // cache policy 2 = nt: weights are read once per step, and streaming them
        // non-temporally keeps them from evicting the exchange words being polled
        __builtin_amdgcn_global_load_lds(s + (size_t)c * 16, d + c0 * 16, 16, 0, 2);
    }
}

// Workgroup agreement on a failed wait: a flag in LDS, set by any wave that
// gave up, read by every wave after the barrier that ends each gather.  A wave
// that gives up also raises the device-wide abort word and marks every row of
// the step as failed (sampled id -1, row inactive, so the sampler that may
// follow writes -1 too): a generation loop stops instead of reusing stale ids.
struct Sync {
    int* fail;
    int32_t* sampled;
    int32_t* active_out;
    int B;
};
__device__ __forceinline__ void give_up(const Sync& sy, uint32_t* ctl) {
    *sy.fail = 1;
    __hip_atomic_store(ctl + 1, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    for (int b = 0; b < sy.B; ++b) {
        sy.sampled[b] = -1;
        sy.active_out[b] = 0;
    }
}

// Compute waves: wait until the n exchange words all carry `epoch` and leave their
// values in dst (LDS); idx(j) maps value j to its word.  Each wave polls its own
// words (device-scope relaxed atomic loads) with two rounds in flight -- the next
// round goes out before the previous one is checked, re-reading only words not
// yet seen -- so a word is picked up about half a round trip after it lands
// rather than up to a full one.  The workgroup then meets at one barrier.
// Returns false when a wave's wait ran out or another group gave up.
//
// With sentinels (sent.n > 0, at most 64), wave 0 first polls only those
// consecutive words (one per producer, stored after its data; each group reads
// the replica of its own index mod kDoneReplicas, so that the many waiting groups
// do not all hammer the same few lines), the workgroup meets at a barrier, and
// then every wave reads its share of the full set.  A group that waits through a
// long phase thus sends one small request per round instead of many.
struct NoSentinels {
    static constexpr int n = 0;
    const uint64_t* w = nullptr;
};
struct Sentinels {
    const uint64_t* w;  // n consecutive words
    int n;
};
template <int U, typename Idx, typename Sent = NoSentinels>
__device__ __forceinline__ bool gather(const uint64_t* src, int n, Idx idx, uint32_t epoch, float* dst, uint32_t* ctl,
                                       Sync& sy, Sent sent = Sent{}, int mark = -1) {
    const int tid = fresh_tid();
    bool failed = false;
    if (sent.n > 0) {
        if (tid < 64) {
            const uint64_t* w = sent.w + min(tid, sent.n - 1);
            unsigned spins = 0;
            uint64_t a0 = __hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            while (true) {
                const uint32_t ab = ld_agent(ctl + 1);
                const uint64_t a1 = __hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                if (__all((uint32_t)(a0 >> 32) == epoch)) break;
                if (++spins > kSpinLimit || ab != 0) {
                    failed = true;
                    break;
                }
                a0 = __hip_atomic_load(w, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                if (__all((uint32_t)(a1 >> 32) == epoch)) break;
            }
            if (failed && tid == 0) give_up(sy, ctl);
        }
        bar();
        failed = *sy.fail != 0;
    }
    for (int base = 0; base < n && !failed; base += NC * U) {
        uint64_t va[U], vb[U];
        bool seen[U];
#pragma unroll
        for (int u = 0; u < U; ++u) seen[u] = false;
        // Every round reads all U words, so the compiler can wait for one round
        // while the next is in flight (loads retire in order).
        auto issue = [&](uint64_t (&v)[U]) {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int j = min(base + tid + NC * u, n - 1);
                v[u] = __hip_atomic_load(src + idx(j), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
        };
        auto take = [&](const uint64_t (&v)[U]) {  // record newly arrived words; true when all have
            bool all = true;
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if (!seen[u] && (uint32_t)(v[u] >> 32) == epoch) {
                    seen[u] = true;
                    const int j = base + tid + NC * u;
                    if (j < n) dst[j] = __uint_as_float((uint32_t)v[u]);
                }
                all = all && seen[u];
            }
            return __all(all);
        };
        unsigned spins = 0;
        issue(va);
        while (true) {
            const uint32_t ab = ld_agent(ctl + 1);  // abort word, older than the round issued next
            issue(vb);
            if (take(va)) break;
            if (++spins > kSpinLimit || ab != 0) {
                failed = true;
                break;
            }
            issue(va);
            if (take(vb)) break;
        }
    }
    if (mark >= 0) MEGA_MARK(mark + 1);
    if (failed && (tid & 63) == 0) give_up(sy, ctl);
    bar();
    return *sy.fail == 0;
}
struct Flat {
    __device__ int operator()(int j) const { return j; }
};

// Copy wave: the barrier that ends a gather.
__device__ __forceinline__ bool follow(Sync& sy) {
    bar();
    return *sy.fail == 0;
}

// One phase's share of a weight matrix: rows [r0, r0 + R) in an LDS buffer
// (copied there by the copy wave); per-row bias and quantisation parameters of
// this thread's row in registers.
// W4A16 dot of one 4-byte chunk (8 codes, columns 8c .. 8c+7, one quantisation
// group): the zero-point enters through the chunk's own activation sum.
template <int B_>
__device__ __forceinline__ void dot_w4_word(uint32_t word, const float* xs, int stride, int B, float (&acc)[B_],
                                            float s4, float z4) {
    float wf[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) wf[i] = (float)((word >> (4 * i)) & 0xFu);
#pragma unroll
    for (int b = 0; b < B_; ++b) {
        if (b < B) {
            const float4 x0 = *reinterpret_cast<const float4*>(xs + b * stride);
            const float4 x1 = *reinterpret_cast<const float4*>(xs + b * stride + 4);
            float t = 0.f;
            t = fmaf(wf[0], x0.x, t);
            t = fmaf(wf[1], x0.y, t);
            t = fmaf(wf[2], x0.z, t);
            t = fmaf(wf[3], x0.w, t);
            t = fmaf(wf[4], x1.x, t);
            t = fmaf(wf[5], x1.y, t);
            t = fmaf(wf[6], x1.z, t);
            t = fmaf(wf[7], x1.w, t);
            const float sx = ((x0.x + x0.y) + (x0.z + x0.w)) + ((x1.x + x1.y) + (x1.z + x1.w));
            acc[b] = fmaf(s4, fmaf(-z4, sx, t), acc[b]);
        }
    }
}

template <int WT, int LPR, int NCH, int K>
struct Share {
    static constexpr int ROW_BYTES = row_bytes<WT, K>();
    // bytes per chunk: 16 (one uint4) for 16-bit and int8 weights, 4 (8 codes) for W4A16
    static constexpr int CB = WT == FTTS_W4A16 ? 4 : 16;
    static constexpr int EPC = WT == FTTS_W4A16 ? 8 : WInfo<WT>::EPC;  // weights per chunk
    static_assert(LPR * NCH * CB == ROW_BYTES, "tiling must cover a row");
    static_assert(WT != FTTS_W4A16 || NCH * EPC <= 128, "a W4A16 lane must stay within two groups");
    float s4[2], z4[2];
    float rs, bias;
    int R;
    const char* buf;
    __device__ __forceinline__ void params(const void* S, const void* Z, const void* bias_p, int r0, int nrows,
                                           const char* lds) {
        const int li = threadIdx.x & (LPR - 1);
        const int row = r0 + min((int)threadIdx.x / LPR, nrows - 1);
        R = nrows;
        buf = lds;
        bias = bf16_to_f32(reinterpret_cast<const uint16_t*>(bias_p)[row]);
        rs = 1.f;
        if constexpr (WT == FTTS_W8A16) rs = bf16_to_f32(reinterpret_cast<const uint16_t*>(S)[row]);
        // W4A16: a lane takes NCH consecutive 4-byte chunks (at most 128 columns), so
        // it meets at most two quantisation groups: g0 and g0 + 1.
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            s4[i] = 0.f;
            z4[i] = 0.f;
            if constexpr (WT == FTTS_W4A16) {
                const int g = min(((li * NCH * EPC) >> 7) + i, K / 128 - 1);
                s4[i] = bf16_to_f32(reinterpret_cast<const uint16_t*>(S)[(size_t)row * (K / 128) + g]);
                z4[i] = bf16_to_f32(reinterpret_cast<const uint16_t*>(Z)[(size_t)row * (K / 128) + g]);
            }
        }
    }
    // acc[b] = dot product of this thread's row with s_in[b] (+ bias); every lane of the row gets it.
    template <int B_>
    __device__ __forceinline__ void dot(const float* s_in, int B, float (&acc)[B_]) const {
        const int t = fresh_tid();
        const int li = t & (LPR - 1);
        const int slot = min(t / LPR, R - 1);
#pragma unroll
        for (int b = 0; b < B_; ++b) acc[b] = 0.f;
        if constexpr (WT == FTTS_W4A16) {
            const uint32_t* wrow = reinterpret_cast<const uint32_t*>(buf + slot * ROW_BYTES);
            const int g0 = (li * NCH * EPC) >> 7;
#pragma unroll
            for (int i = 0; i < NCH; ++i) {
                const int c = li * NCH + i;
                const bool second = ((c * EPC) >> 7) != g0;
                dot_w4_word<B_>(wrow[c], s_in + c * EPC, K, B, acc, second ? s4[1] : s4[0], second ? z4[1] : z4[0]);
            }
        } else {
            const uint4* wrow = reinterpret_cast<const uint4*>(buf + slot * ROW_BYTES);
#pragma unroll
            for (int i = 0; i < NCH; ++i) {
                const int c = li + i * LPR;
                dot_chunk<WT, B_>(wrow[c], s_in + c * EPC, K, B, acc, 0.f, 0.f, nullptr, 0);
            }
        }
#pragma unroll
        for (int b = 0; b < B_; ++b) acc[b] = fmaf(group_sum<LPR>(acc[b]), rs, bias);
    }
};

// LayerNorm gains of columns 4t .. 4t+3 (thread t < 320), packed bf16.
struct LnCols {
    uint2 g, b;
    __device__ __forceinline__ void load(const void* gp, const void* bp) {
        const int c = min((int)threadIdx.x, D / 4 - 1);
        g = reinterpret_cast<const uint2*>(gp)[c];
        b = reinterpret_cast<const uint2*>(bp)[c];
    }
};

// LayerNorm of the B rows of s_x into s_in.  Thread t < 320 (waves 0-4) normalises columns
// 4t .. 4t+3 of every row, so consecutive lanes touch consecutive LDS words;
// each of those waves forms every row's mean and variance itself, so no
// barrier is needed until the result is complete.
template <int BMAX>
__device__ __forceinline__ void layer_norm(const float* s_x, float* s_in, const LnCols& ln, float eps, int B) {
    const int tid = fresh_tid(), lane = tid & 63;
    if (tid >= D / 4) return;  // whole waves
#pragma unroll
    for (int b = 0; b < BMAX; ++b) {
        if (b < B) {
            const float* x = s_x + b * D;
            float4 xv[D / 256];
            float s = 0.f;
#pragma unroll
            for (int i = 0; i < D / 256; ++i) {
                xv[i] = *reinterpret_cast<const float4*>(x + i * 256 + lane * 4);
                s += (xv[i].x + xv[i].y) + (xv[i].z + xv[i].w);
            }
            const float m = wave_sum(s) * (1.0f / (float)D);
            float q = 0.f;
#pragma unroll
            for (int i = 0; i < D / 256; ++i) {
                const float d0 = xv[i].x - m, d1 = xv[i].y - m, d2 = xv[i].z - m, d3 = xv[i].w - m;
                q = fmaf(d0, d0, q);
                q = fmaf(d1, d1, q);
                q = fmaf(d2, d2, q);
                q = fmaf(d3, d3, q);
            }
            const float r = 1.0f / sqrtf(wave_sum(q) * (1.0f / (float)D) + eps);
            const float4 v = *reinterpret_cast<const float4*>(x + tid * 4);
            float4 y;
            y.x = fmaf((v.x - m) * r, bf16lo(ln.g.x), bf16lo(ln.b.x));
            y.y = fmaf((v.y - m) * r, bf16hi(ln.g.x), bf16hi(ln.b.x));
            y.z = fmaf((v.z - m) * r, bf16lo(ln.g.y), bf16lo(ln.b.y));
            y.w = fmaf((v.w - m) * r, bf16hi(ln.g.y), bf16hi(ln.b.y));
            *reinterpret_cast<float4*>(s_in + b * D + tid * 4) = y;
        }
    }
}


// Online-softmax update of one wave's (m, lsum, o) with one 64-token page of
// keys and values (page p of the sequence).  Slots at or past ncache, or of an
// invalid page, may hold anything (NaN included): their scores are replaced by
// -inf (a select, so a NaN key never reaches the max) and, on a page that has
// such slots, their values are zeroed first, so 0 * value stays 0.
__device__ __forceinline__ void attend_page(PageRegs<false>& pg, bool ok, int p, int ncache, const float (&q)[8],
                                            int grp, float& m, float& lsum, float (&o)[8]) {
    if (!(ok && (p + 1) * kPage <= ncache)) {
#pragma unroll
        for (int i = 0; i < 8; ++i)
            if (!(ok && p * kPage + i * 8 + grp < ncache)) pg.v[i] = make_uint4(0u, 0u, 0u, 0u);
    }
    float sc[8];
    float pm = -INFINITY;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        float kv[8];
        unpack8<false>(pg, false, i, kv);
        float t = 0.f;
#pragma unroll
        for (int d = 0; d < 8; ++d) t = fmaf(q[d], kv[d], t);
        t = group_sum<8>(t);
        sc[i] = (ok && p * kPage + i * 8 + grp < ncache) ? t : -INFINITY;
        pm = fmaxf(pm, sc[i]);
    }
    pm = stride8_max(pm);
    if (pm > -INFINITY) {
        const float mn = fmaxf(m, pm);
        const float alpha = __expf(m - mn);
        m = mn;
        lsum *= alpha;
#pragma unroll
        for (int d = 0; d < 8; ++d) o[d] *= alpha;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            float vv[8];
            unpack8<false>(pg, true, i, vv);
            const float pr = __expf(sc[i] - m);  // 0 for a left-out slot
            lsum += pr;
#pragma unroll
            for (int d = 0; d < 8; ++d) o[d] = fmaf(pr, vv[d], o[d]);
        }
    }
}

template <int BMAX> constexpr int ux() { return (BMAX * D + NC - 1) / NC; }           // words per thread: x, o
template <int BMAX> constexpr int uh() { return (BMAX * FF + NC - 1) / NC < 12 ? (BMAX * FF + NC - 1) / NC : 12; }  // h
template <int BMAX> constexpr int uo() {  // attention partials, S <= kMaxSplit
    return (BMAX * NH * kMaxSplit * kPartWords + NC - 1) / NC;
}
template <int BMAX> constexpr int ua() { return (G * BMAX * 2 + NC - 1) / NC; }        // argmax candidates

// The copy wave's program: every share copy, and the barriers of the compute
// waves' program in the same order.
template <int WT, int BMAX>
__device__ __forceinline__ void copy_wave(const Args& a, char* s_w, Sync& sy) {
    using O = Ops<WT>;
    const int wg = blockIdx.x, B = a.B;
    const int q0 = 3 * D / G * wg, d0 = D / G * wg, f0 = FF / G * wg;
    const int v0 = a.V * wg / G, nv = a.V * (wg + 1) / G - v0;
    const int nA = min(nv, kBuf / (2 * D));
    const bool is_att = wg < B * NH * a.att_split;
    constexpr int RD = row_bytes<WT, D>(), RF = row_bytes<WT, FF>();

    dma_rows(a.qkv_w.at(0), RD, q0, 3 * D / G, s_w);
    for (int l = 0; l < a.n_layer; ++l) {
        // P0
        bar();
        MEGA_LMARK(l, 0);
        if (l == 0) bar();
        else if (!follow(sy)) goto out;
        dma_rows(a.out_w.at(l), RD, d0, D / G, s_w + kBuf);
        wait_vm<O::PO>();  // q/k/v share in LDS
        MEGA_LMARK(l, 1);
        bar();             // LN1 done
        // P1
        bar();
        MEGA_LMARK(l, 2);
        if (!is_att) dma_rows(a.fc1_w.at(l), RD, f0, FF / G, s_w);
        if (is_att) {
            if (!follow(sy)) goto out;
            bar();  // wave partials in LDS
        }
        // P2
        if (is_att) wait_vm<0>(); else wait_vm<O::P1>();  // out-proj share in LDS
        MEGA_LMARK(l, 3);
        if (!follow(sy)) goto out;
        if (is_att) dma_rows(a.fc1_w.at(l), RD, f0, FF / G, s_w);
        // P3
        bar();
        MEGA_LMARK(l, 4);
        if (!follow(sy)) goto out;
        dma_rows(a.fc2_w.at(l), RF, d0, D / G, s_w + kBuf);
        wait_vm<O::P2>();  // FC1 share in LDS
        MEGA_LMARK(l, 5);
        bar();             // LN2 done
        // P4
        bar();
        MEGA_LMARK(l, 6);
        wait_vm<0>();  // FC2 share in LDS
        MEGA_LMARK(l, 7);
        if (!follow(sy)) goto out;
        if (l + 1 < a.n_layer) dma_rows(a.qkv_w.at(l + 1), RD, q0, 3 * D / G, s_w);
        else dma_rows(a.head_w, 2 * D, v0, nA, s_w);
    }
    // head
    bar();
    if (nv > nA) dma_rows(a.head_w, 2 * D, v0 + nA, nv - nA, s_w + kBuf);
    if (!follow(sy)) goto out;
    wait_vm<0>();
    bar();  // LN_f done
    if (a.greedy) {
        bar();  // candidates in LDS
        if (wg == 0) follow(sy);
    }
out:
    wait_vm<0>();
}

template <int WT, int BMAX>
__global__ __launch_bounds__(NT) void decode_mega_kernel(const Args a) {
    using T = Tiles<WT>;
    __shared__ __attribute__((aligned(1024))) char s_w[2 * kBuf];     // weight shares, two buffers
    __shared__ __attribute__((aligned(16))) float s_in[BMAX * FF];    // phase input (normalised for LN phases)
    __shared__ __attribute__((aligned(16))) float s_x[BMAX * D];      // residual stream as last gathered
    __shared__ __attribute__((aligned(16))) float s_q[3 * 64];        // attention: q, k, v of the new token
    __shared__ float s_pm[NWC], s_pl[NWC], s_po[NWC][64];             // attention wave partials
    __shared__ float s_cv[BMAX][NC / HL];                             // head: per-slot best value
    __shared__ int s_ci[BMAX][NC / HL];                               //       and its row
    __shared__ int s_active[BMAX], s_tok[BMAX], s_pos[BMAX], s_slot[BMAX], s_phys[BMAX];  // per sequence
    __shared__ int s_fail;
    __shared__ int s_abort;

    const int wg = blockIdx.x, tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int B = a.B;
    const uint32_t step = ld_agent(a.ctl);
    auto E = [&](int ev) { return (step << 8) | (uint32_t)ev; };
    if (tid == 0) {
        s_abort = ld_agent(a.ctl + 1) != 0;
        s_fail = 0;
    }
    __syncthreads();
    if (tid < B) {  // the sequence's token, position and KV slot; inactive rows produce nothing
        const int b = tid;
        const int t = a.tokens[b], p = a.positions[b], s = a.seq_lens[b];
        bool act = t >= 0 && t < a.V && p >= 0 && p < a.n_pos && s >= 0 && s < a.max_pages * kPage;
        int phys = -1;
        if (act) {
            phys = a.block_table[(size_t)b * a.max_pages + s / kPage];
            act = phys >= 0 && phys < a.n_pages;
        }
        // after an earlier step gave up, every step fails at once: no row is
        // active and every sampled id is -1 until a prefill clears the abort word
        if (s_abort) act = false;
        s_active[b] = act;
        s_tok[b] = t;
        s_pos[b] = p;
        s_slot[b] = s;
        s_phys[b] = phys;
        if (wg == 0) {
            a.active_out[b] = act;
            if (s_abort) a.sampled[b] = -1;
        }
    }
    __syncthreads();
    if (s_abort) return;
    Sync sy{&s_fail, a.sampled, a.active_out, B};
    MEGA_MARK(0);
    if (wave == DW) {
        copy_wave<WT, BMAX>(a, s_w, sy);
        return;
    }

    const int q0 = 3 * D / G * wg, q1 = q0 + 3 * D / G;
    const int d0 = D / G * wg, d1 = d0 + D / G;
    const int f0 = FF / G * wg, f1 = f0 + FF / G;
    const int v0 = a.V * wg / G, v1 = a.V * (wg + 1) / G;
    // Attention: S groups per (sequence, head); split s takes the sequence's pages
    // s, s + S, s + 2S, ..., and its wave w every seventh of those from the w-th.
    const int S = a.att_split;
    const bool is_att = wg < B * NH * S;
    const int att_b = wg / (NH * S), att_h = wg / S % NH, att_s = wg % S;

    Share<WT, T::QL, T::QC, D> pq;
    Share<WT, T::OL, T::OC, D> po;
    Share<WT, T::AL, T::AC, D> p1;
    Share<WT, T::BL, T::BC, FF> p2;
    const int sq = tid / T::QL, so = tid / T::OL, s1 = tid / T::AL, s2 = tid / T::BL, sh = tid / HL;
    LnCols ln;
    pq.params(a.qkv_s.at(0), a.qkv_z.at(0), a.qkv_b.at(0), q0, q1 - q0, s_w);
    // Attention groups: the sequence's cached slots (the new token excluded) are
    // the same in every layer; this wave's pages are wave, wave + 7, ... and lane
    // j holds the physical id of its j-th (and j+64-th) one.
    int ncache = 0, my_pages = 0, my_phys0 = -1, my_phys1 = -1;
    if (is_att && s_active[att_b]) {
        ncache = s_slot[att_b];
        const int npg = (ncache + kPage - 1) / kPage;
        const int nsplit = npg > att_s ? (npg - att_s + S - 1) / S : 0;  // pages of this split
        const int32_t* bt = a.block_table + (size_t)att_b * a.max_pages;
        const int lp0 = att_s + S * (wave + NWC * lane), lp1 = att_s + S * (wave + NWC * (lane + 64));
        my_phys0 = lp0 < npg ? bt[lp0] : -1;
        my_phys1 = lp1 < npg ? bt[lp1] : -1;
        my_pages = nsplit > wave ? (nsplit - wave + NWC - 1) / NWC : 0;
    }

    for (int l = 0; l < a.n_layer; ++l) {
        // ---------------- P0: LN1 + q/k/v -------------------------------------------------
        bar();  // P4's reads of s_w[1], s_in and s_x are done
        MEGA_LMARK(l, 0);
        ln.load(a.ln1_g.at(l), a.ln1_b.at(l));
        po.params(a.out_s.at(l), a.out_z.at(l), a.out_b.at(l), d0, d1 - d0, s_w + kBuf);
        if (l == 0) {  // the embedding, computed locally by every group
            for (int b = 0; b < B; ++b) {
                const bool act = s_active[b];
                const int t = s_tok[b], p = s_pos[b];
                for (int k = tid; k < D; k += NC)
                    s_x[b * D + k] = act ? ld_act<false>(a.tok_emb, (size_t)t * D + k) +
                                               ld_act<false>(a.pos_emb, (size_t)p * D + k)
                                         : 0.f;
            }
            bar();
        } else if (!gather<ux<BMAX>()>(a.ex_x, B * D, Flat{}, E(5 * l), s_x, a.ctl, sy)) {
            return;
        }
        MEGA_LMARK(l, 1);
        layer_norm<BMAX>(s_x, s_in, ln, a.eps, B);
        MEGA_LMARK(l, 13);
        bar();  // s_in complete; the copy wave has waited for the q/k/v share
        MEGA_LMARK(l, 2);
        {
            float acc[BMAX];
            pq.template dot<BMAX>(s_in, B, acc);
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
                            st_act<false>(a.kv,
                                          kv_offset(l, a.n_pages, s_phys[b], kvsel, NH, r / 64, s_slot[b] % kPage) +
                                              r % 64,
                                          acc[b]);
                        }
                    }
                }
            }
        }
        // ---------------- P1: attention, one group per (sequence, head) ---------------------
        bar();  // P0's reads of s_w[0] are done
        MEGA_LMARK(l, 3);
        p1.params(a.fc1_s.at(l), a.fc1_z.at(l), a.fc1_b.at(l), f0, f1 - f0, s_w);
        if (is_att) {
            const int b = att_b, h = att_h;
            const int grp = lane >> 3, sub = lane & 7;
            auto bases = [&](int j, size_t& kb, size_t& vb) {
                int phys = j < 64 ? __builtin_amdgcn_readlane(my_phys0, j & 63)
                                  : __builtin_amdgcn_readlane(my_phys1, j & 63);
                const bool ok = phys >= 0 && phys < a.n_pages;
                phys = ok ? phys : 0;
                kb = kv_offset(l, a.n_pages, phys, 0, NH, h, 0);
                vb = kv_offset(l, a.n_pages, phys, 1, NH, h, 0);
                return ok;
            };
            PageRegs<false> cur;
            bool ok_cur = false;
            size_t kb, vb;
            // the first page goes out before the new token's q/k/v arrive
            if (my_pages > 0) {
                ok_cur = bases(0, kb, vb);
                load_page<false>(a.kv, kb, vb, lane, cur);
            }
            const uint64_t* src = a.ex_qkv + (size_t)b * 3 * D + h * 64;
            auto seg = [](int j) { return (j >> 6) * D + (j & 63); };  // q, k, v of head h
            if (!gather<1>(src, 3 * 64, seg, E(5 * l + 1), s_q, a.ctl, sy)) return;
            MEGA_LMARK(l, 4);
            float q[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) q[j] = s_q[sub * 8 + j] * 0.125f;  // 1/sqrt(64), exact
            // The cache holds keys and values in bf16; attend to the new token as cached.
            auto cached = [](float v) { return bf16_to_f32(f32_to_bf16(v)); };
            float m = -INFINITY, lsum = 0.f, o[8];
#pragma unroll
            for (int j = 0; j < 8; ++j) o[j] = 0.f;
            if (att_s == 0 && wave == 0 && s_active[b]) {  // the new token itself, straight from the exchange
                float t = 0.f;
#pragma unroll
                for (int j = 0; j < 8; ++j) t = fmaf(q[j], cached(s_q[64 + sub * 8 + j]), t);
                m = group_sum<8>(t);
                if (grp == 0) {
                    lsum = 1.f;
#pragma unroll
                    for (int j = 0; j < 8; ++j) o[j] = cached(s_q[128 + sub * 8 + j]);
                }
            }
            MEGA_LMARK(l, 14);
            for (int j = 0; j < my_pages; ++j) {
                const int p = att_s + S * (wave + NWC * j);
                if (j > 0) {
                    ok_cur = bases(j, kb, vb);
                    load_page<false>(a.kv, kb, vb, lane, cur);
                }
                attend_page(cur, ok_cur, p, ncache, q, grp, m, lsum, o);
            }
            MEGA_LMARK(l, 15);
#pragma unroll
            for (int d = 0; d < 8; ++d) o[d] = stride8_sum(o[d]);
            lsum = stride8_sum(lsum);
            if (lane < 8) {
#pragma unroll
                for (int d = 0; d < 8; ++d) s_po[wave][lane * 8 + d] = o[d];
            }
            if (lane == 0) {
                s_pm[wave] = m;
                s_pl[wave] = lsum;
            }
            MEGA_LMARK(l, 16);
            bar();
            MEGA_LMARK(l, 5);
            if (wave == 0) {  // log-sum-exp merge of the wave partials: the head's output, normalised
                float M = -INFINITY;
#pragma unroll
                for (int i = 0; i < NWC; ++i) M = fmaxf(M, s_pm[i]);
                float L = 0.f, acc = 0.f;
#pragma unroll
                for (int i = 0; i < NWC; ++i) {
                    if (s_pm[i] > -INFINITY) {
                        const float wgt = expf(s_pm[i] - M);
                        L = fmaf(s_pl[i], wgt, L);
                        acc = fmaf(s_po[i][lane], wgt, acc);
                    }
                }
                put(a.ex_o + (size_t)b * D + h * 64 + lane, E(5 * l + 2), (s_active[b] && L > 0.f) ? acc / L : 0.f);
            }
        }
        // ---------------- P2: out-proj + residual --------------------------------------------
        // o of every head, straight from the attention groups (s_in was last read
        // by P0's dot, before P1's barrier)
        if (!gather<ux<BMAX>()>(a.ex_o, B * D, Flat{}, E(5 * l + 2), s_in, a.ctl, sy)) return;
        MEGA_LMARK(l, 6);
        {
            float acc[BMAX];
            po.template dot<BMAX>(s_in, B, acc);
            const int row = d0 + so;
            const int li = tid & (T::OL - 1);
            if (so < d1 - d0) {
#pragma unroll
                for (int b = 0; b < BMAX; ++b)
                    if (b < B && li == b) put(a.ex_x + (size_t)b * D + row, E(5 * l + 3), s_x[b * D + row] + acc[b]);
            }
        }
        // ---------------- P3: LN2 + FC1 + GELU -----------------------------------------------
        bar();  // P2's reads of s_in / s_x / s_w[1] are done
        MEGA_LMARK(l, 7);
        ln.load(a.ln2_g.at(l), a.ln2_b.at(l));
        p2.params(a.fc2_s.at(l), a.fc2_z.at(l), a.fc2_b.at(l), d0, d1 - d0, s_w + kBuf);
        if (!gather<ux<BMAX>()>(a.ex_x, B * D, Flat{}, E(5 * l + 3), s_x, a.ctl, sy)) return;
        MEGA_LMARK(l, 8);
        layer_norm<BMAX>(s_x, s_in, ln, a.eps, B);
        bar();  // s_in complete; the copy wave has waited for the FC1 share
        MEGA_LMARK(l, 9);
        {
            float acc[BMAX];
            p1.template dot<BMAX>(s_in, B, acc);
            const int row = f0 + s1;
            const int li = tid & (T::AL - 1);
            if (s1 < f1 - f0) {
#pragma unroll
                for (int b = 0; b < BMAX; ++b)
                    if (b < B && li == b) put(a.ex_h + (size_t)b * FF + row, E(5 * l + 4), gelu_tanh(acc[b]));
            }
        }
        // ---------------- P4: FC2 + residual -------------------------------------------------
        bar();  // P3's reads of s_in / s_w[0] are done
        MEGA_LMARK(l, 10);
        if (l + 1 < a.n_layer)
            pq.params(a.qkv_s.at(l + 1), a.qkv_z.at(l + 1), a.qkv_b.at(l + 1), q0, q1 - q0, s_w);
        if (!gather<uh<BMAX>()>(a.ex_h, B * FF, Flat{}, E(5 * l + 4), s_in, a.ctl, sy)) return;
        MEGA_LMARK(l, 11);
        {
            float acc[BMAX];
            p2.template dot<BMAX>(s_in, B, acc);
            const int row = d0 + s2;
            const int li = tid & (T::BL - 1);
            if (s2 < d1 - d0) {
#pragma unroll
                for (int b = 0; b < BMAX; ++b)
                    if (b < B && li == b) put(a.ex_x + (size_t)b * D + row, E(5 * l + 5), s_x[b * D + row] + acc[b]);
            }
        }
        MEGA_LMARK(l, 12);
    }

    // ---------------- LN_f + LM head (+ greedy argmax) -------------------------------------
    bar();  // the last FC2's reads of s_w[1] / s_in / s_x are done
    Share<FTTS_BF16, HL, HC, D> ph;
    ph.params(nullptr, nullptr, a.head_b, v0, v1 - v0, s_w);
    ln.load(a.lnf_g, a.lnf_b);
    if (!gather<ux<BMAX>()>(a.ex_x, B * D, Flat{}, E(5 * a.n_layer), s_x, a.ctl, sy)) return;
    MEGA_MARK(1 + a.n_layer * kMarksPerLayer);
    layer_norm<BMAX>(s_x, s_in, ln, a.eps, B);
    bar();  // s_in complete; the copy wave has waited for the head share
    MEGA_MARK(2 + a.n_layer * kMarksPerLayer);
    if (a.hidden && wg == 0) {  // the step's last-layer hidden state (every group holds the same rows)
        for (int i = tid; i < B * D / 4; i += NC)
            reinterpret_cast<float4*>(a.hidden)[i] = reinterpret_cast<const float4*>(s_in)[i];
    }
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
    bar();
    if (tid < B) {  // this group's best row for each sequence
        float bv = -INFINITY;
        int bi = 0x7FFFFFFF;
        for (int s = 0; s < NC / HL; ++s) {
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
    if (!gather<ua<BMAX>()>(a.ex_arg, G * B * 2, Flat{}, E(5 * a.n_layer + 1), s_in, a.ctl, sy)) return;
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
    MEGA_MARK(3 + a.n_layer * kMarksPerLayer);
    if (tid == 0) st_agent(a.ctl, step + 1);
}

}  // namespace mega

#ifdef FTTS_MEGA_TRACE
extern "C" int ftts_mega_trace_read(void* host, size_t bytes) {
    if (bytes < sizeof(mega::g_mega_marks)) return -1;
    return hipMemcpyFromSymbol(host, HIP_SYMBOL(mega::g_mega_marks), sizeof(mega::g_mega_marks)) == hipSuccess ? 0 : -1;
}
#endif

// Workgroups of the persistent step that fit one CU at once (the step needs 1:
// its 256 groups must all be resident, one per CU, for the exchanges to end).
int decode_mega_blocks_per_cu(int wdtype, int B) {
    using namespace mega;
    static int cache[3][2] = {{-1, -1}, {-1, -1}, {-1, -1}};
    const int wi = wdtype == FTTS_BF16 ? 0 : wdtype == FTTS_W8A16 ? 1 : wdtype == FTTS_W4A16 ? 2 : -1;
    if (wi < 0) return 0;
    const int bi = B <= 1 ? 0 : 1;
    if (cache[wi][bi] >= 0) return cache[wi][bi];
    int n = 0;
    hipError_t e = hipErrorInvalidValue;
    switch (wi * 2 + bi) {
        case 0: e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, decode_mega_kernel<FTTS_BF16, 1>, NT, 0); break;
        case 1: e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, decode_mega_kernel<FTTS_BF16, BM>, NT, 0); break;
        case 2: e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, decode_mega_kernel<FTTS_W8A16, 1>, NT, 0); break;
        case 3: e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, decode_mega_kernel<FTTS_W8A16, BM>, NT, 0); break;
        case 4: e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, decode_mega_kernel<FTTS_W4A16, 1>, NT, 0); break;
        case 5: e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, decode_mega_kernel<FTTS_W4A16, BM>, NT, 0); break;
    }
    if (e != hipSuccess) {
        (void)hipGetLastError();
        n = 0;
    }
    cache[wi][bi] = n;
    return n;
}

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
