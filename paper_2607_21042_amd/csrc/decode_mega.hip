// Persistent single-launch decode step for the IndexTTS-2 GPT shape
// (d_model 1280, 20 heads of 64, d_ff 5120), batch 1-2, bf16 / W8A16 / W4A16.
//
// Why: at batch 1 one step is about 121 dependent phases (5 per layer plus the
// head) over 0.97 GB of bf16 weights.  Separate kernels pay a launch gap and a
// cold memory ramp per phase; here one launch covers the whole step.
//
// Layout: one 512-thread workgroup per CU (256), in two roles.
//  * Attention groups, one per (sequence, head) (the first B x 20 groups), do
//    only attention: all 8 waves hold the sequence's cached KV pages of the
//    head (one page per wave in registers, one more per wave in LDS), loaded
//    for layer l + 1 as soon as layer l's output is published, so when the new
//    token's q, k, v arrive only arithmetic is left.  Each publishes its head's
//    normalised 64 outputs.
//  * GEMV groups (the other 236, or 216 at batch 2) own every weight row: each
//    takes a contiguous range of the rows of every matrix (16-18 q/k/v rows,
//    5-6 out-projection rows, 21-24 FC1 rows, 5-6 FC2 rows, 34-48 LM-head rows).
//    Waves 0-6 compute; wave 7 only moves weights: it copies each phase's share
//    of a weight matrix into LDS with direct global->LDS loads, a phase or more
//    ahead, at points where no exchange of the group is waiting behind them.
//    A wave's vector loads retire in issue order, so keeping the weight stream
//    in a wave of its own lets the compute waves' polls and parameter loads
//    return without waiting behind it.  The copy wave takes part in every
//    workgroup barrier and, before the barrier that releases a phase's dot
//    products, waits with an explicit vmcnt for the share that phase needs.
// Workgroup barriers are bare s_barrier (plus an LDS wait), never
// __syncthreads, whose memory fence would wait for every outstanding load.
//
// Exchange: every value crossing workgroups travels in a 64-bit word
// (32 value bits | epoch << 32) written and read with device-coherent (sc1)
// accesses; the value bits are one fp32 (residual stream, q/k/v) or two bf16
// (attention and FC1 outputs, which only ever enter a linear as bf16).  A consumer knows its data has arrived when every word carries the
// epoch of the current (step, event); no flags, counters or fences are needed.
// Each phase depends on all producers of the previous one, so a single buffer
// per kind of data is never overwritten before every reader has consumed it.
// Waits are bounded: on timeout a workgroup raises the abort word and every
// workgroup leaves at its next wait (ftts_check_workspace reports it).
//
// Per layer (GEMV groups; activations enter the dot products as bf16):
//   P0  LN1 + q/k/v rows, k/v also appended to the KV pool
//   P1  (attention groups) attention over the cached pages and the new token
//   P2  out-proj rows + residual of the group's own x rows
//   P3  LN2 + FC1 rows + GELU
//   P4  FC2 rows + residual
// then LN_f + LM head rows and, for greedy decoding, the argmax over every
// GEMV group's candidates.
#include "gemv_impl.hpp"
#include "kv_page.hpp"

namespace ftts {
namespace mega {

constexpr int NT = 512;                    // threads per workgroup (8 waves)
constexpr int NC = 448;                    // compute threads of a GEMV group (waves 0-6)
constexpr int NWC = NC / 64;               // compute waves
constexpr int DW = NWC;                    // the copy wave
constexpr int NAW = NT / 64;               // attention waves of an attention group
constexpr unsigned kSpinLimit = 1u << 19;  // about a second of polling
constexpr int kBuf = 61440;                // one LDS weight buffer: 24 x 1280 or 6 x 5120 bf16
constexpr int kPageBytes = 2 * kPage * kHeadDim * 2;  // one page of one head: K then V, bf16
constexpr int kLdsPages = 2 * kBuf / kPageBytes;       // pages an attention group stages in LDS (7)
static_assert(kLdsPages < NAW, "one staged page per wave at most");

// Workgroups per role for a kernel instantiated for batches up to BMAX.
template <int BMAX> struct Roles {
    static constexpr int NA = BMAX * NH;  // attention groups
    static constexpr int NG = G - NA;     // GEMV groups
};
// Rows [r0, r0 + n) of an N-row matrix held by GEMV group k of NG.
__device__ __forceinline__ void rows_of(int N, int k, int NG, int& r0, int& n) {
    r0 = (int)((long long)N * k / NG);
    n = (int)((long long)N * (k + 1) / NG) - r0;
}
constexpr int max_rows(int N, int NG) { return (N + NG - 1) / NG; }
// The same for FC1, in whole pairs of rows: its outputs cross the device two
// bf16 values to an exchange word, so no word straddles two groups.
__device__ __forceinline__ void pair_rows_of(int N, int k, int NG, int& r0, int& n) {
    rows_of(N / 2, k, NG, r0, n);
    r0 *= 2;
    n *= 2;
}
constexpr int max_pair_rows(int N, int NG) { return 2 * max_rows(N / 2, NG); }

// (lanes per row, chunks per lane) of each phase: a chunk is 8 weights in every
// mode (16 bytes of bf16, 8 of int8 codes, 4 of W4A16 codes), so the three share
// one tiling and a lane does the same number of products in each.
template <int WT> struct Tiles {
    static constexpr int QL = 16, QC = 10, OL = 32, OC = 5, AL = 16, AC = 10, BL = 64, BC = 10;
};
constexpr int HL = 8, HC = 20;  // LM head (bf16)

template <int WT, int K>
constexpr int row_bytes() { return WT == FTTS_W4A16 ? K / 2 : WT == FTTS_W8A16 ? K : 2 * K; }
// Direct-to-LDS instructions (1 KB each) that copy `bytes`.
constexpr int dma_ops(int bytes) { return (bytes + 1023) / 1024; }
// Every share of a phase is copied with the same number of instructions (that of
// the largest), so the copy wave's vmcnt waits are compile-time constants.
template <int WT, int BMAX> struct Ops {
    static constexpr int NG = Roles<BMAX>::NG;
    static constexpr int PQ = dma_ops(max_rows(3 * D, NG) * row_bytes<WT, D>());
    static constexpr int PO = dma_ops(max_rows(D, NG) * row_bytes<WT, D>());
    static constexpr int P1 = dma_ops(max_pair_rows(FF, NG) * row_bytes<WT, D>());
    static constexpr int P2 = dma_ops(max_rows(D, NG) * row_bytes<WT, FF>());
    static_assert(PQ <= 63 && PO <= 63 && P1 <= 63 && P2 <= 63, "vmcnt holds 63");
    static_assert(PQ * 1024 <= kBuf && PO * 1024 <= kBuf && P1 * 1024 <= kBuf && P2 * 1024 <= kBuf,
                  "share exceeds an LDS buffer");
    static_assert(max_rows(3 * D, NG) * 16 <= NC && max_pair_rows(FF, NG) * 16 <= NC && max_rows(D, NG) * 64 <= NC,
                  "a phase's rows fit the compute threads");
};
// LDS of a GEMV group's weight shares.  For bf16 weights at batch 1 there are
// three regions -- A: q/k/v then FC1, B: out-projection, C: FC2 -- so every
// share of a layer but q/k/v can be requested while attention runs; otherwise
// FC2 follows the out-projection in B (the quantised shares are small enough
// to go out after a gather without holding up the next barrier for long, and
// measured faster that way).  The LM head takes [0, kBuf) and [kBuf, 2 kBuf)
// once the last layer's shares have been read.
template <int WT, int BMAX> struct Lds {
    using O = Ops<WT, BMAX>;
    static constexpr bool kThree = BMAX == 1 && WT == FTTS_BF16;
    // quantised shares at batch 1 are small enough for four regions: q/k/v, FC1 and
    // the out-projection in [0, kBuf), FC2 in [kBuf, 2 kBuf), so FC1, FC2 and the
    // next layer's q/k/v all go out while attention runs and no copy lands during
    // a dot or a gather
    static constexpr bool kFour = BMAX == 1 && WT != FTTS_BF16;
    static constexpr int kOffD = kFour ? O::PQ * 1024 : 0;  // FC1
    static constexpr int kA = (O::PQ > O::P1 ? O::PQ : O::P1) * 1024;
    static constexpr int kOffB = kThree ? kA : kFour ? kOffD + O::P1 * 1024 : kBuf;
    static constexpr int kEnd = kOffB + (O::PO + O::P2) * 1024;
    static constexpr int kBytes = kThree && kEnd > 2 * kBuf ? kEnd : 2 * kBuf;
    static constexpr int kOffC = kThree ? kBytes - O::P2 * 1024 : kBuf;  // C at the top
    static_assert(!kThree || kOffB + O::PO * 1024 <= kOffC, "regions apart");
    static_assert(!kFour || kOffB + O::PO * 1024 <= kBuf, "the first three regions within one buffer");
    static_assert(!kFour || (O::P1 + O::P2 <= 63 && O::P2 + O::PQ <= 63), "copy waits within vmcnt");
};
constexpr int kHeadRowsPerBuf = kBuf / (2 * D);  // LM-head rows in one buffer
static_assert(BM * NH < G, "attention groups leave GEMV groups");
static_assert(2 * kHeadRowsPerBuf * (G - BM * NH) >= 10240, "LM-head rows of the largest vocabulary fit");

// Optional phase timeline (built only with FTTS_MEGA_TRACE): thread 0 of wave 0
// and of wave 7 stamps the 100 MHz wall clock at fixed points of every layer.
constexpr int kMarksPerLayer = 20, kMarkSlots = 1 + 50 * kMarksPerLayer + 8;
#ifdef FTTS_MEGA_TRACE
__device__ unsigned long long g_mega_marks[G][2][kMarkSlots];  // [group][wave 0 | wave 7]
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

// Two values as bf16 in one exchange word: lo in the low half (the even column).
// Two floats rounded to nearest even into packed bf16 (lo in bits 0-15): one
// gfx950 conversion instruction, the same bits as f32_to_bf16 for finite values.
typedef __bf16 bf16x2_cvt_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
    const bf16x2_cvt_t v = {(__bf16)lo, (__bf16)hi};
    return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ void put2(uint64_t* p, uint32_t epoch, float lo, float hi) {
    const uint32_t v = pack_bf16(lo, hi);
    __hip_atomic_store(p, ((uint64_t)epoch << 32) | v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
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
// 16-byte aligned) into LDS with exactly OPS instructions of 1 KB.  Lanes past
// the share repeat its last 16 bytes, so OPS KB are written in all.
template <int OPS>
__device__ __forceinline__ void dma_rows(const void* W, int row_b, int r0, int nrows, char* dst) {
    const int lane = threadIdx.x & 63;
    const int n = nrows * row_b >> 4;
    const char* s = reinterpret_cast<const char*>(W) + (size_t)r0 * row_b;
    lds_char* d = (lds_char*)(dst);
#pragma unroll 2
    for (int i = 0; i < OPS; ++i) {
        const int c = min(i * 64 + lane, n - 1);
        // cache policy 2 = nt: weights are read once per step, and streaming them
        // non-temporally keeps them from evicting the exchange words being polled
        __builtin_amdgcn_global_load_lds(s + (size_t)c * 16, d + i * 1024, 16, 0, 2);
    }
}

// One 8 KB block (one head's keys or values of one page) into LDS.
__device__ __forceinline__ void dma_block(const void* src, char* dst) {
    const int lane = threadIdx.x & 63;
    const char* s = reinterpret_cast<const char*>(src);
    lds_char* d = (lds_char*)(dst);
#pragma unroll
    for (int c0 = 0; c0 < kPage * kHeadDim * 2 / 16; c0 += 64)
        __builtin_amdgcn_global_load_lds(s + (size_t)(c0 + lane) * 16, d + c0 * 16, 16, 0, 0);
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

// A word's 32 value bits into LDS: an fp32 value as is or rounded to bf16, or a
// pair of bf16 values as they were packed.
__device__ __forceinline__ void store_to(float* dst, int j, uint32_t v) { dst[j] = __uint_as_float(v); }
__device__ __forceinline__ void store_to(uint16_t* dst, int j, uint32_t v) { dst[j] = (uint16_t)pack_bf16(__uint_as_float(v), 0.f); }
__device__ __forceinline__ void store_to(uint32_t* dst, int j, uint32_t v) { dst[j] = v; }

// The NTH threads that poll: wait until the n exchange words all carry `epoch`
// and leave their values in dst (LDS, fp32 or rounded to bf16); idx(j) maps value
// j to its word.  Each wave polls its own words (device-scope relaxed atomic
// loads) with two rounds in flight -- the next round goes out before the
// previous one is checked, re-reading only words not yet seen -- so a word is
// picked up about half a round trip after it lands rather than up to a full
// one.  The workgroup then meets at one barrier.  Returns false when a wave's
// wait ran out or another group gave up.
template <int U, int NTH, typename Idx, typename Dst>
__device__ __forceinline__ bool gather(const uint64_t* src, int n, Idx idx, uint32_t epoch, Dst* dst, uint32_t* ctl,
                                       Sync& sy) {
    const int tid = fresh_tid();
    bool failed = false;
    for (int base = 0; base < n && !failed; base += NTH * U) {
        uint64_t va[U], vb[U];
        bool seen[U];
#pragma unroll
        for (int u = 0; u < U; ++u) seen[u] = false;
        // Every round reads all U words, so the compiler can wait for one round
        // while the next is in flight (loads retire in order).
        auto issue = [&](uint64_t (&v)[U]) {
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int j = min(base + tid + NTH * u, n - 1);
                v[u] = __hip_atomic_load(src + idx(j), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
        };
        auto take = [&](const uint64_t (&v)[U]) {  // record newly arrived words; true when all have
            bool all = true;
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if (!seen[u] && (uint32_t)(v[u] >> 32) == epoch) {
                    seen[u] = true;
                    const int j = base + tid + NTH * u;
                    if (j < n) store_to(dst, j, (uint32_t)v[u]);
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

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
// a.x * b.x + a.y * b.y + c over packed bf16 pairs, accumulated in fp32
__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c) {
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a), __builtin_bit_cast(bf16x2_t, b), c,
                                           false);
}

// W4A16 dot of one 4-byte chunk (8 codes, columns 8c .. 8c+7, one quantisation
// group) with 8 bf16 activations per row, already in registers: the zero-point
// enters through the chunk's own activation sum.
template <int B_>
__device__ __forceinline__ void dot_w4_word(uint32_t word, const uint4 (&xv)[B_], float (&acc)[B_], float s4,
                                            float z4) {
    // Codes c0..c7 sit at bits 4i, so c_i and c_{i+4} are 16 bits apart: masking
    // the word shifted by 4i with 0x000F000F and setting 0x4300 in both halves
    // gives the bf16 pair (128 + c_i, 128 + c_{i+4}), exactly.  The products
    // with x are exact too, and the 128 is taken out with the chunk's sum of x.
    uint32_t cp[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) cp[i] = ((word >> (4 * i)) & 0x000F000Fu) | 0x43004300u;
    constexpr uint32_t kOnes = 0x3F803F80u;  // bf16 (1, 1)
#pragma unroll
    for (int b = 0; b < B_; ++b) {
        const uint4 x = xv[b];
        // (x_i, x_{i+4}) pairs from the (x_2j, x_2j+1) pairs in LDS
        const uint32_t x04 = __builtin_amdgcn_perm(x.z, x.x, 0x05040100u);
        const uint32_t x15 = __builtin_amdgcn_perm(x.z, x.x, 0x07060302u);
        const uint32_t x26 = __builtin_amdgcn_perm(x.w, x.y, 0x05040100u);
        const uint32_t x37 = __builtin_amdgcn_perm(x.w, x.y, 0x07060302u);
        float t = dot2_bf16(cp[0], x04, 0.f);
        t = dot2_bf16(cp[1], x15, t);
        t = dot2_bf16(cp[2], x26, t);
        t = dot2_bf16(cp[3], x37, t);
        float sx = dot2_bf16(x.x, kOnes, 0.f);
        sx = dot2_bf16(x.y, kOnes, sx);
        sx = dot2_bf16(x.z, kOnes, sx);
        sx = dot2_bf16(x.w, kOnes, sx);
        acc[b] = fmaf(s4, fmaf(-(128.f + z4), sx, t), acc[b]);
    }
}

// One 16-byte chunk of bf16 weights (8 columns) against the rows' 8 activations, in registers.
template <int B_>
__device__ __forceinline__ void dot_bf16_chunk(const uint4 wv, const uint4 (&xv)[B_], float (&acc)[B_]) {
#pragma unroll
    for (int b = 0; b < B_; ++b) {
        float t = acc[b];
        t = dot2_bf16(wv.x, xv[b].x, t);
        t = dot2_bf16(wv.y, xv[b].y, t);
        t = dot2_bf16(wv.z, xv[b].z, t);
        t = dot2_bf16(wv.w, xv[b].w, t);
        acc[b] = t;
    }
}

// One 8-byte chunk of W8A16 codes (8 int8 weights, columns 8c .. 8c+7) against
// the rows' 8 activations, in registers.  Every int8 code is a bf16 value
// exactly (at most 8 significant bits), so each code becomes fp32 in one
// conversion that selects and sign-extends its byte, two of them are packed as a
// bf16 pair (their upper halves), and the pairs meet the activation pairs in
// fp32-accumulating dot products.
__device__ __forceinline__ uint32_t w8_pair(uint32_t w, int hi) {
    const float a = (float)(int)(signed char)(w >> (16 * hi));
    const float b = (float)(int)(signed char)(w >> (16 * hi + 8));
    return __builtin_amdgcn_perm(__float_as_uint(b), __float_as_uint(a), 0x07060302u);
}
template <int B_>
__device__ __forceinline__ void dot_w8_chunk(const uint2 wv, const uint4 (&xv)[B_], float (&acc)[B_]) {
    const uint32_t wp[4] = {w8_pair(wv.x, 0), w8_pair(wv.x, 1), w8_pair(wv.y, 0), w8_pair(wv.y, 1)};
#pragma unroll
    for (int b = 0; b < B_; ++b) {
        float t = acc[b];
        t = dot2_bf16(wp[0], xv[b].x, t);
        t = dot2_bf16(wp[1], xv[b].y, t);
        t = dot2_bf16(wp[2], xv[b].z, t);
        t = dot2_bf16(wp[3], xv[b].w, t);
        acc[b] = t;
    }
}

template <int WT, int LPR, int NCH, int K>
struct Share {
    static constexpr int ROW_BYTES = row_bytes<WT, K>();
    // a chunk is 8 weights: 16 bytes of bf16, 8 of int8 codes, 4 of W4A16 codes
    static constexpr int CB = WT == FTTS_W4A16 ? 4 : WT == FTTS_W8A16 ? 8 : 16;
    static constexpr int EPC = 8;
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
    // acc[b] = dot product of this thread's row with the bf16 row s_in[b] (+ bias); every lane of the row gets it.
    template <int B_>
    __device__ __forceinline__ void dot(const uint16_t* s_in, int B, float (&acc)[B_]) const {
        (void)B;  // every row slot is computed; callers use the rows below B
        const int t = fresh_tid();
        const int li = t & (LPR - 1);
        const int slot = min(t / LPR, R - 1);
#pragma unroll
        for (int b = 0; b < B_; ++b) acc[b] = 0.f;
        // A wave whose rows all lie past the share's last row has nothing to
        // compute (its threads would re-read row R - 1) and skips the reads: the
        // dots are bound by the LDS bandwidth all waves of the CU share.  Its
        // acc stays 0 and its callers keep rows past R out of every store.
        if (__builtin_amdgcn_readfirstlane(t & ~(kWave - 1)) / LPR >= R) return;
        // Every LDS read of the thread's share (weights and the rows'
        // activations) is issued before the first product, so the reads overlap
        // and the thread waits once, not once per chunk.  Rows past the batch
        // are read and multiplied too (the buffers hold BMAX rows; their sums
        // are never used).
        if constexpr (WT == FTTS_W4A16) {
            const uint32_t* wrow = reinterpret_cast<const uint32_t*>(buf + slot * ROW_BYTES);
            const int g0 = (li * NCH * EPC) >> 7;
            uint32_t wv[NCH];
            uint4 xv[NCH][B_];
#pragma unroll
            for (int i = 0; i < NCH; ++i) {
                const int c = li * NCH + i;
                wv[i] = wrow[c];
#pragma unroll
                for (int b = 0; b < B_; ++b) xv[i][b] = *reinterpret_cast<const uint4*>(s_in + c * EPC + b * K);
            }
#pragma unroll
            for (int i = 0; i < NCH; ++i) {
                const bool second = (((li * NCH + i) * EPC) >> 7) != g0;
                dot_w4_word<B_>(wv[i], xv[i], acc, second ? s4[1] : s4[0], second ? z4[1] : z4[0]);
            }
        } else if constexpr (WT == FTTS_BF16) {
            const uint4* wrow = reinterpret_cast<const uint4*>(buf + slot * ROW_BYTES);
            uint4 wv[NCH], xv[NCH][B_];
#pragma unroll
            for (int i = 0; i < NCH; ++i) {
                const int c = li + i * LPR;
                wv[i] = wrow[c];
#pragma unroll
                for (int b = 0; b < B_; ++b) xv[i][b] = *reinterpret_cast<const uint4*>(s_in + c * EPC + b * K);
            }
#pragma unroll
            for (int i = 0; i < NCH; ++i) dot_bf16_chunk<B_>(wv[i], xv[i], acc);
        } else {  // W8A16
            const uint2* wrow = reinterpret_cast<const uint2*>(buf + slot * ROW_BYTES);
            uint2 wv[NCH];
            uint4 xv[NCH][B_];
#pragma unroll
            for (int i = 0; i < NCH; ++i) {
                const int c = li + i * LPR;
                wv[i] = wrow[c];
#pragma unroll
                for (int b = 0; b < B_; ++b) xv[i][b] = *reinterpret_cast<const uint4*>(s_in + c * EPC + b * K);
            }
#pragma unroll
            for (int i = 0; i < NCH; ++i) dot_w8_chunk<B_>(wv[i], xv[i], acc);
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

// LayerNorm of the B rows of s_x into s_in (bf16, the linears' input; the
// optional hid receives the same rows in fp32).  Thread t < 320 (waves 0-4) normalises columns
// 4t .. 4t+3 of every row, so consecutive lanes touch consecutive LDS words;
// each of those waves forms every row's mean and variance itself, so no
// barrier is needed until the result is complete.
template <int BMAX>
__device__ __forceinline__ void layer_norm(const float* s_x, uint16_t* s_in, const LnCols& ln, float eps, int B,
                                           float* hid = nullptr) {
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
            // this thread's columns 4 tid .. 4 tid + 3 are xv[wave] (tid = 64 wave + lane)
            const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
            float4 v = xv[0];
#pragma unroll
            for (int i = 1; i < D / 256; ++i)
                if (w == i) v = xv[i];
            float4 y;
            y.x = fmaf((v.x - m) * r, bf16lo(ln.g.x), bf16lo(ln.b.x));
            y.y = fmaf((v.y - m) * r, bf16hi(ln.g.x), bf16hi(ln.b.x));
            y.z = fmaf((v.z - m) * r, bf16lo(ln.g.y), bf16lo(ln.b.y));
            y.w = fmaf((v.w - m) * r, bf16hi(ln.g.y), bf16hi(ln.b.y));
            uint2 pk;
            pk.x = pack_bf16(y.x, y.y);
            pk.y = pack_bf16(y.z, y.w);
            *reinterpret_cast<uint2*>(s_in + b * D + tid * 4) = pk;
            if (hid) *reinterpret_cast<float4*>(hid + b * D + tid * 4) = y;  // fp32, before rounding
        }
    }
}


// Online-softmax update of one wave's (m, lsum, o) with one 64-token page of
// keys and values (page p of the sequence).  Slots at or past ncache, or of an
// invalid page, may hold anything (NaN included): their scores are replaced by
// -inf (a select, so a NaN key never reaches the max) and, on a page that has
// such slots, their values are zeroed first, so 0 * value stays 0.
__device__ __forceinline__ void attend_page(PageRegs<false>& pg, bool ok, int p, int ncache, const uint32_t (&qh)[4],
                                            const uint32_t (&ql)[4], int grp, float& m, float& lsum, float (&o)[8]) {
    if (!(ok && (p + 1) * kPage <= ncache)) {
#pragma unroll
        for (int i = 0; i < 8; ++i)
            if (!(ok && p * kPage + i * 8 + grp < ncache)) pg.v[i] = make_uint4(0u, 0u, 0u, 0u);
    }
    float sc[8];
    float pm = -INFINITY;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        // bf16 key pairs against the query's bf16 high and low halves: the
        // products are exact and q = hi + lo to about 2^-17 of its size
        const uint4 kw = pg.k[i];
        float t = dot2_bf16(kw.x, qh[0], 0.f);
        t = dot2_bf16(kw.y, qh[1], t);
        t = dot2_bf16(kw.z, qh[2], t);
        t = dot2_bf16(kw.w, qh[3], t);
        t = dot2_bf16(kw.x, ql[0], t);
        t = dot2_bf16(kw.y, ql[1], t);
        t = dot2_bf16(kw.z, ql[2], t);
        t = dot2_bf16(kw.w, ql[3], t);
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

template <int BMAX> constexpr int ux() { return (BMAX * D + NC - 1) / NC; }           // words per thread: x
template <int BMAX> constexpr int uo() { return (BMAX * D / 2 + NC - 1) / NC; }       // o (bf16 pairs)
template <int BMAX> constexpr int uh() { return (BMAX * FF / 2 + NC - 1) / NC < 12 ? (BMAX * FF / 2 + NC - 1) / NC : 12; }  // h (bf16 pairs)
template <int BMAX> constexpr int ua() { return (G * BMAX * 2 + NC - 1) / NC; }        // argmax candidates

// An attention group: sequence b, head h, all 8 waves.  Wave w attends to the
// sequence's cached pages w, w + 8, w + 16, ...: the first in registers and the
// second (waves 0-6) in an LDS slot, both requested for layer l + 1 as soon as
// layer l's output is out, so a step's attention waits only for the new
// token's q, k, v; further pages (contexts beyond 15 pages) are read in turn.
template <int BMAX>
__device__ __forceinline__ void attention_group(const Args& a, int b, int h, int ncache, bool active, uint32_t step,
                                                char* s_w, float* s_q, float* s_pm, float* s_pl,
                                                float (*s_po)[kHeadDim], Sync& sy) {
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int grp = lane >> 3, sub = lane & 7;
    auto E = [&](int ev) { return (step << 8) | (uint32_t)ev; };
    const int npg = (ncache + kPage - 1) / kPage;
    const int32_t* bt = a.block_table + (size_t)b * a.max_pages;
    // lane j holds the physical id of this wave's j-th page (page wave + 8 j)
    const int lp = wave + NAW * lane;
    const int my_phys = lp < npg ? bt[lp] : -1;
    const int my_pages = npg > wave ? (npg - wave + NAW - 1) / NAW : 0;
    const bool staged = wave < kLdsPages && my_pages > 1;  // this wave's second page comes through LDS
    char* slot = s_w + wave * kPageBytes;
    auto bases = [&](int l, int j, size_t& kb, size_t& vb) {
        int phys = __builtin_amdgcn_readlane(my_phys, j);
        const bool ok = phys >= 0 && phys < a.n_pages;
        phys = ok ? phys : 0;
        kb = kv_offset(l, a.n_pages, phys, 0, NH, h, 0);
        vb = kv_offset(l, a.n_pages, phys, 1, NH, h, 0);
        return ok;
    };
    PageRegs<false> cur;
    bool ok0 = false;
    auto prefetch = [&](int l) {
        size_t kb, vb;
        if (my_pages > 0) {
            ok0 = bases(l, 0, kb, vb);
            load_page<false>(a.kv, kb, vb, lane, cur);
        }
        if (staged) {
            bases(l, 1, kb, vb);
            const uint16_t* kv = reinterpret_cast<const uint16_t*>(a.kv);
            dma_block(kv + kb, slot);
            dma_block(kv + vb, slot + kPageBytes / 2);
        }
    };
    prefetch(0);
    const uint64_t* src = a.ex_qkv + (size_t)b * 3 * D + h * 64;
    auto seg = [](int j) { return (j >> 6) * D + (j & 63); };  // q, k, v of head h
    for (int l = 0; l < a.n_layer; ++l) {
        MEGA_LMARK(l, 0);
        if (!gather<1, NT>(src, 3 * 64, seg, E(5 * l + 1), s_q, a.ctl, sy)) return;
        MEGA_LMARK(l, 1);
        float q[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) q[j] = s_q[sub * 8 + j] * 0.125f;  // 1/sqrt(64), exact
        uint32_t qh[4], ql[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            qh[j] = pack_bf16(q[2 * j], q[2 * j + 1]);
            ql[j] = pack_bf16(q[2 * j] - __uint_as_float(qh[j] << 16), q[2 * j + 1] - __uint_as_float(qh[j] & 0xFFFF0000u));
        }
        // The cache holds keys and values in bf16; attend to the new token as cached.
        auto cached = [](float v) { return __uint_as_float(pack_bf16(v, 0.f) << 16); };
        float m = -INFINITY, lsum = 0.f, o[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) o[j] = 0.f;
        if (wave == 0 && active) {  // the new token itself, straight from the exchange
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
        if (my_pages > 0) attend_page(cur, ok0, wave, ncache, qh, ql, grp, m, lsum, o);
        for (int j = 1; j < my_pages; ++j) {
            size_t kb, vb;
            const bool ok = bases(l, j, kb, vb);
            if (j == 1 && staged) {
                wait_vm<0>();  // this wave's own copy of the page has landed
                const uint4* pg = reinterpret_cast<const uint4*>(slot);
#pragma unroll
                for (int i = 0; i < 8; ++i) cur.k[i] = pg[i * 64 + lane];
#pragma unroll
                for (int i = 0; i < 8; ++i) cur.v[i] = pg[kPageBytes / 32 + i * 64 + lane];
            } else {
                load_page<false>(a.kv, kb, vb, lane, cur);
            }
            attend_page(cur, ok, wave + NAW * j, ncache, qh, ql, grp, m, lsum, o);
        }
        MEGA_LMARK(l, 2);
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
        bar();  // wave partials in LDS; every wave is done with its LDS page
        if (wave == 0) {  // log-sum-exp merge of the wave partials: the head's output, normalised
            float M = -INFINITY;
#pragma unroll
            for (int i = 0; i < NAW; ++i) M = fmaxf(M, s_pm[i]);
            // lane i < 8 forms wave i's weight once; every lane takes the eight from them
            const float mi = s_pm[lane & (NAW - 1)];
            const float wl = mi > -INFINITY ? __expf(mi - M) : 0.f;
            float L = 0.f, acc = 0.f;
#pragma unroll
            for (int i = 0; i < NAW; ++i) {
                const float wgt = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(wl), i));
                L = fmaf(s_pl[i], wgt, L);
                acc = fmaf(s_po[i][lane], wgt, acc);
            }
            const float ov = (active && L > 0.f) ? acc / L : 0.f;
            const float on = __shfl_down(ov, 1, kWave);
            if (!(lane & 1)) put2(a.ex_o + ((size_t)b * D + h * 64 + lane) / 2, E(5 * l + 2), ov, on);
        }
        MEGA_LMARK(l, 3);
        bar();  // the head's output is on its way before any page request of the next layer
        if (l + 1 < a.n_layer) prefetch(l + 1);
    }
    wait_vm<0>();
}

// The copy wave of a GEMV group: every share copy, and the barriers of the
// compute waves' program in the same order.  A share request holds up the
// wave's memory operations behind it (the exchange words' polls and stores of
// the same CU wait for the copies ahead of them, and every group's copies load
// the memory system the exchanges cross), so where a share goes out is a trade
// between holding up a barrier and slowing an exchange.  With three regions:
// q/k/v while x is gathered, the out-projection during LN1, FC1 and FC2
// together while attention runs elsewhere.  With four (quantised, batch 1):
// FC1, FC2 and the next layer's q/k/v together while attention runs.  With two
// (batch 2): FC2 waits for the out-projection's buffer and goes out after x is
// gathered, and q/k/v of the next layer once h is gathered.
template <int WT, int BMAX>
__device__ __forceinline__ void copy_wave(const Args& a, int k, char* s_w, Sync& sy) {
    using O = Ops<WT, BMAX>;
    using L = Lds<WT, BMAX>;
    constexpr int NG = Roles<BMAX>::NG;
    constexpr int RD = row_bytes<WT, D>(), RF = row_bytes<WT, FF>();
    constexpr int HO = dma_ops(kHeadRowsPerBuf * 2 * D);
    int q0, nq, d0, nd, f0, nf, v0, nv;
    rows_of(3 * D, k, NG, q0, nq);
    rows_of(D, k, NG, d0, nd);
    pair_rows_of(FF, k, NG, f0, nf);
    rows_of(a.V, k, NG, v0, nv);
    const int nA = min(nv, kHeadRowsPerBuf);

    dma_rows<O::PQ>(a.qkv_w.at(0), RD, q0, nq, s_w);
    for (int l = 0; l < a.n_layer; ++l) {
        // P0
        bar();
        MEGA_LMARK(l, 0);
        if constexpr (L::kThree) {
            if (l > 0) dma_rows<O::PQ>(a.qkv_w.at(l), RD, q0, nq, s_w);
        }
        if (l == 0) bar();
        else if (!follow(sy)) goto out;  // x gathered
        dma_rows<O::PO>(a.out_w.at(l), RD, d0, nd, s_w + L::kOffB);
        wait_vm<O::PO>();  // q/k/v share in LDS
        MEGA_LMARK(l, 1);
        bar();             // LN1 done
        // P1: the FC1 share (and at batch 1 the FC2 share) go out while attention runs
        bar();             // the q/k/v share has been read
        MEGA_LMARK(l, 2);
        dma_rows<O::P1>(a.fc1_w.at(l), RD, f0, nf, s_w + L::kOffD);
        if constexpr (L::kFour) {
            // FC2 follows at once; the next layer's q/k/v after the out-projection's
            // share has landed, so every wait below is an exact count
            dma_rows<O::P2>(a.fc2_w.at(l), RF, d0, nd, s_w + L::kOffC);
            wait_vm<O::P1 + O::P2>();  // out-proj share in LDS
            if (l + 1 < a.n_layer) dma_rows<O::PQ>(a.qkv_w.at(l + 1), RD, q0, nq, s_w);
        } else {
            wait_vm<O::P1>();  // out-proj share in LDS
            if constexpr (L::kThree) dma_rows<O::P2>(a.fc2_w.at(l), RF, d0, nd, s_w + L::kOffC);
        }
        MEGA_LMARK(l, 3);
        if (!follow(sy)) goto out;  // o of every head gathered
        // P3
        bar();  // the out-proj share has been read
        MEGA_LMARK(l, 4);
        if (!follow(sy)) goto out;  // x gathered
        if constexpr (L::kFour) {
            if (l + 1 < a.n_layer) wait_vm<O::P2 + O::PQ>();  // FC1 share in LDS
            else wait_vm<O::P2>();
        } else {
            if constexpr (!L::kThree) dma_rows<O::P2>(a.fc2_w.at(l), RF, d0, nd, s_w + L::kOffC);
            wait_vm<O::P2>();  // FC1 share in LDS
        }
        MEGA_LMARK(l, 5);
        bar();             // LN2 done
        // P4
        bar();  // the FC1 share has been read
        MEGA_LMARK(l, 6);
        if (L::kFour && l + 1 < a.n_layer) wait_vm<O::PQ>();  // FC2 share in LDS
        else wait_vm<0>();
        MEGA_LMARK(l, 7);
        // after the last layer's FC1 share has been read, [0, kBuf) holds nothing
        // the FC2 phase reads, so the head's first rows go out now
        if (l + 1 == a.n_layer) dma_rows<HO>(a.head_w, 2 * D, v0, nA, s_w);
        if (!follow(sy)) goto out;  // h gathered
        if constexpr (!L::kThree && !L::kFour) {
            if (l + 1 < a.n_layer) dma_rows<O::PQ>(a.qkv_w.at(l + 1), RD, q0, nq, s_w);
        }
    }
    // head
    bar();  // the FC2 share has been read
    if (nv > nA) dma_rows<HO>(a.head_w, 2 * D, v0 + nA, nv - nA, s_w + kBuf);
    if (!follow(sy)) goto out;  // x gathered
    wait_vm<0>();
    bar();  // LN_f done
    if (a.greedy) {
        bar();  // candidates in LDS
        if (k == 0) follow(sy);
    }
out:
    wait_vm<0>();
}

template <int WT, int BMAX>
__global__ __launch_bounds__(NT) void decode_mega_kernel(const Args a) {
    using T = Tiles<WT>;
    constexpr int NA = Roles<BMAX>::NA, NG = Roles<BMAX>::NG;
    using L = Lds<WT, BMAX>;
    __shared__ __attribute__((aligned(1024))) char s_w[L::kBytes];    // weight shares / staged KV pages
    __shared__ __attribute__((aligned(16))) uint16_t s_in[BMAX * FF];  // phase input, bf16 (normalised for LN phases)
    __shared__ __attribute__((aligned(16))) float s_x[BMAX * D];      // residual stream as last gathered
    __shared__ __attribute__((aligned(16))) float s_q[3 * 64];        // attention: q, k, v of the new token
    __shared__ float s_pm[NAW], s_pl[NAW], s_po[NAW][kHeadDim];       // attention wave partials
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
    if (wg < NA) {
        const int b = wg / NH, h = wg % NH;
        const bool act = b < B && s_active[b];
        attention_group<BMAX>(a, b, h, act ? s_slot[b] : 0, act, step, s_w, s_q, s_pm, s_pl, s_po, sy);
        return;
    }
    const int k = wg - NA;  // GEMV group index
    if (wave == DW) {
        copy_wave<WT, BMAX>(a, k, s_w, sy);
        return;
    }

    int q0, nq, d0, nd, f0, nf, v0, nv;
    rows_of(3 * D, k, NG, q0, nq);
    rows_of(D, k, NG, d0, nd);
    pair_rows_of(FF, k, NG, f0, nf);
    rows_of(a.V, k, NG, v0, nv);
    Share<WT, T::QL, T::QC, D> pq;
    Share<WT, T::OL, T::OC, D> po;
    Share<WT, T::AL, T::AC, D> p1;
    Share<WT, T::BL, T::BC, FF> p2;
    const int sq = tid / T::QL, so = tid / T::OL, s1 = tid / T::AL, s2 = tid / T::BL, sh = tid / HL;
    LnCols ln;
    pq.params(a.qkv_s.at(0), a.qkv_z.at(0), a.qkv_b.at(0), q0, nq, s_w);

    for (int l = 0; l < a.n_layer; ++l) {
        // ---------------- P0: LN1 + q/k/v -------------------------------------------------
        bar();  // P4's reads of s_w[1], s_in and s_x are done
        MEGA_LMARK(l, 0);
        ln.load(a.ln1_g.at(l), a.ln1_b.at(l));
        po.params(a.out_s.at(l), a.out_z.at(l), a.out_b.at(l), d0, nd, s_w + L::kOffB);
        if (l == 0) {  // the embedding, computed locally by every group
            for (int b = 0; b < B; ++b) {
                const bool act = s_active[b];
                const int t = s_tok[b], p = s_pos[b];
                for (int c = tid; c < D; c += NC)
                    s_x[b * D + c] = act ? ld_act<false>(a.tok_emb, (size_t)t * D + c) +
                                               ld_act<false>(a.pos_emb, (size_t)p * D + c)
                                         : 0.f;
            }
            bar();
        } else if (!gather<ux<BMAX>(), NC>(a.ex_x, B * D, Flat{}, E(5 * l), s_x, a.ctl, sy)) {
            return;
        }
        MEGA_LMARK(l, 1);
        layer_norm<BMAX>(s_x, s_in, ln, a.eps, B);
        bar();  // s_in complete; the copy wave has waited for the q/k/v share
        MEGA_LMARK(l, 2);
        {
            float acc[BMAX];
            pq.template dot<BMAX>(s_in, B, acc);
            const int row = q0 + sq;
            const int li = tid & (T::QL - 1);
            if (sq < nq) {
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
        // ---------------- P1 + P2: attention elsewhere; out-proj + residual ------------------
        bar();  // P0's reads of s_w[0] are done
        MEGA_LMARK(l, 3);
        p1.params(a.fc1_s.at(l), a.fc1_z.at(l), a.fc1_b.at(l), f0, nf, s_w + L::kOffD);
        // o of every head, straight from the attention groups (s_in was last read by P0's dot)
        if (!gather<uo<BMAX>(), NC>(a.ex_o, B * D / 2, Flat{}, E(5 * l + 2), reinterpret_cast<uint32_t*>(s_in), a.ctl,
                                    sy))
            return;
        MEGA_LMARK(l, 4);
        {
            float acc[BMAX];
            po.template dot<BMAX>(s_in, B, acc);
            const int row = d0 + so;
            const int li = tid & (T::OL - 1);
            if (so < nd) {
#pragma unroll
                for (int b = 0; b < BMAX; ++b)
                    if (b < B && li == b) put(a.ex_x + (size_t)b * D + row, E(5 * l + 3), s_x[b * D + row] + acc[b]);
            }
        }
        // ---------------- P3: LN2 + FC1 + GELU -----------------------------------------------
        bar();  // P2's reads of s_in / s_x / s_w[1] are done
        MEGA_LMARK(l, 5);
        ln.load(a.ln2_g.at(l), a.ln2_b.at(l));
        p2.params(a.fc2_s.at(l), a.fc2_z.at(l), a.fc2_b.at(l), d0, nd, s_w + L::kOffC);
        if (!gather<ux<BMAX>(), NC>(a.ex_x, B * D, Flat{}, E(5 * l + 3), s_x, a.ctl, sy)) return;
        MEGA_LMARK(l, 6);
        layer_norm<BMAX>(s_x, s_in, ln, a.eps, B);
        bar();  // s_in complete; the copy wave has waited for the FC1 share
        MEGA_LMARK(l, 7);
        {
            float acc[BMAX];
            p1.template dot<BMAX>(s_in, B, acc);
            const int row = f0 + s1;  // even for even s1: the row pair (s1, s1 + 1) sits in one wave
            const int li = tid & (T::AL - 1);
            static_assert(64 % (2 * T::AL) == 0, "an FC1 row pair within a wave");
#pragma unroll
            for (int b = 0; b < BMAX; ++b) {
                const float g = gelu_tanh(acc[b]);
                const float gn = __shfl_down(g, T::AL, kWave);
                if (b < B && li == b && !(s1 & 1) && s1 < nf)
                    put2(a.ex_h + ((size_t)b * FF + row) / 2, E(5 * l + 4), g, gn);
            }
        }
        // ---------------- P4: FC2 + residual -------------------------------------------------
        bar();  // P3's reads of s_in / s_w[0] are done
        MEGA_LMARK(l, 8);
        if (l + 1 < a.n_layer) pq.params(a.qkv_s.at(l + 1), a.qkv_z.at(l + 1), a.qkv_b.at(l + 1), q0, nq, s_w);
        if (!gather<uh<BMAX>(), NC>(a.ex_h, B * FF / 2, Flat{}, E(5 * l + 4), reinterpret_cast<uint32_t*>(s_in), a.ctl,
                                    sy))
            return;
        MEGA_LMARK(l, 9);
        {
            float acc[BMAX];
            p2.template dot<BMAX>(s_in, B, acc);
            const int row = d0 + s2;
            const int li = tid & (T::BL - 1);
            if (s2 < nd) {
#pragma unroll
                for (int b = 0; b < BMAX; ++b)
                    if (b < B && li == b) put(a.ex_x + (size_t)b * D + row, E(5 * l + 5), s_x[b * D + row] + acc[b]);
            }
        }
        MEGA_LMARK(l, 10);
    }

    // ---------------- LN_f + LM head (+ greedy argmax) -------------------------------------
    bar();  // the last FC2's reads of s_w[1] / s_in / s_x are done
    Share<FTTS_BF16, HL, HC, D> ph;
    ph.params(nullptr, nullptr, a.head_b, v0, nv, s_w);
    ln.load(a.lnf_g, a.lnf_b);
    if (!gather<ux<BMAX>(), NC>(a.ex_x, B * D, Flat{}, E(5 * a.n_layer), s_x, a.ctl, sy)) return;
    MEGA_MARK(1 + a.n_layer * kMarksPerLayer);
    // the step's last-layer hidden state (every group forms the same rows; GEMV group 0 writes them)
    layer_norm<BMAX>(s_x, s_in, ln, a.eps, B, k == 0 ? a.hidden : nullptr);
    bar();  // s_in complete; the copy wave has waited for the head share
    MEGA_MARK(2 + a.n_layer * kMarksPerLayer);
    {
        float acc[BMAX];
        ph.template dot<BMAX>(s_in, B, acc);
        const int row = v0 + sh;
        const int li = tid & (HL - 1);
        const bool mine = sh < nv;
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
        if (k == 0 && tid == 0) st_agent(a.ctl, step + 1);
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
        put(a.ex_arg + ((size_t)k * B + tid) * 2, E(5 * a.n_layer + 1), bv);
        put(a.ex_arg + ((size_t)k * B + tid) * 2 + 1, E(5 * a.n_layer + 1), __int_as_float(bi));
    }
    if (k != 0) return;
    float* s_cand = reinterpret_cast<float*>(s_w);  // the head share has been read (barrier above)
    if (!gather<ua<BMAX>(), NC>(a.ex_arg, NG * B * 2, Flat{}, E(5 * a.n_layer + 1), s_cand, a.ctl, sy)) return;
    if (wave < B) {
        const int b = wave;
        float bv = -INFINITY;
        int bi = 0x7FFFFFFF;
        for (int g = lane; g < NG; g += 64) {
            const float v = s_cand[(g * B + b) * 2];
            const int i = __float_as_int(s_cand[(g * B + b) * 2 + 1]);
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
