// Internal declarations shared by the HIP translation units of libftts.
// Device helpers (bf16 conversion, wave reductions) and the launch-argument
// structs of every kernel family.  Nothing here is part of the C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "ftts.h"

namespace ftts {

constexpr int kWave = 64;        // CDNA wavefront width
constexpr int kPage = 64;        // KV tokens per page
constexpr int kHeadDim = 64;     // attention head width
constexpr int kMaxPages = 512;   // logical pages per sequence (32768 tokens)

// ---- bf16 <-> fp32 --------------------------------------------------------------
__device__ __forceinline__ float bf16_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }
__device__ __forceinline__ float bf16lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// Round to nearest bf16, ties to even (NaN stays NaN, quietened): gfx950's
// packed conversion, one instruction.
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    typedef __bf16 bf16x2_rne_t __attribute__((ext_vector_type(2)));
    const bf16x2_rne_t v = {(__bf16)f, (__bf16)0.f};
    return (uint16_t)__builtin_bit_cast(uint32_t, v);
}

// 16-byte streaming load (weights are read once per call; the hint keeps them from
// displacing activations in the caches).
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 ld_stream(const uint4* p) {
    const u32x4_t v = __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
}

// Workgroup barrier for LDS traffic only.  __syncthreads() also waits for every
// outstanding global load of the wave; this one leaves the weight stream in
// flight.  Global data exchanged through it must have been waited for already.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// Activation/parameter element: fp32 in FTTS_F32 mode, bf16 in the 16-bit modes.
template <bool F32>
__device__ __forceinline__ float ld_act(const void* p, size_t i) {
    if constexpr (F32) return reinterpret_cast<const float*>(p)[i];
    else return bf16_to_f32(reinterpret_cast<const uint16_t*>(p)[i]);
}
template <bool F32>
__device__ __forceinline__ void st_act(void* p, size_t i, float v) {
    if constexpr (F32) reinterpret_cast<float*>(p)[i] = v;
    else reinterpret_cast<uint16_t*>(p)[i] = f32_to_bf16(v);
}

// ---- cross-lane reductions ----------------------------------------------------------
// Built from DPP lane moves within 16-lane rows and the gfx950 row swaps
// (v_permlane16_swap / v_permlane32_swap), which stay in the VALU instead of
// going through the LDS crossbar as ds_bpermute does.  Every lane of a group
// ends with the same bits (each step adds a pair in both orders, and fp32
// addition is commutative).  The whole wave must be active.
template <int CTRL>
__device__ __forceinline__ float dpp_mov(float v) {
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}
constexpr int kDppQuadSwap1 = 0xB1;      // quad_perm [1,0,3,2]
constexpr int kDppQuadSwap2 = 0x4E;      // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141;    // lane i <-> 7 - i within each 8
constexpr int kDppMirror = 0x140;        // lane i <-> 15 - i within each 16
constexpr int kDppRor8 = 0x128;          // lane i <- (i + 8) mod 16 within each 16
struct RowPair { float a, b; };
__device__ __forceinline__ RowPair swap16(float v) {  // a: own row pair's even row, b: its odd row
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return {__uint_as_float(r[0]), __uint_as_float(r[1])};
}
__device__ __forceinline__ RowPair swap32(float v) {  // a: lanes 0-31 value, b: lanes 32-63 value
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return {__uint_as_float(r[0]), __uint_as_float(r[1])};
}

// Sum / max over aligned groups of W consecutive lanes (W a power of two <= 64).
template <int W>
__device__ __forceinline__ float group_sum(float v) {
    if constexpr (W >= 2) v += dpp_mov<kDppQuadSwap1>(v);
    if constexpr (W >= 4) v += dpp_mov<kDppQuadSwap2>(v);
    if constexpr (W >= 8) v += dpp_mov<kDppHalfMirror>(v);
    if constexpr (W >= 16) v += dpp_mov<kDppMirror>(v);
    if constexpr (W >= 32) { const RowPair p = swap16(v); v = p.a + p.b; }
    if constexpr (W >= 64) { const RowPair p = swap32(v); v = p.a + p.b; }
    return v;
}
template <int W>
__device__ __forceinline__ float group_max(float v) {
    if constexpr (W >= 2) v = fmaxf(v, dpp_mov<kDppQuadSwap1>(v));
    if constexpr (W >= 4) v = fmaxf(v, dpp_mov<kDppQuadSwap2>(v));
    if constexpr (W >= 8) v = fmaxf(v, dpp_mov<kDppHalfMirror>(v));
    if constexpr (W >= 16) v = fmaxf(v, dpp_mov<kDppMirror>(v));
    if constexpr (W >= 32) { const RowPair p = swap16(v); v = fmaxf(p.a, p.b); }
    if constexpr (W >= 64) { const RowPair p = swap32(v); v = fmaxf(p.a, p.b); }
    return v;
}
// Sum / max over the 8 lanes sharing lane % 8 (lanes i, i + 8, ..., i + 56).
__device__ __forceinline__ float stride8_sum(float v) {
    v += dpp_mov<kDppRor8>(v);
    { const RowPair p = swap16(v); v = p.a + p.b; }
    { const RowPair p = swap32(v); v = p.a + p.b; }
    return v;
}
__device__ __forceinline__ float stride8_max(float v) {
    v = fmaxf(v, dpp_mov<kDppRor8>(v));
    { const RowPair p = swap16(v); v = fmaxf(p.a, p.b); }
    { const RowPair p = swap32(v); v = fmaxf(p.a, p.b); }
    return v;
}
__device__ __forceinline__ float wave_sum(float v) { return group_sum<kWave>(v); }
__device__ __forceinline__ float wave_max(float v) { return group_max<kWave>(v); }

// Row statistics of one 32-column tile held by the 32 lanes of a half wave (one
// value per lane): (sum, sum of squared deviations from the tile's own mean).
// LayerNorm consumers merge the tiles of a row exactly by the law of total
// variance, so no pass over the row is needed.  The whole wave must be active.
constexpr int kStatTile = 32;
__device__ __forceinline__ float2 tile_stats32(float v) {
    const float s = group_sum<kStatTile>(v);
    const float dv = v - s * (1.0f / kStatTile);
    return make_float2(s, group_sum<kStatTile>(dv * dv));
}

// GPT-2 tanh GELU.
__device__ __forceinline__ float gelu_tanh(float u) {
    const float c = 0.7978845608028654f;  // sqrt(2/pi)
    return 0.5f * u * (1.0f + tanhf(c * (u + 0.044715f * u * u * u)));
}

// Element offset of (layer, physical page, k|v, head, slot, dim) in the KV pool.
__device__ __forceinline__ size_t kv_offset(int layer, int n_pages, int phys, int kv, int n_head, int head,
                                            int slot) {
    return ((((size_t)layer * n_pages + phys) * 2 + kv) * n_head + head) * (size_t)(kPage * kHeadDim) +
           (size_t)slot * kHeadDim;
}

// ---- launch arguments -------------------------------------------------------------
// A per-layer tensor stored at a fixed stride: layer l lives at p + l * s bytes.
struct Strided {
    const char* p;
    long long s;
    __host__ __device__ const void* at(int l) const { return p ? p + (long long)l * s : nullptr; }
};

enum Epi { EPI_STORE = 0, EPI_QKV = 1, EPI_GELU = 2, EPI_RESID = 3 };

struct KvAppend {            // where the QKV epilogue writes keys and values
    void* base;
    int n_pages, layer, n_head, d_model, max_pages;
    const int32_t* block_table;
    const int32_t* seq_lens;  // decode: slot = seq_lens[b]
    const int32_t* active;    // decode: per-row flag
};

struct GemvArgs {
    const void* w;           // [N][K] weights in the mode's storage
    const uint16_t* scale;   // W8: [N]; W4: [N][K/128]
    const uint16_t* zero;    // W4: [N][K/128]
    const void* bias;        // [N] activation dtype
    int N, K, B;
    const float* act;        // [B][K] fp32 input (x when LayerNorm is fused)
    const void* ln_g;        // LayerNorm gain / bias (activation dtype) or null
    const void* ln_b;
    float eps;
    float* out;              // [B][out_stride] fp32
    int out_stride;
    KvAppend kv;
    float* hidden;           // LayerNorm rows: [B][K] copy of the normalised input (LM head), or null
};

struct AttnDecodeArgs {
    const float* qkv;        // [B][3d] fp32; q of head h at h*64
    int qkv_stride;
    const void* kv_base;
    int n_pages, layer, n_head, max_pages;
    const int32_t* block_table;
    const int32_t* seq_lens;
    const int32_t* active;
    float* o;                // [B][o_stride] fp32 attention output
    int o_stride;
    uint16_t* o_bf16;        // if set, the output goes here as bf16 instead
};

// Batched decode linear on the matrix cores (bgemm.hip).
struct BgemmArgs {
    const void* w;           // [N][K] weights in the mode's storage
    const uint16_t* scale;   // W8: [N]; W4: [N][K/128]
    const uint16_t* zero;    // W4: [N][K/128]
    const void* bias;        // [N] bf16
    int N, K, B;
    const void* act;         // [B][K] bf16 input
    float* out;              // STORE / QKV: written, RESID: added to; [B][out_stride] fp32
    void* out_bf16;          // GELU: [B][out_stride] bf16
    int out_stride;
    float* part;             // [S][B][N] fp32 split-K partials
    uint32_t* count;         // [ceil(N/32)] arrival counters, zero between calls
    KvAppend kv;             // EPI_QKV: decode form (slot = seq_lens[b], only active rows)
    // LayerNorm on the input side: when ln_x is set, act is ignored and the input
    // row m is LN(ln_x[m]) with gain ln_g / bias ln_b, its mean and variance
    // merged from ln_stats (tile statistics, [K/32][stats_ld], see tile_stats32).
    const float* ln_x;       // [B][K] fp32
    const void* ln_g;
    const void* ln_b;
    float ln_eps;
    const float2* ln_stats;
    // EPI_RESID: tile statistics of the updated rows go to stats_out [N/32][stats_ld].
    float2* stats_out;
    int stats_ld;
    float* hidden;           // with ln_x: [B][K] copy of the normalised rows (LM head), or null
};
// Decode batches of at least this many take the MFMA linears: 5 (16-bit and
// int8 weights: the GEMV tilings fall behind from 5 rows on), 3 for W4A16.
inline int batched_min(int wdtype) { return wdtype == FTTS_W4A16 ? 3 : 5; }

constexpr int kMaxPrefillSeqs = FTTS_MAX_BATCH;
struct SeqTable {            // packed varlen sequences, passed by value
    int n;
    int cu[kMaxPrefillSeqs + 1];  // row offsets
};

struct GemmArgs {
    const void* a;           // [M][K] activation dtype
    const void* w;           // [N][K] weights
    const uint16_t* scale;
    const uint16_t* zero;
    const void* bias;
    int M, N, K;
    void* out;               // STORE/QKV/GELU: [M][N] activation dtype; RESID: fp32 [M][N] in place
    KvAppend kv;             // QKV epilogue (prefill form: slot = position within the sequence)
    SeqTable seqs;
    float* part;             // split K: [S][M][N] fp32 partial tiles
    uint32_t* count;         // split K: per-tile arrival counters, zero between calls
};
struct GemmPlan {            // 16-bit-mode prefill GEMM launch shape
    int mt;                  // 64-row blocks per tile (1 or 2)
    int tiles_m, tiles_n, splits;
};
GemmPlan gemm_plan(int M, int N, int K);

struct AttnPrefillArgs {
    const void* qkv;         // [M][3d] activation dtype
    void* o;                 // [M][d] activation dtype
    int d_model, n_head;
    SeqTable seqs;
    int tiles_cu[kMaxPrefillSeqs + 1];  // prefix sums of query tiles (prefill_tile_rows) per sequence
};

// Prefill input assembly: sequence b's rows are its cond_lens[b] conditioning
// rows as given (no position embedding), then its text rows
// tok_emb[vocab + id] + pos_emb[text_pos0 + i] (merged token table, text range
// of the position table).
struct AssembleArgs {
    SeqTable seqs;                        // row offsets of the assembled prefixes
    int cond_cu[kMaxPrefillSeqs + 1];     // prefix sums of the conditioning rows
    const void* cond;                     // [sum cond][d] activation dtype
    const int32_t* text_ids;              // [sum text] (text row i of b at seqs.cu[b] - cond_cu[b] + i)
    const void* tok_emb;
    const void* pos_emb;
    int d, vocab, text_vocab, text_pos0;
    float* x;                             // [sum lens][d] fp32 out
};

// ---- launchers (each returns a hipError_t from the launch) --------------------------
hipError_t launch_embed(int wdtype, const void* tok_emb, const void* pos_emb, int vocab, int n_pos, int d,
                        const int32_t* tokens, const int32_t* positions, const int32_t* seq_lens,
                        const int32_t* block_table, int max_pages, int n_pages, int B, float* x,
                        int32_t* active, float2* stats, uint32_t* zero, int n_zero, hipStream_t st);
hipError_t launch_gemv(int wdtype, int epi, bool ln, const GemvArgs& a, hipStream_t st);
bool gemv_supported(int wdtype, int K, bool ln);
hipError_t launch_attn_decode(int wdtype, const AttnDecodeArgs& a, int B, hipStream_t st);
hipError_t launch_sample(const float* logits, int B, int V, const ftts_sampling& s, const float* uniforms,
                         const int32_t* active, int32_t* out, hipStream_t st);
hipError_t launch_quantize(int wdtype, const float* w, int64_t N, int64_t K, int group, void* codes,
                           uint16_t* scales, uint16_t* zeros, hipStream_t st);
hipError_t launch_ln_rows(int wdtype, const float* x, const void* g, const void* b, float eps, int M, int d,
                          void* out, hipStream_t st);
hipError_t launch_gemm(int wdtype, int epi, const GemmArgs& a, hipStream_t st);
hipError_t launch_attn_prefill(int wdtype, const AttnPrefillArgs& a, int total_tiles, hipStream_t st);
int prefill_tile_rows(int wdtype);  // queries per prefill-attention workgroup
// Attention without a mask (every query sees every key of its sequence), bf16; the
// launcher sets its own query tiling (tiles_cu of `a` is ignored).
hipError_t launch_attn_full_bf16(const AttnPrefillArgs& a, hipStream_t st);
hipError_t launch_gather_rows(const float* x, int d, const SeqTable& seqs, float* out, hipStream_t st);
hipError_t launch_advance(int32_t* tokens, int32_t* positions, int32_t* seq_lens, int32_t* sampled,
                          int32_t* remaining, int32_t stop_token, bool retire_on_stop, int32_t* history,
                          int32_t* step_counter, int max_steps, int B, hipStream_t st);
hipError_t launch_fill_u32(uint32_t* p, size_t n, uint32_t v, hipStream_t st);
hipError_t launch_bgemm(int wdtype, int epi, const BgemmArgs& a, hipStream_t st);
int bgemm_splits(int wdtype, int N, int K, bool ln);
bool bgemm_supported(int wdtype, int K, bool ln);
hipError_t launch_act_to_f32(int wdtype, const void* src, int rows, int d, float* dst, hipStream_t st);
hipError_t launch_assemble_prefix(int wdtype, const AssembleArgs& a, int rows, hipStream_t st);

// Flow-matching DiT step (bf16): time embedding, input rows and guidance.
struct DitPrepareArgs {
    int T, n_mel, d_cond, d_model;
    const float* x;          // [T][n_mel] state
    const void* cond;        // [T][d_cond] bf16
    const float* e;          // [d_model] time embedding
    void* inp;               // [2T][n_mel + d_cond] bf16 out
    float* h;                // [2T][d_model] out: every row = e
    float* vel;              // [2T][n_mel] out: zeros
    uint32_t* count;         // [n_count] out: zeros
    size_t n_count;
};
hipError_t launch_dit_time(float t, const void* w1, const void* b1, const void* w2, const void* b2, int D, int t_dim,
                           float* u, float* e, hipStream_t st);
hipError_t launch_dit_prepare(const DitPrepareArgs& a, hipStream_t st);
hipError_t launch_dit_guide(const float* vel, int T, int n_mel, float w, float dt, const float* x, float* x_out,
                            float* v_out, hipStream_t st);

namespace mega {
constexpr int D = 1280, FF = 5120, NH = 20;
constexpr int G = 256;   // workgroups of the persistent decode step, one per CU
constexpr int BM = 2;    // largest batch it takes
struct Args {
    int n_layer, V, n_pos, B, max_pages, n_pages, greedy;
    float eps;
    Strided ln1_g, ln1_b, ln2_g, ln2_b;
    Strided qkv_w, qkv_s, qkv_z, qkv_b, out_w, out_s, out_z, out_b;
    Strided fc1_w, fc1_s, fc1_z, fc1_b, fc2_w, fc2_s, fc2_z, fc2_b;
    const void *tok_emb, *pos_emb, *lnf_g, *lnf_b, *head_w, *head_b;
    const int32_t *tokens, *positions, *seq_lens, *block_table;
    void* kv;
    float* logits;
    float* hidden;           // [B][d] LN_f output of the step (the LM head's input), or null
    int32_t* sampled;
    int32_t* active_out;
    // exchange words (32 value bits | epoch << 32): x [B][d] fp32, q/k/v [B][3d] fp32,
    // o [B][d/2] and h [B][d_ff/2] bf16 pairs, argmax candidates [groups][B][2]
    uint64_t *ex_x, *ex_qkv, *ex_o, *ex_h, *ex_arg;
    uint32_t* ctl;  // [0] step counter, [1] abort
};

}
hipError_t launch_decode_mega(int wdtype, const mega::Args& a, hipStream_t st);
int decode_mega_blocks_per_cu(int wdtype, int B);

}  // namespace ftts
