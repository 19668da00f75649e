// Dispatch of the decode GEMV family: picks an exact tiling of K for the weight
// type and batch, and splits the batch into groups of at most 16 rows (smaller
// when a LayerNorm-fused row would not fit the LDS budget in one pass).
#include "gemv_impl.hpp"

namespace ftts {

static int elems_per_chunk(int wdtype) {
    return wdtype == FTTS_F32 ? 4 : wdtype == FTTS_BF16 ? 8 : wdtype == FTTS_W8A16 ? 16 : 32;
}

static int bmax_for(int B) { return B <= 1 ? 1 : B <= 4 ? 4 : 16; }

// Fewest passes over K, then most lanes per row; LayerNorm-fused rows need one pass.
static bool pick_tiling(int wdtype, int K, int bmax, bool single_pass, Tiling* out) {
    static const Tiling cands[] = {{64, 10}, {64, 5}, {64, 4}, {32, 5}, {32, 4}, {16, 5},
                                   {16, 4},  {16, 2}, {8, 5},  {8, 4},  {8, 2},  {8, 1}};
    const int epc = elems_per_chunk(wdtype);
    if (K % epc) return false;
    const int chunks = K / epc;
    const int budget = kGemvLdsFloats / bmax;
    int best_passes = 1 << 30;
    for (const Tiling& t : cands) {
        const int per = t.lpr * t.nch;
        if (chunks % per || per * epc > budget) continue;
        const int passes = chunks / per;
        if (single_pass && passes != 1) continue;
        if (passes < best_passes) {
            best_passes = passes;
            *out = t;
        }
    }
    return best_passes != (1 << 30);
}

static hipError_t dispatch(int wdtype, int epi, bool ln, const GemvArgs& a, Tiling t, hipStream_t st) {
    switch (wdtype) {
        case FTTS_F32: return ln ? gemv_ln_f32(epi, a, t, st) : gemv_res_f32(epi, a, t, st);
        case FTTS_BF16: return ln ? gemv_ln_bf16(epi, a, t, st) : gemv_res_bf16(epi, a, t, st);
        case FTTS_W8A16: return ln ? gemv_ln_w8(epi, a, t, st) : gemv_res_w8(epi, a, t, st);
        case FTTS_W4A16: return ln ? gemv_ln_w4(epi, a, t, st) : gemv_res_w4(epi, a, t, st);
    }
    return hipErrorInvalidValue;
}

bool gemv_supported(int wdtype, int K, bool ln) {
    Tiling t;
    return pick_tiling(wdtype, K, 1, ln, &t) && pick_tiling(wdtype, K, 16, ln, &t);
}

hipError_t launch_gemv(int wdtype, int epi, bool ln, const GemvArgs& in, hipStream_t st) {
    // The LM head is never quantised: fp32 in FTTS_F32 mode, bf16 otherwise.
    const int wt = epi == EPI_STORE ? (wdtype == FTTS_F32 ? FTTS_F32 : FTTS_BF16) : wdtype;
    int group = 16;
    if (ln) {
        const int fit = kGemvLdsFloats / in.K;  // rows whose full K fits the LDS budget
        group = fit < group ? fit : group;
        if (group < 1) return hipErrorInvalidValue;
    }
    for (int b0 = 0; b0 < in.B; b0 += group) {
        GemvArgs a = in;
        a.B = in.B - b0 < group ? in.B - b0 : group;
        a.act = in.act + (size_t)b0 * in.K;
        a.out = in.out + (size_t)b0 * in.out_stride;
        if (epi == EPI_QKV) {
            a.kv.seq_lens = in.kv.seq_lens + b0;
            a.kv.active = in.kv.active + b0;
            a.kv.block_table = in.kv.block_table + (size_t)b0 * in.kv.max_pages;
        }
        Tiling t;
        if (!pick_tiling(wt, a.K, bmax_for(a.B), ln, &t)) return hipErrorInvalidValue;
        const hipError_t e = dispatch(wt, epi, ln, a, t, st);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace ftts
