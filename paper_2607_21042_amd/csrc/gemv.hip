// Dispatch of the decode GEMV family by weight type and batch size.  The kernel
// template is instantiated for up to 16 batch rows; larger batches run in
// passes of 16 rows over the same weights.
#include "gemv_impl.hpp"

namespace ftts {

// Lanes per row: enough 16-byte chunks per lane (about five) to keep loads in flight.
static int pick_lpr(int wdtype, int K) {
    const int epc = wdtype == FTTS_F32 ? 4 : wdtype == FTTS_BF16 ? 8 : wdtype == FTTS_W8A16 ? 16 : 32;
    const int chunks = K / epc;
    if (chunks >= 320) return 64;
    if (chunks >= 160) return 32;
    if (chunks >= 80) return 16;
    return 8;
}

static hipError_t dispatch(int wdtype, int epi, bool ln, const GemvArgs& a, hipStream_t st) {
    switch (wdtype) {
        case FTTS_F32: return gemv_f32(epi, ln, a, st);
        case FTTS_BF16: return gemv_bf16(epi, ln, a, st);
        case FTTS_W8A16: return gemv_w8(epi, ln, a, st);
        case FTTS_W4A16: return gemv_w4(epi, ln, a, st);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_gemv(int wdtype, int epi, bool ln, const GemvArgs& in, hipStream_t st) {
    // The LM head is never quantised: fp32 in FTTS_F32 mode, bf16 otherwise.
    const int wt = epi == EPI_STORE ? (wdtype == FTTS_F32 ? FTTS_F32 : FTTS_BF16) : wdtype;
    for (int b0 = 0; b0 < in.B; b0 += 16) {
        GemvArgs a = in;
        a.lpr = pick_lpr(wt, a.K);
        a.B = in.B - b0 < 16 ? in.B - b0 : 16;
        a.act = in.act + (size_t)b0 * in.K;
        a.out = in.out + (size_t)b0 * in.out_stride;
        if (epi == EPI_QKV) {
            a.kv.seq_lens = in.kv.seq_lens + b0;
            a.kv.active = in.kv.active + b0;
            a.kv.block_table = in.kv.block_table + (size_t)b0 * in.kv.max_pages;
        }
        const hipError_t e = dispatch(wt, epi, ln, a, st);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

}  // namespace ftts
