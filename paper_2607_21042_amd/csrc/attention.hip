// Attention kernels.
//
// Decode (one query row per sequence and head, over its paged KV cache):
//   o_h = softmax(q_h K_h^T / sqrt(64)) V_h over cached slots 0 .. seq_len
// split over contiguous runs of `pps` logical pages (flash-decoding).  Each
// split is one wave: a 64x64 K or V page is read as 8 fully coalesced 1 KB
// wave loads, lane l holding dims (l%8)*8 .. +7 of tokens i*8 + l/8.  Scores
// are reduced over the 8 lanes of a token, the page's softmax is folded into a
// running (max, sum, output) triple, and the partial of each split is merged
// with the log-sum-exp rule by a second kernel.  Splits follow logical pages,
// so the result does not depend on where the pages live in the pool.
//
// Prefill (causal attention over each prefix, queries in tiles of 64): one
// thread per query row keeps q and the output in registers and streams 64-key
// tiles of K and V through LDS.
#include "ftts_internal.hpp"

namespace ftts {

template <bool F32>
__device__ __forceinline__ void load8(const void* base, size_t elem, float (&v)[8]) {
    if constexpr (F32) {
        const float4* p = reinterpret_cast<const float4*>(reinterpret_cast<const float*>(base) + elem);
        const float4 a = p[0], b = p[1];
        v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
        v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
    } else {
        const uint4 w = *reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(base) + elem);
        v[0] = bf16lo(w.x); v[1] = bf16hi(w.x); v[2] = bf16lo(w.y); v[3] = bf16hi(w.y);
        v[4] = bf16lo(w.z); v[5] = bf16hi(w.z); v[6] = bf16lo(w.w); v[7] = bf16hi(w.w);
    }
}

template <bool F32>
__global__ __launch_bounds__(64) void attn_decode_split(const AttnDecodeArgs a) {
    const int s = blockIdx.x, h = blockIdx.y, b = blockIdx.z;
    const int lane = threadIdx.x;
    if (!a.active[b]) return;
    const int ctx = a.seq_lens[b] + 1;                 // cached slots incl. the new token
    const int n_pages_ctx = (ctx + kPage - 1) / kPage;
    const int p0 = s * a.pps;
    if (p0 >= n_pages_ctx) return;
    const int p1 = min(p0 + a.pps, n_pages_ctx);

    const int grp = lane >> 3, sub = lane & 7;         // token within 8-token row, dim block
    float q[8];
    {
        const float* qp = a.qkv + (size_t)b * a.qkv_stride + h * kHeadDim + sub * 8;
#pragma unroll
        for (int j = 0; j < 8; ++j) q[j] = qp[j] * 0.125f;  // 1/sqrt(64), exact
    }
    float m = -INFINITY, l = 0.f, o[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) o[j] = 0.f;

    for (int p = p0; p < p1; ++p) {
        const int phys = a.block_table[(size_t)b * a.max_pages + p];
        if (phys < 0 || phys >= a.n_pages) continue;
        const size_t kbase = kv_offset(a.layer, a.n_pages, phys, 0, a.n_head, h, 0);
        const size_t vbase = kv_offset(a.layer, a.n_pages, phys, 1, a.n_head, h, 0);
        float sc[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            float kv[8];
            load8<F32>(a.kv_base, kbase + (size_t)(i * 64 + lane) * 8, kv);
            float t = 0.f;
#pragma unroll
            for (int j = 0; j < 8; ++j) t = fmaf(q[j], kv[j], t);
            sc[i] = t;
        }
        float pm = -INFINITY;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            float t = sc[i];
            t += __shfl_xor(t, 1, kWave);
            t += __shfl_xor(t, 2, kWave);
            t += __shfl_xor(t, 4, kWave);
            const int tok = p * kPage + i * 8 + grp;
            sc[i] = tok < ctx ? t : -INFINITY;
            pm = fmaxf(pm, sc[i]);
        }
        pm = fmaxf(pm, __shfl_xor(pm, 8, kWave));
        pm = fmaxf(pm, __shfl_xor(pm, 16, kWave));
        pm = fmaxf(pm, __shfl_xor(pm, 32, kWave));
        const float mn = fmaxf(m, pm);
        const float alpha = expf(m - mn);              // 0 on the first page (m = -inf)
        m = mn;
        l *= alpha;
#pragma unroll
        for (int j = 0; j < 8; ++j) o[j] *= alpha;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            // Slots past the context hold whatever the pool held: never let them
            // into the sum (0 * NaN would poison it).
            if (p * kPage + i * 8 + grp < ctx) {
                const float pr = expf(sc[i] - m);
                float vv[8];
                load8<F32>(a.kv_base, vbase + (size_t)(i * 64 + lane) * 8, vv);
                l += pr;
#pragma unroll
                for (int j = 0; j < 8; ++j) o[j] = fmaf(pr, vv[j], o[j]);
            }
        }
    }
    // Sum over the 8 token groups (lanes with equal l % 8 hold the same dims).
#pragma unroll
    for (int j = 0; j < 8; ++j) {
        float t = o[j];
        t += __shfl_xor(t, 8, kWave);
        t += __shfl_xor(t, 16, kWave);
        t += __shfl_xor(t, 32, kWave);
        o[j] = t;
    }
    l += __shfl_xor(l, 8, kWave);
    l += __shfl_xor(l, 16, kWave);
    l += __shfl_xor(l, 32, kWave);
    float* part = a.part + (((size_t)b * a.n_head + h) * a.n_splits + s) * kPartStride;
    if (lane < 8) {
#pragma unroll
        for (int j = 0; j < 8; ++j) part[lane * 8 + j] = o[j];
    }
    if (lane == 0) {
        part[64] = m;
        part[65] = l;
    }
}

__global__ __launch_bounds__(64) void attn_decode_merge(const AttnDecodeArgs a) {
    const int h = blockIdx.x, b = blockIdx.y, d = threadIdx.x;
    float* out = a.o + (size_t)b * a.o_stride + h * kHeadDim + d;
    if (!a.active[b]) {
        *out = 0.f;
        return;
    }
    const int ctx = a.seq_lens[b] + 1;
    const int n_pages_ctx = (ctx + kPage - 1) / kPage;
    const int ns = (n_pages_ctx + a.pps - 1) / a.pps;
    const float* part = a.part + ((size_t)b * a.n_head + h) * a.n_splits * kPartStride;
    float M = -INFINITY;
    for (int s = 0; s < ns; ++s) M = fmaxf(M, part[s * kPartStride + 64]);
    float L = 0.f, acc = 0.f;
    for (int s = 0; s < ns; ++s) {
        const float ms = part[s * kPartStride + 64];
        if (ms == -INFINITY) continue;                 // split held no valid page
        const float w = expf(ms - M);
        L = fmaf(part[s * kPartStride + 65], w, L);
        acc = fmaf(part[s * kPartStride + d], w, acc);
    }
    *out = L > 0.f ? acc / L : 0.f;
}

hipError_t launch_attn_decode(int wdtype, const AttnDecodeArgs& a, int B, hipStream_t st) {
    const dim3 g1(a.n_splits, a.n_head, B);
    if (wdtype == FTTS_F32) hipLaunchKernelGGL(attn_decode_split<true>, g1, dim3(64), 0, st, a);
    else hipLaunchKernelGGL(attn_decode_split<false>, g1, dim3(64), 0, st, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(attn_decode_merge, dim3(a.n_head, B), dim3(64), 0, st, a);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------------------
// Causal prefill attention.  Block = one (sequence, 64-query tile, head); thread t owns
// query row tile*64 + t of that sequence.
template <bool F32>
__global__ __launch_bounds__(64) void attn_prefill_kernel(const AttnPrefillArgs a) {
    __shared__ float sk[64][kHeadDim + 1];
    __shared__ float sv[64][kHeadDim + 1];
    const int h = blockIdx.y, t = threadIdx.x;
    int gt = blockIdx.x, sq = 0;
    while (sq + 1 < a.seqs.n && a.tiles_cu[sq + 1] <= gt) ++sq;
    const int tile = gt - a.tiles_cu[sq];
    const int row0 = a.seqs.cu[sq];
    const int len = a.seqs.cu[sq + 1] - row0;
    const int qi = tile * 64 + t;                        // query position in the sequence
    const bool qok = qi < len;
    const int ld = 3 * a.d_model;

    float q[kHeadDim], o[kHeadDim];
#pragma unroll
    for (int j = 0; j < kHeadDim; ++j) {
        q[j] = qok ? ld_act<F32>(a.qkv, (size_t)(row0 + qi) * ld + h * kHeadDim + j) * 0.125f : 0.f;
        o[j] = 0.f;
    }
    float m = -INFINITY, l = 0.f;
    const int kend = min(len, tile * 64 + 64);            // keys needed by this tile
    for (int k0 = 0; k0 < kend; k0 += 64) {
        __syncthreads();
        for (int i = t; i < 64 * kHeadDim; i += 64) {
            const int r = i / kHeadDim, c = i % kHeadDim;
            const int kr = k0 + r;
            float kv = 0.f, vv = 0.f;
            if (kr < len) {
                const size_t base = (size_t)(row0 + kr) * ld + h * kHeadDim + c;
                kv = ld_act<F32>(a.qkv, base + a.d_model);
                vv = ld_act<F32>(a.qkv, base + 2 * a.d_model);
            }
            sk[r][c] = kv;
            sv[r][c] = vv;
        }
        __syncthreads();
        if (!qok) continue;
        const int nk = min(64, qi - k0 + 1);               // keys k0 .. qi are visible
        if (nk <= 0) continue;
        float sc[64];
        float tm = -INFINITY;
#pragma unroll
        for (int r = 0; r < 64; ++r) {
            float s = 0.f;
#pragma unroll
            for (int j = 0; j < kHeadDim; ++j) s = fmaf(q[j], sk[r][j], s);
            sc[r] = r < nk ? s : -INFINITY;
            tm = fmaxf(tm, sc[r]);
        }
        const float mn = fmaxf(m, tm);
        const float alpha = expf(m - mn);
        m = mn;
        l *= alpha;
#pragma unroll
        for (int j = 0; j < kHeadDim; ++j) o[j] *= alpha;
#pragma unroll
        for (int r = 0; r < 64; ++r) {
            const float p = expf(sc[r] - m);
            l += p;
#pragma unroll
            for (int j = 0; j < kHeadDim; ++j) o[j] = fmaf(p, sv[r][j], o[j]);
        }
    }
    if (!qok) return;
    const float inv = 1.0f / l;
#pragma unroll
    for (int j = 0; j < kHeadDim; ++j)
        st_act<F32>(a.o, (size_t)(row0 + qi) * a.d_model + h * kHeadDim + j, o[j] * inv);
}

hipError_t launch_attn_prefill(int wdtype, const AttnPrefillArgs& a, int total_tiles, hipStream_t st) {
    const dim3 g(total_tiles, a.n_head);
    if (wdtype == FTTS_F32) hipLaunchKernelGGL(attn_prefill_kernel<true>, g, dim3(64), 0, st, a);
    else hipLaunchKernelGGL(attn_prefill_kernel<false>, g, dim3(64), 0, st, a);
    return hipGetLastError();
}

}  // namespace ftts
