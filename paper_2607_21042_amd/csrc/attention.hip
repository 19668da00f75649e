// Attention kernels.
//
// Decode (one query row per sequence and head, over its paged KV cache):
//   o_h = softmax(q_h K_h^T / sqrt(64)) V_h over cached slots 0 .. seq_len
// One workgroup per (head, sequence) whose 8 waves stride over the logical
// pages (split-K inside the workgroup).  A 64x64 K or V page is read as 8 fully
// coalesced 1 KB wave loads, lane l holding dims (l%8)*8 .. +7 of tokens
// i*8 + l/8 (with 16-bit pages the next page's K and V would be loaded while
// the current one is used; only the fp32 instantiation is launched).
// Scores are reduced over the 8 lanes of a token, each page's softmax is
// folded into a running (max, sum, output) triple, and the 8 wave partials
// are merged in LDS with the log-sum-exp rule.  The walk follows logical
// pages, so the result does not depend on where pages live in the pool.  This
// is the fp32-KV kernel; the 16-bit KV kernel (attn_decode_bf16_kernel, below)
// keeps one page per wave in registers so that two groups share a CU.
//
// Prefill (causal attention over each prefix).  16-bit activations run on the
// matrix cores: a workgroup of 4 waves takes 128 queries of one head, each wave
// 32 of them, and walks 32-key tiles.  A wave forms S^T = K Q^T (keys as rows,
// so every lane ends up holding 16 scores of its own query), applies the online
// softmax per lane, and accumulates O^T = V^T P^T with the probabilities taken
// straight from its score registers: the MFMA k order is a permutation shared by
// both operands, so P needs no reshuffle.  V is transposed through LDS (double
// buffered, one barrier per tile).  fp32 activations keep a VALU kernel: one
// thread per query row streams 64-key tiles of K and V through LDS.
//
// Full attention (no mask: the flow-matching DiT's frames all see each other)
// has two matrix-core kernels: attn_full_mfma_kernel splits the keys of a
// 32-query tile over the waves of a workgroup (short grids), and
// attn_full_shared_kernel shares each K and V tile among 128 queries (wide grids).
#include "kv_page.hpp"

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

constexpr int kAttnWaves = 8;

// One workgroup per (head, sequence); wave w walks logical pages w, w + 8, ...
template <bool F32>
__global__ __launch_bounds__(kAttnWaves * 64) void attn_decode_kernel(const AttnDecodeArgs a) {
    __shared__ float s_m[kAttnWaves], s_l[kAttnWaves];
    __shared__ float s_o[kAttnWaves][kHeadDim];
    const int h = blockIdx.x, b = blockIdx.y;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    float* out = a.o + (size_t)b * a.o_stride + h * kHeadDim;
    uint16_t* out16 = a.o_bf16 ? a.o_bf16 + (size_t)b * a.o_stride + h * kHeadDim : nullptr;
    if (!a.active[b]) {
        if (tid < kHeadDim) {
            if (out16) out16[tid] = 0;
            else out[tid] = 0.f;
        }
        return;
    }
    const int ctx = a.seq_lens[b] + 1;                 // cached slots incl. the new token
    const int npg = (ctx + kPage - 1) / kPage;
    const int grp = lane >> 3, sub = lane & 7;

    // This wave's page ids: lane j holds the id of its j-th page (logical page w + 8 j).
    const int lp = w + kAttnWaves * lane;
    int my_phys = lp < npg ? a.block_table[(size_t)b * a.max_pages + lp] : -1;
    float q[8];
    {
        const float* qp = a.qkv + (size_t)b * a.qkv_stride + h * kHeadDim + sub * 8;
#pragma unroll
        for (int j = 0; j < 8; ++j) q[j] = qp[j] * 0.125f;  // 1/sqrt(64), exact
    }
    float m = -INFINITY, l = 0.f, o[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) o[j] = 0.f;

    auto page_base = [&](int j, size_t& kb, size_t& vb) {
        int phys = __shfl(my_phys, j, kWave);
        const bool ok = phys >= 0 && phys < a.n_pages;
        phys = ok ? phys : 0;
        kb = kv_offset(a.layer, a.n_pages, phys, 0, a.n_head, h, 0);
        vb = kv_offset(a.layer, a.n_pages, phys, 1, a.n_head, h, 0);
        return ok;
    };

    const int my_pages = npg > w ? (npg - w + kAttnWaves - 1) / kAttnWaves : 0;
    PageRegs<F32> cur, nxt;
    size_t kb, vb;
    bool ok_cur = false, ok_nxt = false;
    if (my_pages > 0) {
        ok_cur = page_base(0, kb, vb);
        load_page<F32>(a.kv_base, kb, vb, lane, cur);
    }
    for (int j = 0; j < my_pages; ++j) {
        const int p = w + kAttnWaves * j;
        if (!F32 && j + 1 < my_pages) {                 // prefetch the next page (bf16 only)
            ok_nxt = page_base(j + 1, kb, vb);
            load_page<F32>(a.kv_base, kb, vb, lane, nxt);
        }
        float sc[8];
        float pm = -INFINITY;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            float kv[8];
            unpack8<F32>(cur, false, i, kv);
            float t = 0.f;
#pragma unroll
            for (int d = 0; d < 8; ++d) t = fmaf(q[d], kv[d], t);
            t = group_sum<8>(t);
            const int tok = p * kPage + i * 8 + grp;
            sc[i] = (ok_cur && tok < ctx) ? t : -INFINITY;
            pm = fmaxf(pm, sc[i]);
        }
        pm = stride8_max(pm);
        if (pm > -INFINITY) {
            const float mn = fmaxf(m, pm);
            const float alpha = expf(m - mn);          // 0 on this wave's first valid page
            m = mn;
            l *= alpha;
#pragma unroll
            for (int d = 0; d < 8; ++d) o[d] *= alpha;
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                // Slots past the context (or of an invalid page) hold whatever the pool
                // held: keep them out of the sum (0 * NaN would poison it).
                if (sc[i] > -INFINITY) {
                    const float pr = expf(sc[i] - m);
                    float vv[8];
                    unpack8<F32>(cur, true, i, vv);
                    l += pr;
#pragma unroll
                    for (int d = 0; d < 8; ++d) o[d] = fmaf(pr, vv[d], o[d]);
                }
            }
        }
        if (j + 1 < my_pages) {
            if constexpr (F32) {
                ok_cur = page_base(j + 1, kb, vb);
                load_page<F32>(a.kv_base, kb, vb, lane, cur);
            } else {
                cur = nxt;
                ok_cur = ok_nxt;
            }
        }
    }
    // Sum over the 8 token groups (lanes with equal l % 8 hold the same dims).
#pragma unroll
    for (int d = 0; d < 8; ++d) o[d] = stride8_sum(o[d]);
    l = stride8_sum(l);
    if (lane < 8) {
#pragma unroll
        for (int d = 0; d < 8; ++d) s_o[w][lane * 8 + d] = o[d];
    }
    if (lane == 0) {
        s_m[w] = m;
        s_l[w] = l;
    }
    __syncthreads();
    if (tid < kHeadDim) {                               // log-sum-exp merge of the wave partials
        float M = -INFINITY;
#pragma unroll
        for (int i = 0; i < kAttnWaves; ++i) M = fmaxf(M, s_m[i]);
        float L = 0.f, acc = 0.f;
#pragma unroll
        for (int i = 0; i < kAttnWaves; ++i) {
            if (s_m[i] > -INFINITY) {
                const float wgt = expf(s_m[i] - M);
                L = fmaf(s_l[i], wgt, L);
                acc = fmaf(s_o[i][tid], wgt, acc);
            }
        }
        const float r = L > 0.f ? acc / L : 0.f;
        if (out16) out16[tid] = f32_to_bf16(r);
        else out[tid] = r;
    }
}

// 16-bit KV cache.  Same walk and merge as above with a register budget that lets
// two workgroups share a CU (at most 128 VGPRs): a page's K and V live in one set
// of registers each, and the next page's K is requested as soon as the scores are
// formed, its V as soon as the products are accumulated.  The activity flag, the
// length, this wave's page ids and the query are requested together at the start
// (nothing waits for the flag).  Scores use bf16 pair dot products against the
// query split into hi + lo bf16 halves (about 16 significant bits), in the exp2
// domain (query prescaled by 1/sqrt(64) * log2 e).
__device__ __forceinline__ float dot8_bf16(const uint4 k, const uint32_t (&hi)[4], const uint32_t (&lo)[4], float t) {
    typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
    const uint32_t kw[4] = {k.x, k.y, k.z, k.w};
#pragma unroll
    for (int e = 0; e < 4; ++e)
        t = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, kw[e]), __builtin_bit_cast(bf16x2, lo[e]), t,
                                            false);
#pragma unroll
    for (int e = 0; e < 4; ++e)
        t = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, kw[e]), __builtin_bit_cast(bf16x2, hi[e]), t,
                                            false);
    return t;
}

__device__ __forceinline__ void load_half_page(const uint16_t* base, size_t off, int lane, uint4 (&r)[8]) {
    const uint4* p = reinterpret_cast<const uint4*>(base + off);
#pragma unroll
    for (int i = 0; i < 8; ++i) r[i] = p[i * 64 + lane];
}

__global__ __launch_bounds__(kAttnWaves * 64, 4) void attn_decode_bf16_kernel(const AttnDecodeArgs a) {
    __shared__ float s_m[kAttnWaves], s_l[kAttnWaves];
    __shared__ float s_o[kAttnWaves][kHeadDim];
    const int h = blockIdx.x, b = blockIdx.y;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const int grp = lane >> 3, sub = lane & 7;
    const uint16_t* kvb = reinterpret_cast<const uint16_t*>(a.kv_base);
    // independent loads, all in flight together
    const int act = a.active[b];
    const int len = a.seq_lens[b];
    const int lp = w + kAttnWaves * lane;  // lane j: logical page w + 8 j
    const int phys_l = a.block_table[(size_t)b * a.max_pages + min(lp, a.max_pages - 1)];
    const float4* qp = reinterpret_cast<const float4*>(a.qkv + (size_t)b * a.qkv_stride + h * kHeadDim + sub * 8);
    const float4 qa = qp[0], qb = qp[1];

    const int ctx = act ? len + 1 : 0;      // cached slots incl. the new token
    const int npg = (ctx + kPage - 1) / kPage;
    const int my_pages = npg > w ? (npg - w + kAttnWaves - 1) / kAttnWaves : 0;
    uint32_t qh[4], ql[4];
    {
        const float kScale = 0.125f * 1.44269504088896340736f;
        const float qv[8] = {qa.x, qa.y, qa.z, qa.w, qb.x, qb.y, qb.z, qb.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float x0 = qv[2 * e] * kScale, x1 = qv[2 * e + 1] * kScale;
            const uint16_t h0 = f32_to_bf16(x0), h1 = f32_to_bf16(x1);
            qh[e] = (uint32_t)h0 | ((uint32_t)h1 << 16);
            ql[e] = (uint32_t)f32_to_bf16(x0 - bf16_to_f32(h0)) | ((uint32_t)f32_to_bf16(x1 - bf16_to_f32(h1)) << 16);
        }
    }
    auto page_off = [&](int j, int kv, bool& ok) {
        int phys = __shfl(phys_l, j, kWave);
        ok = phys >= 0 && phys < a.n_pages;
        phys = ok ? phys : 0;
        return kv_offset(a.layer, a.n_pages, phys, kv, a.n_head, h, 0);
    };
    float m = -INFINITY, l = 0.f, o[8];
#pragma unroll
    for (int d = 0; d < 8; ++d) o[d] = 0.f;
    uint4 K[8], V[8];
    bool ok_k = false, ok_v = false;
    if (my_pages > 0) {
        load_half_page(kvb, page_off(0, 0, ok_k), lane, K);
        load_half_page(kvb, page_off(0, 1, ok_v), lane, V);
    }
    for (int j = 0; j < my_pages; ++j) {
        const int p = w + kAttnWaves * j;
        const bool ok = ok_k;
        float sc[8];
        float pm = -INFINITY;
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const float t = group_sum<8>(dot8_bf16(K[i], qh, ql, 0.f));
            const int tok = p * kPage + i * 8 + grp;
            sc[i] = (ok && tok < ctx) ? t : -INFINITY;
            pm = fmaxf(pm, sc[i]);
        }
        if (j + 1 < my_pages) load_half_page(kvb, page_off(j + 1, 0, ok_k), lane, K);
        pm = stride8_max(pm);
        if (pm > -INFINITY) {
            const float mn = fmaxf(m, pm);
            const float alpha = exp2f(m - mn);  // 0 on this wave's first valid page
            m = mn;
            l *= alpha;
#pragma unroll
            for (int d = 0; d < 8; ++d) o[d] *= alpha;
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                // slots past the context (or of an invalid page) may hold anything:
                // keep them out of the sum (0 * NaN would poison it)
                if (sc[i] > -INFINITY) {
                    const float pr = exp2f(sc[i] - m);
                    float vv[8];
                    vv[0] = bf16lo(V[i].x); vv[1] = bf16hi(V[i].x); vv[2] = bf16lo(V[i].y); vv[3] = bf16hi(V[i].y);
                    vv[4] = bf16lo(V[i].z); vv[5] = bf16hi(V[i].z); vv[6] = bf16lo(V[i].w); vv[7] = bf16hi(V[i].w);
                    l += pr;
#pragma unroll
                    for (int d = 0; d < 8; ++d) o[d] = fmaf(pr, vv[d], o[d]);
                }
            }
        }
        if (j + 1 < my_pages) load_half_page(kvb, page_off(j + 1, 1, ok_v), lane, V);
    }
#pragma unroll
    for (int d = 0; d < 8; ++d) o[d] = stride8_sum(o[d]);
    l = stride8_sum(l);
    if (lane < 8) {
#pragma unroll
        for (int d = 0; d < 8; ++d) s_o[w][lane * 8 + d] = o[d];
    }
    if (lane == 0) {
        s_m[w] = m;
        s_l[w] = l;
    }
    __syncthreads();
    if (tid < kHeadDim) {                   // log-sum-exp merge of the wave partials (exp2 domain)
        float M = -INFINITY;
#pragma unroll
        for (int i = 0; i < kAttnWaves; ++i) M = fmaxf(M, s_m[i]);
        float L = 0.f, acc = 0.f;
#pragma unroll
        for (int i = 0; i < kAttnWaves; ++i) {
            if (s_m[i] > -INFINITY) {
                const float wgt = exp2f(s_m[i] - M);
                L = fmaf(s_l[i], wgt, L);
                acc = fmaf(s_o[i][tid], wgt, acc);
            }
        }
        const float r = L > 0.f ? acc / L : 0.f;
        const size_t oi = (size_t)b * a.o_stride + h * kHeadDim + tid;
        if (a.o_bf16) a.o_bf16[oi] = f32_to_bf16(r);
        else a.o[oi] = r;
    }
}

hipError_t launch_attn_decode(int wdtype, const AttnDecodeArgs& a, int B, hipStream_t st) {
    const dim3 g(a.n_head, B);
    if (wdtype == FTTS_F32) hipLaunchKernelGGL(attn_decode_kernel<true>, g, dim3(kAttnWaves * 64), 0, st, a);
    else hipLaunchKernelGGL(attn_decode_bf16_kernel, g, dim3(kAttnWaves * 64), 0, st, a);
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

typedef __bf16 pf_bf16x8 __attribute__((ext_vector_type(8)));
typedef float pf_f32x16 __attribute__((ext_vector_type(16)));
constexpr int kPfWaves = 4, kPfQ = kPfWaves * 32;  // queries per workgroup
constexpr int kPfK = 32;                           // keys per tile
constexpr int kVtStride = kPfK + 8;                // bf16 per transposed-V row (one head dim)

__device__ __forceinline__ pf_bf16x8 pf_op(uint4 v) { return __builtin_bit_cast(pf_bf16x8, v); }

__global__ __launch_bounds__(kPfWaves * 64) void attn_prefill_mfma_kernel(const AttnPrefillArgs a) {
    __shared__ __attribute__((aligned(16))) uint16_t vt[2][kHeadDim][kVtStride];
    const int h = blockIdx.y, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    int gt = blockIdx.x, sq = 0;
    while (sq + 1 < a.seqs.n && a.tiles_cu[sq + 1] <= gt) ++sq;
    const int tile = gt - a.tiles_cu[sq];
    const int row0 = a.seqs.cu[sq], len = a.seqs.cu[sq + 1] - row0;
    if (len <= 0) return;
    const size_t ld = 3 * (size_t)a.d_model;
    const uint16_t* qkv = reinterpret_cast<const uint16_t*>(a.qkv);
    const int ql = lane & 31, hh = lane >> 5;
    const int qw = tile * kPfQ + wave * 32;  // this wave's first query
    const int qi = qw + ql;                  // this lane's query (a column of S^T)
    // exp2 domain: scores scaled by 1/sqrt(64) * log2(e)
    const float kScale = 0.125f * 1.44269504088896340736f;

    // Q as the B operand of S^T = K Q^T: lane (q, hh) holds dims kk*16 + hh*8 .. +7.
    uint4 qr[4];
    {
        const uint16_t* qrow = qkv + (size_t)(row0 + min(qi, len - 1)) * ld + h * kHeadDim;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) qr[kk] = *reinterpret_cast<const uint4*>(qrow + kk * 16 + hh * 8);
    }
    // V tile staging: thread t carries key t / 8, dims (t % 8) * 8 .. +7.
    const int vkey = tid >> 3, vd0 = (tid & 7) * 8;
    auto load_v = [&](int t) {
        const int key = min(t * kPfK + vkey, len - 1);
        return *reinterpret_cast<const uint4*>(qkv + (size_t)(row0 + key) * ld + 2 * a.d_model + h * kHeadDim + vd0);
    };
    auto store_v = [&](uint4 v, int buf) {
        const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            vt[buf][vd0 + 2 * i][vkey] = (uint16_t)(w[i] & 0xFFFFu);
            vt[buf][vd0 + 2 * i + 1][vkey] = (uint16_t)(w[i] >> 16);
        }
    };

    pf_f32x16 o0, o1;  // O^T, dims 0..31 and 32..63: o[i] is dim (i/4)*8 + hh*4 + i%4 of query qi
#pragma unroll
    for (int i = 0; i < 16; ++i) o0[i] = o1[i] = 0.f;
    float m = -INFINITY, l = 0.f;
    const int kend = min(len, tile * kPfQ + kPfQ);  // keys any query of this workgroup sees
    const int ntiles = (kend + kPfK - 1) / kPfK;
    store_v(load_v(0), 0);
    __syncthreads();
    for (int t = 0; t < ntiles; ++t) {
        const int buf = t & 1, k0 = t * kPfK;
        uint4 vnext = make_uint4(0, 0, 0, 0);
        if (t + 1 < ntiles) vnext = load_v(t + 1);
        if (k0 <= qw + 31 && qw < len) {  // some query of this wave sees a key of this tile
            // K as the A operand: lane (key k0 + ql, hh) holds dims kk*16 + hh*8 .. +7
            const uint16_t* krow = qkv + (size_t)(row0 + min(k0 + ql, len - 1)) * ld + a.d_model + h * kHeadDim;
            uint4 kr[4];
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) kr[kk] = *reinterpret_cast<const uint4*>(krow + kk * 16 + hh * 8);
            pf_f32x16 s;
#pragma unroll
            for (int i = 0; i < 16; ++i) s[i] = 0.f;
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(pf_op(kr[kk]), pf_op(qr[kk]), s, 0, 0, 0);
            // s[i]: key k0 + (i/4)*8 + hh*4 + i%4 of query qi; causal and length masks
            float tmax = -INFINITY;
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int key = k0 + (i >> 2) * 8 + hh * 4 + (i & 3);
                s[i] = key <= qi && key < len ? s[i] * kScale : -INFINITY;
                tmax = fmaxf(tmax, s[i]);
            }
            {
                const RowPair pr = swap32(tmax);  // the other 16 keys of this query
                tmax = fmaxf(pr.a, pr.b);
            }
            const float mn = fmaxf(m, tmax);
            const float ms = mn == -INFINITY ? 0.f : mn;
            const float alpha = exp2f(m - ms);
            m = mn;
            // probabilities, rounded to bf16 once: the same values feed P V and the row sum
            uint32_t pw[8];
            float rs = 0.f;
#pragma unroll
            for (int i = 0; i < 16; i += 2) {
                const uint16_t lo = f32_to_bf16(exp2f(s[i] - ms)), hi = f32_to_bf16(exp2f(s[i + 1] - ms));
                rs += bf16_to_f32(lo) + bf16_to_f32(hi);
                pw[i / 2] = (uint32_t)lo | ((uint32_t)hi << 16);
            }
            {
                const RowPair pr = swap32(rs);
                rs = pr.a + pr.b;
            }
            l = l * alpha + rs;
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                o0[i] *= alpha;
                o1[i] *= alpha;
            }
            // O^T += V^T P^T.  k slots hh*8 .. +7 of step st carry keys
            // st*16 + hh*4 + 0..3 and st*16 + 8 + hh*4 + 0..3 on both operands.
#pragma unroll
            for (int st2 = 0; st2 < 2; ++st2) {
                const pf_bf16x8 pb = pf_op(make_uint4(pw[4 * st2], pw[4 * st2 + 1], pw[4 * st2 + 2], pw[4 * st2 + 3]));
                const int c = st2 * 16 + hh * 4;
                const uint2 a0 = *reinterpret_cast<const uint2*>(&vt[buf][ql][c]);
                const uint2 a1 = *reinterpret_cast<const uint2*>(&vt[buf][ql][c + 8]);
                const uint2 b0 = *reinterpret_cast<const uint2*>(&vt[buf][32 + ql][c]);
                const uint2 b1 = *reinterpret_cast<const uint2*>(&vt[buf][32 + ql][c + 8]);
                o0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(pf_op(make_uint4(a0.x, a0.y, a1.x, a1.y)), pb, o0, 0, 0, 0);
                o1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(pf_op(make_uint4(b0.x, b0.y, b1.x, b1.y)), pb, o1, 0, 0, 0);
            }
        }
        if (t + 1 < ntiles) store_v(vnext, buf ^ 1);  // that buffer was last read before the previous barrier
        __syncthreads();
    }
    if (qi >= len) return;
    const float inv = 1.0f / l;
    uint16_t* orow = reinterpret_cast<uint16_t*>(a.o) + (size_t)(row0 + qi) * a.d_model + h * kHeadDim;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
        const int dd = g * 8 + hh * 4;
        *reinterpret_cast<uint2*>(orow + dd) =
            make_uint2((uint32_t)f32_to_bf16(o0[4 * g] * inv) | ((uint32_t)f32_to_bf16(o0[4 * g + 1] * inv) << 16),
                       (uint32_t)f32_to_bf16(o0[4 * g + 2] * inv) | ((uint32_t)f32_to_bf16(o0[4 * g + 3] * inv) << 16));
        *reinterpret_cast<uint2*>(orow + 32 + dd) =
            make_uint2((uint32_t)f32_to_bf16(o1[4 * g] * inv) | ((uint32_t)f32_to_bf16(o1[4 * g + 1] * inv) << 16),
                       (uint32_t)f32_to_bf16(o1[4 * g + 2] * inv) | ((uint32_t)f32_to_bf16(o1[4 * g + 3] * inv) << 16));
    }
}

// Attention without a mask (every query sees every key of its sequence), bf16,
// for short grids.  A workgroup takes 32 queries of one head; its 4 waves split
// the 32-key tiles round-robin (wave w takes tiles w, w + 4, ...), so a
// sequence of L keys keeps ceil(L / 32) * 4 waves busy per head and each wave's
// dependent chain is a quarter of the keys.  Every wave forms S^T = K Q^T and
// O^T = V^T P^T as in the prefill kernel, transposes its own V tile through a
// private LDS slice (no workgroup barrier in the loop) and prefetches the next
// tile's K and V rows into registers.  The four (max, sum, output) partials are
// merged by the log-sum-exp rule through LDS at the end.
constexpr int kFaWaves = 4, kFaQ = 32, kFaK = 32;
typedef __bf16 fa_bf16x2 __attribute__((ext_vector_type(2)));
typedef float fa_f32x2 __attribute__((ext_vector_type(2)));

// Two floats to packed bf16 (round to nearest even, one instruction).
__device__ __forceinline__ uint32_t fa_pack_bf16(float lo, float hi) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((fa_f32x2){lo, hi}, fa_bf16x2));
}

__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Workgroups are dealt to the 8 XCDs round-robin by linear id.  Give each XCD a
// contiguous run of (head, query tile) pairs, query tiles fastest, so the query
// tiles of one (sequence, head) share an XCD and its K and V rows are fetched
// into one L2 (used by the wide-grid kernel; measured neutral-to-worse for the
// key-split one, whose query tiles each read all keys anyway).
struct FaTile { int tile, head; };
__device__ __forceinline__ FaTile fa_tile() {
    const int T = gridDim.x * gridDim.y, b = blockIdx.y * gridDim.x + blockIdx.x;
    const int x = b & 7, l = b >> 3, q = T >> 3, r = T & 7;
    const int t = (x < r ? x * (q + 1) : r * (q + 1) + (x - r) * q) + l;
    return FaTile{(int)(t % gridDim.x), (int)(t / gridDim.x)};
}

// CAUSAL: the prefill's masked form -- query tile j sees key tiles 0 .. j only,
// and in tile j (keys and queries aligned, 32 each) key k only for queries >= k.
template <bool CAUSAL>
__global__ __launch_bounds__(kFaWaves * 64, 3) void attn_full_mfma_kernel(const AttnPrefillArgs a) {
    __shared__ __attribute__((aligned(16))) uint16_t vt[kFaWaves][kHeadDim][kVtStride];
    __shared__ float mrg[kFaWaves - 1][34][64];  // waves 1..3: 32 output values, max, sum per lane
    const int h = blockIdx.y, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    int gt = blockIdx.x, sq = 0;
    while (sq + 1 < a.seqs.n && a.tiles_cu[sq + 1] <= gt) ++sq;
    const int tile = gt - a.tiles_cu[sq];
    const int row0 = a.seqs.cu[sq], len = a.seqs.cu[sq + 1] - row0;
    if (len <= 0) return;  // uniform over the workgroup
    const size_t ld = 3 * (size_t)a.d_model;
    const uint16_t* qkv = reinterpret_cast<const uint16_t*>(a.qkv);
    const int ql = lane & 31, hh = lane >> 5;
    const int qi = tile * kFaQ + ql;
    const float kScale = 0.125f * 1.44269504088896340736f;  // 1/sqrt(64) * log2(e)

    uint4 qr[4];
    {
        const uint16_t* qrow = qkv + (size_t)(row0 + min(qi, len - 1)) * ld + h * kHeadDim;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) qr[kk] = *reinterpret_cast<const uint4*>(qrow + kk * 16 + hh * 8);
    }
    // V staging: lane l carries keys 2p, 2p + 1 (p = l % 16) of the tile, dims g*16 .. +15 (g = l / 16)
    const int vp = lane & 15, vg = lane >> 4;
    auto load_k = [&](int t, uint4 (&kr)[4]) {
        const uint16_t* krow = qkv + (size_t)(row0 + min(t * kFaK + ql, len - 1)) * ld + a.d_model + h * kHeadDim;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) kr[kk] = *reinterpret_cast<const uint4*>(krow + kk * 16 + hh * 8);
    };
    auto load_v = [&](int t, uint4 (&vr)[4]) {
#pragma unroll
        for (int e = 0; e < 2; ++e) {
            const int key = min(t * kFaK + 2 * vp + e, len - 1);
            const uint16_t* vrow = qkv + (size_t)(row0 + key) * ld + 2 * a.d_model + h * kHeadDim + vg * 16;
            vr[2 * e] = *reinterpret_cast<const uint4*>(vrow);
            vr[2 * e + 1] = *reinterpret_cast<const uint4*>(vrow + 8);
        }
    };
    static_assert(kFaK == kFaQ, "the causal diagonal is one key tile");
    const int kend = CAUSAL ? min(len, tile * kFaQ + kFaQ) : len;  // keys any query of the tile sees
    const int nt = (kend + kFaK - 1) / kFaK;
    const int t0 = wave;

    pf_f32x16 o0, o1;
#pragma unroll
    for (int i = 0; i < 16; ++i) o0[i] = o1[i] = 0.f;
    float m = -INFINITY, l = 0.f;
    uint4 kr[4], vr[4];
    if (t0 < nt) {
        load_k(t0, kr);
        load_v(t0, vr);
    }
    for (int t = t0; t < nt; t += kFaWaves) {
        // V^T of this tile into the wave's LDS slice: one 32-bit word = two keys of one dim
        const uint32_t w0[8] = {vr[0].x, vr[0].y, vr[0].z, vr[0].w, vr[1].x, vr[1].y, vr[1].z, vr[1].w};
        const uint32_t w1[8] = {vr[2].x, vr[2].y, vr[2].z, vr[2].w, vr[3].x, vr[3].y, vr[3].z, vr[3].w};
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            const uint32_t lo = (j & 1) ? (w0[j >> 1] >> 16) : (w0[j >> 1] & 0xFFFFu);
            const uint32_t hi = (j & 1) ? (w1[j >> 1] >> 16) : (w1[j >> 1] & 0xFFFFu);
            *reinterpret_cast<uint32_t*>(&vt[wave][vg * 16 + j][2 * vp]) = lo | (hi << 16);
        }
        uint4 kc[4];
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) kc[kk] = kr[kk];
        if (t + kFaWaves < nt) {  // next tile's rows, in flight during this one
            load_k(t + kFaWaves, kr);
            load_v(t + kFaWaves, vr);
        }
        const int k0 = t * kFaK;
        pf_f32x16 s;
#pragma unroll
        for (int i = 0; i < 16; ++i) s[i] = 0.f;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(pf_op(kc[kk]), pf_op(qr[kk]), s, 0, 0, 0);
        // raw scores; keys past the end exist only in a sequence's last tile, and
        // (causal) keys after the query only in the diagonal tile, whose first key
        // every query of the tile sees
        if (k0 + kFaK > len || (CAUSAL && t == tile)) {
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int key = k0 + (i >> 2) * 8 + hh * 4 + (i & 3);
                if (key >= len || (CAUSAL && key > qi)) s[i] = -INFINITY;
            }
        }
        float tmax = s[0];
#pragma unroll
        for (int i = 1; i < 16; ++i) tmax = fmaxf(tmax, s[i]);
        {
            const RowPair pr = swap32(tmax);
            tmax = fmaxf(pr.a, pr.b);
        }
        const float mn = fmaxf(m, tmax * kScale);  // finite: key k0 < len is in this tile
        // probabilities exp2(s * scale - max) (arguments <= 0; the hardware exp2 flushes
        // results below 2^-126 to 0), rounded to bf16 once: the same values feed P V
        // and the row sum
        uint32_t pw[8];
        float rs = 0.f;
#pragma unroll
        for (int i = 0; i < 16; i += 2) {
            pw[i / 2] = fa_pack_bf16(__builtin_amdgcn_exp2f(fmaf(s[i], kScale, -mn)),
                                     __builtin_amdgcn_exp2f(fmaf(s[i + 1], kScale, -mn)));
            rs += __uint_as_float(pw[i / 2] << 16) + __uint_as_float(pw[i / 2] & 0xFFFF0000u);
        }
        {
            const RowPair pr = swap32(rs);
            rs = pr.a + pr.b;
        }
        // rescale the running sums only when some lane's maximum grew (alpha = 1 elsewhere)
        if (__any(mn > m)) {
            const float alpha = __builtin_amdgcn_exp2f(m - mn);  // m = -inf on the first tile: 0
            l *= alpha;
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                o0[i] *= alpha;
                o1[i] *= alpha;
            }
        }
        m = mn;
        l += rs;
        wave_lds_sync();  // the V^T words of every lane are in LDS
#pragma unroll
        for (int st2 = 0; st2 < 2; ++st2) {
            const pf_bf16x8 pb = pf_op(make_uint4(pw[4 * st2], pw[4 * st2 + 1], pw[4 * st2 + 2], pw[4 * st2 + 3]));
            const int c = st2 * 16 + hh * 4;
            const uint2 a0 = *reinterpret_cast<const uint2*>(&vt[wave][ql][c]);
            const uint2 a1 = *reinterpret_cast<const uint2*>(&vt[wave][ql][c + 8]);
            const uint2 b0 = *reinterpret_cast<const uint2*>(&vt[wave][32 + ql][c]);
            const uint2 b1 = *reinterpret_cast<const uint2*>(&vt[wave][32 + ql][c + 8]);
            o0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(pf_op(make_uint4(a0.x, a0.y, a1.x, a1.y)), pb, o0, 0, 0, 0);
            o1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(pf_op(make_uint4(b0.x, b0.y, b1.x, b1.y)), pb, o1, 0, 0, 0);
        }
        wave_lds_sync();  // every lane has read the slice before the next tile overwrites it
    }
    // merge: waves 1..3 hand (o, m, l) to wave 0 lane for lane
    if (wave > 0) {
        float* mw = &mrg[wave - 1][0][0];
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            mw[i * 64 + lane] = o0[i];
            mw[(16 + i) * 64 + lane] = o1[i];
        }
        mw[32 * 64 + lane] = m;
        mw[33 * 64 + lane] = l;
    }
    __syncthreads();
    if (wave > 0 || qi >= len) return;
    // wave 0 always holds tile 0, so m is finite; an idle wave has m = -inf, l = 0, o = 0
    float mm = m;
#pragma unroll
    for (int w = 0; w < kFaWaves - 1; ++w) mm = fmaxf(mm, mrg[w][32][lane]);
    float sc = exp2f(m - mm);
    l *= sc;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        o0[i] *= sc;
        o1[i] *= sc;
    }
#pragma unroll
    for (int w = 0; w < kFaWaves - 1; ++w) {
        const float f = exp2f(mrg[w][32][lane] - mm);
        l += mrg[w][33][lane] * f;
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            o0[i] += mrg[w][i][lane] * f;
            o1[i] += mrg[w][16 + i][lane] * f;
        }
    }
    const float inv = 1.0f / l;
    uint16_t* orow = reinterpret_cast<uint16_t*>(a.o) + (size_t)(row0 + qi) * a.d_model + h * kHeadDim;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
        const int dd = g * 8 + hh * 4;
        *reinterpret_cast<uint2*>(orow + dd) =
            make_uint2((uint32_t)f32_to_bf16(o0[4 * g] * inv) | ((uint32_t)f32_to_bf16(o0[4 * g + 1] * inv) << 16),
                       (uint32_t)f32_to_bf16(o0[4 * g + 2] * inv) | ((uint32_t)f32_to_bf16(o0[4 * g + 3] * inv) << 16));
        *reinterpret_cast<uint2*>(orow + 32 + dd) =
            make_uint2((uint32_t)f32_to_bf16(o1[4 * g] * inv) | ((uint32_t)f32_to_bf16(o1[4 * g + 1] * inv) << 16),
                       (uint32_t)f32_to_bf16(o1[4 * g + 2] * inv) | ((uint32_t)f32_to_bf16(o1[4 * g + 3] * inv) << 16));
    }
}

// The same attention for wide grids: the 4 waves of a workgroup take 128
// consecutive queries (32 each) and share every 32-key tile, which all 256
// threads stage once into double-buffered LDS (K as rows, V transposed), one
// workgroup barrier per tile.  Each K and V row is read from L2 once per 128
// queries instead of once per 32, the bound of the per-wave kernel above.
constexpr int kFsK = kHeadDim + 8;  // bf16 per K row in LDS (16-byte aligned, staggered banks)

__global__ __launch_bounds__(kFaWaves * 64, 2) void attn_full_shared_kernel(const AttnPrefillArgs a) {
    __shared__ __attribute__((aligned(16))) uint16_t ks[2][kFaK][kFsK];
    __shared__ __attribute__((aligned(16))) uint16_t vs[2][kHeadDim][kVtStride];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const FaTile ft = fa_tile();
    const int h = ft.head;
    int gt = ft.tile, sq = 0;
    while (sq + 1 < a.seqs.n && a.tiles_cu[sq + 1] <= gt) ++sq;
    const int tile = gt - a.tiles_cu[sq];
    const int row0 = a.seqs.cu[sq], len = a.seqs.cu[sq + 1] - row0;
    if (len <= 0) return;  // uniform over the workgroup
    const size_t ld = 3 * (size_t)a.d_model;
    const uint16_t* qkv = reinterpret_cast<const uint16_t*>(a.qkv);
    const int ql = lane & 31, hh = lane >> 5;
    const int qi = tile * (kFaWaves * kFaQ) + wave * kFaQ + ql;  // past len: computed, not stored
    const float kScale = 0.125f * 1.44269504088896340736f;

    uint4 qr[4];
    {
        const uint16_t* qrow = qkv + (size_t)(row0 + min(qi, len - 1)) * ld + h * kHeadDim;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) qr[kk] = *reinterpret_cast<const uint4*>(qrow + kk * 16 + hh * 8);
    }
    // staging: thread t carries key t / 8, dims (t % 8) * 8 .. +7 of both K and V
    const int skey = tid >> 3, sd0 = (tid & 7) * 8;
    auto load_kv = [&](int t, uint4& kv, uint4& vv) {
        const uint16_t* r = qkv + (size_t)(row0 + min(t * kFaK + skey, len - 1)) * ld + h * kHeadDim + sd0;
        kv = *reinterpret_cast<const uint4*>(r + a.d_model);
        vv = *reinterpret_cast<const uint4*>(r + 2 * a.d_model);
    };
    auto store_kv = [&](const uint4& kv, const uint4& vv, int buf) {
        *reinterpret_cast<uint4*>(&ks[buf][skey][sd0]) = kv;
        const uint32_t w[4] = {vv.x, vv.y, vv.z, vv.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            vs[buf][sd0 + 2 * i][skey] = (uint16_t)(w[i] & 0xFFFFu);
            vs[buf][sd0 + 2 * i + 1][skey] = (uint16_t)(w[i] >> 16);
        }
    };
    const int nt = (len + kFaK - 1) / kFaK;
    pf_f32x16 o0, o1;
#pragma unroll
    for (int i = 0; i < 16; ++i) o0[i] = o1[i] = 0.f;
    float m = -INFINITY, l = 0.f;
    {
        uint4 kv, vv;
        load_kv(0, kv, vv);
        store_kv(kv, vv, 0);
    }
    __syncthreads();
    for (int t = 0; t < nt; ++t) {
        const int buf = t & 1, k0 = t * kFaK;
        uint4 kn = make_uint4(0, 0, 0, 0), vn = make_uint4(0, 0, 0, 0);
        if (t + 1 < nt) load_kv(t + 1, kn, vn);  // in flight during this tile
        uint4 kc[4];
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) kc[kk] = *reinterpret_cast<const uint4*>(&ks[buf][ql][kk * 16 + hh * 8]);
        pf_f32x16 s;
#pragma unroll
        for (int i = 0; i < 16; ++i) s[i] = 0.f;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(pf_op(kc[kk]), pf_op(qr[kk]), s, 0, 0, 0);
        if (k0 + kFaK > len) {
#pragma unroll
            for (int i = 0; i < 16; ++i)
                if (k0 + (i >> 2) * 8 + hh * 4 + (i & 3) >= len) s[i] = -INFINITY;
        }
        float tmax = s[0];
#pragma unroll
        for (int i = 1; i < 16; ++i) tmax = fmaxf(tmax, s[i]);
        {
            const RowPair pr = swap32(tmax);
            tmax = fmaxf(pr.a, pr.b);
        }
        const float mn = fmaxf(m, tmax * kScale);
        uint32_t pw[8];
        float rs = 0.f;
#pragma unroll
        for (int i = 0; i < 16; i += 2) {
            pw[i / 2] = fa_pack_bf16(__builtin_amdgcn_exp2f(fmaf(s[i], kScale, -mn)),
                                     __builtin_amdgcn_exp2f(fmaf(s[i + 1], kScale, -mn)));
            rs += __uint_as_float(pw[i / 2] << 16) + __uint_as_float(pw[i / 2] & 0xFFFF0000u);
        }
        {
            const RowPair pr = swap32(rs);
            rs = pr.a + pr.b;
        }
        if (__any(mn > m)) {
            const float alpha = __builtin_amdgcn_exp2f(m - mn);
            l *= alpha;
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                o0[i] *= alpha;
                o1[i] *= alpha;
            }
        }
        m = mn;
        l += rs;
#pragma unroll
        for (int st2 = 0; st2 < 2; ++st2) {
            const pf_bf16x8 pb = pf_op(make_uint4(pw[4 * st2], pw[4 * st2 + 1], pw[4 * st2 + 2], pw[4 * st2 + 3]));
            const int c = st2 * 16 + hh * 4;
            const uint2 a0 = *reinterpret_cast<const uint2*>(&vs[buf][ql][c]);
            const uint2 a1 = *reinterpret_cast<const uint2*>(&vs[buf][ql][c + 8]);
            const uint2 b0 = *reinterpret_cast<const uint2*>(&vs[buf][32 + ql][c]);
            const uint2 b1 = *reinterpret_cast<const uint2*>(&vs[buf][32 + ql][c + 8]);
            o0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(pf_op(make_uint4(a0.x, a0.y, a1.x, a1.y)), pb, o0, 0, 0, 0);
            o1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(pf_op(make_uint4(b0.x, b0.y, b1.x, b1.y)), pb, o1, 0, 0, 0);
        }
        if (t + 1 < nt) store_kv(kn, vn, buf ^ 1);  // that buffer was last read before the previous barrier
        __syncthreads();
    }
    if (qi >= len) return;
    const float inv = 1.0f / l;
    uint16_t* orow = reinterpret_cast<uint16_t*>(a.o) + (size_t)(row0 + qi) * a.d_model + h * kHeadDim;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
        const int dd = g * 8 + hh * 4;
        *reinterpret_cast<uint2*>(orow + dd) = make_uint2(fa_pack_bf16(o0[4 * g] * inv, o0[4 * g + 1] * inv),
                                                          fa_pack_bf16(o0[4 * g + 2] * inv, o0[4 * g + 3] * inv));
        *reinterpret_cast<uint2*>(orow + 32 + dd) = make_uint2(fa_pack_bf16(o1[4 * g] * inv, o1[4 * g + 1] * inv),
                                                               fa_pack_bf16(o1[4 * g + 2] * inv, o1[4 * g + 3] * inv));
    }
}

int prefill_tile_rows(int wdtype) { return wdtype == FTTS_F32 ? 64 : kPfQ; }

hipError_t launch_attn_prefill(int wdtype, const AttnPrefillArgs& a, int total_tiles, hipStream_t st) {
    if (wdtype == FTTS_F32) {
        hipLaunchKernelGGL(attn_prefill_kernel<true>, dim3(total_tiles, a.n_head), dim3(64), 0, st, a);
        return hipGetLastError();
    }
    // 128-query tiles sharing each key tile once they give at least one workgroup
    // per compute unit, else (short prefixes) 32-query tiles with the keys split
    // over the waves, so a query tile's dependent chain is a quarter of its keys
    constexpr int kFillGroups = 256;
    AttnPrefillArgs b = a;
    auto tiles = [&](int q) {
        b.tiles_cu[0] = 0;
        for (int i = 0; i < a.seqs.n; ++i)
            b.tiles_cu[i + 1] = b.tiles_cu[i] + (a.seqs.cu[i + 1] - a.seqs.cu[i] + q - 1) / q;
        return b.tiles_cu[a.seqs.n];
    };
    const int t128 = tiles(kPfQ);
    if (t128 == 0) return hipSuccess;
    if ((long)t128 * a.n_head >= kFillGroups) {
        hipLaunchKernelGGL(attn_prefill_mfma_kernel, dim3(t128, a.n_head), dim3(kPfWaves * 64), 0, st, b);
    } else {
        const int t32 = tiles(kFaQ);
        hipLaunchKernelGGL(attn_full_mfma_kernel<true>, dim3(t32, a.n_head), dim3(kFaWaves * 64), 0, st, b);
    }
    return hipGetLastError();
}

hipError_t launch_attn_full_bf16(const AttnPrefillArgs& a, hipStream_t st) {
    // 128-query tiles sharing K and V once they give at least one workgroup per
    // compute unit, else 32-query tiles with the keys split over the waves
    constexpr int kFillGroups = 256;
    AttnPrefillArgs b = a;
    auto tiles = [&](int q) {
        b.tiles_cu[0] = 0;
        for (int i = 0; i < a.seqs.n; ++i)
            b.tiles_cu[i + 1] = b.tiles_cu[i] + (a.seqs.cu[i + 1] - a.seqs.cu[i] + q - 1) / q;
        return b.tiles_cu[a.seqs.n];
    };
    const int t128 = tiles(kFaWaves * kFaQ);
    if (t128 == 0) return hipSuccess;
    if ((long)t128 * a.n_head >= kFillGroups) {
        hipLaunchKernelGGL(attn_full_shared_kernel, dim3(t128, a.n_head), dim3(kFaWaves * 64), 0, st, b);
    } else {
        const int t32 = tiles(kFaQ);
        hipLaunchKernelGGL(attn_full_mfma_kernel<false>, dim3(t32, a.n_head), dim3(kFaWaves * 64), 0, st, b);
    }
    return hipGetLastError();
}

}  // namespace ftts
