// Small kernels around the hot path: token+position embedding (with the
// per-row activity flag every later kernel reads), LayerNorm over packed rows
// (prefill), row gathers, the next-token sampler and the weight quantiser.
#include <climits>

#include "ftts_internal.hpp"

namespace ftts {

// ---- embedding ------------------------------------------------------------------------
// x[b] = tok_emb[tokens[b]] + pos_emb[positions[b]] (fp32).  A row is active when
// its token, position, KV slot and page are all in range; inactive rows get x = 0.
template <bool F32>
__global__ __launch_bounds__(256) void embed_kernel(const void* tok_emb, const void* pos_emb, int vocab,
                                                    int n_pos, int d, const int32_t* tokens,
                                                    const int32_t* positions, const int32_t* seq_lens,
                                                    const int32_t* block_table, int max_pages, int n_pages,
                                                    float* x, int32_t* active, float2* stats, uint32_t* zero,
                                                    int n_zero) {
    const int b = blockIdx.x, B = gridDim.x;
    const int t = tokens[b], p = positions[b], s = seq_lens[b];
    bool ok = t >= 0 && t < vocab && p >= 0 && p < n_pos && s >= 0 && s < max_pages * kPage;
    if (ok) {
        const int phys = block_table[(size_t)b * max_pages + s / kPage];
        ok = phys >= 0 && phys < n_pages;
    }
    if (threadIdx.x == 0) active[b] = ok ? 1 : 0;
    for (int i = b * 256 + threadIdx.x; i < n_zero; i += B * 256) zero[i] = 0u;
    float* xr = x + (size_t)b * d;
    // the embedding rows are read at clamped indices without waiting for the page
    // check (the value of an inactive row is dropped)
    const int tc = min(max(t, 0), vocab - 1), pc = min(max(p, 0), n_pos - 1);
    // d is a multiple of 64, so every pass of this loop keeps whole waves active
    for (int k = threadIdx.x; k < d; k += blockDim.x) {
        float v = ld_act<F32>(tok_emb, (size_t)tc * d + k) + ld_act<F32>(pos_emb, (size_t)pc * d + k);
        v = ok ? v : 0.f;
        xr[k] = v;
        if (stats) {
            const float2 ts = tile_stats32(v);
            if ((k & (kStatTile - 1)) == 0) stats[(size_t)(k / kStatTile) * B + b] = ts;
        }
    }
}

hipError_t launch_embed(int wdtype, const void* tok_emb, const void* pos_emb, int vocab, int n_pos, int d,
                        const int32_t* tokens, const int32_t* positions, const int32_t* seq_lens,
                        const int32_t* block_table, int max_pages, int n_pages, int B, float* x,
                        int32_t* active, float2* stats, uint32_t* zero, int n_zero, hipStream_t st) {
    if (stats && d % 64 != 0) return hipErrorInvalidValue;
    if (wdtype == FTTS_F32)
        hipLaunchKernelGGL(embed_kernel<true>, dim3(B), dim3(256), 0, st, tok_emb, pos_emb, vocab, n_pos, d,
                           tokens, positions, seq_lens, block_table, max_pages, n_pages, x, active, stats, zero,
                           n_zero);
    else
        hipLaunchKernelGGL(embed_kernel<false>, dim3(B), dim3(256), 0, st, tok_emb, pos_emb, vocab, n_pos, d,
                           tokens, positions, seq_lens, block_table, max_pages, n_pages, x, active, stats, zero,
                           n_zero);
    return hipGetLastError();
}

// ---- block reductions -------------------------------------------------------------------
__device__ __forceinline__ float block_sum256(float v, float* red) {
    v = wave_sum(v);
    const int w = threadIdx.x >> 6;
    __syncthreads();
    if ((threadIdx.x & 63) == 0) red[w] = v;
    __syncthreads();
    return red[0] + red[1] + red[2] + red[3];
}

// ---- LayerNorm over packed rows (prefill): fp32 x -> activation dtype ----------------------
template <bool F32>
__global__ __launch_bounds__(256) void ln_rows_kernel(const float* x, const void* g, const void* bb, float eps,
                                                      int d, void* out) {
    __shared__ float red[4];
    const size_t r = blockIdx.x;
    const float* xr = x + r * d;
    float s = 0.f;
    for (int k = threadIdx.x; k < d; k += 256) s += xr[k];
    const float mean = block_sum256(s, red) / (float)d;
    float v = 0.f;
    for (int k = threadIdx.x; k < d; k += 256) {
        const float t = xr[k] - mean;
        v = fmaf(t, t, v);
    }
    const float var = block_sum256(v, red) / (float)d;
    const float rstd = 1.0f / sqrtf(var + eps);
    for (int k = threadIdx.x; k < d; k += 256)
        st_act<F32>(out, r * d + k, (xr[k] - mean) * rstd * ld_act<F32>(g, k) + ld_act<F32>(bb, k));
}

// One wave per row for rows of up to 2048 columns that split into float4 lanes:
// the row stays in registers, both reductions are cross-lane, no barriers.
template <bool F32>
__global__ __launch_bounds__(256) void ln_rows_wave_kernel(const float* x, const void* g, const void* bb, float eps,
                                                           int M, int d, void* out) {
    constexpr int NMAX = 8;  // float4 per lane: d <= 64 * 4 * 8
    const int r = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
    if (r >= M) return;
    const float4* xr = reinterpret_cast<const float4*>(x + (size_t)r * d);
    const int n4 = d / 4;
    float4 v[NMAX];
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < NMAX; ++i) {
        const int j = lane + 64 * i;
        v[i] = j < n4 ? xr[j] : make_float4(0.f, 0.f, 0.f, 0.f);
        s += (v[i].x + v[i].y) + (v[i].z + v[i].w);
    }
    const float mean = wave_sum(s) / (float)d;
    float q = 0.f;
#pragma unroll
    for (int i = 0; i < NMAX; ++i) {
        if (lane + 64 * i < n4) {
            const float a = v[i].x - mean, b = v[i].y - mean, c = v[i].z - mean, e = v[i].w - mean;
            q = fmaf(a, a, fmaf(b, b, fmaf(c, c, fmaf(e, e, q))));
        }
    }
    const float rstd = 1.0f / sqrtf(wave_sum(q) / (float)d + eps);
#pragma unroll
    for (int i = 0; i < NMAX; ++i) {
        const int j = lane + 64 * i;
        if (j < n4) {
            const float xs[4] = {v[i].x, v[i].y, v[i].z, v[i].w};
            if constexpr (F32) {
#pragma unroll
                for (int k = 0; k < 4; ++k)
                    st_act<F32>(out, (size_t)r * d + 4 * j + k,
                                (xs[k] - mean) * rstd * ld_act<F32>(g, 4 * j + k) + ld_act<F32>(bb, 4 * j + k));
            } else {
                // four bf16 gains, biases and outputs per 8-byte access (rows of d % 4 == 0)
                const uint2 gw = reinterpret_cast<const uint2*>(g)[j];
                const uint2 bw = reinterpret_cast<const uint2*>(bb)[j];
                const uint32_t gs[2] = {gw.x, gw.y}, bs[2] = {bw.x, bw.y};
                uint32_t o[2];
#pragma unroll
                for (int k = 0; k < 2; ++k) {
                    const float y0 = (xs[2 * k] - mean) * rstd * __uint_as_float(gs[k] << 16) +
                                     __uint_as_float(bs[k] << 16);
                    const float y1 = (xs[2 * k + 1] - mean) * rstd * __uint_as_float(gs[k] & 0xFFFF0000u) +
                                     __uint_as_float(bs[k] & 0xFFFF0000u);
                    o[k] = (uint32_t)f32_to_bf16(y0) | ((uint32_t)f32_to_bf16(y1) << 16);
                }
                reinterpret_cast<uint2*>(out)[((size_t)r * d) / 4 + j] = make_uint2(o[0], o[1]);
            }
        }
    }
}

hipError_t launch_ln_rows(int wdtype, const float* x, const void* g, const void* b, float eps, int M, int d,
                          void* out, hipStream_t st) {
    if (d % 4 == 0 && d <= 2048) {
        const dim3 grid((M + 3) / 4);
        if (wdtype == FTTS_F32) hipLaunchKernelGGL(ln_rows_wave_kernel<true>, grid, dim3(256), 0, st, x, g, b, eps, M, d, out);
        else hipLaunchKernelGGL(ln_rows_wave_kernel<false>, grid, dim3(256), 0, st, x, g, b, eps, M, d, out);
        return hipGetLastError();
    }
    if (wdtype == FTTS_F32) hipLaunchKernelGGL(ln_rows_kernel<true>, dim3(M), dim3(256), 0, st, x, g, b, eps, d, out);
    else hipLaunchKernelGGL(ln_rows_kernel<false>, dim3(M), dim3(256), 0, st, x, g, b, eps, d, out);
    return hipGetLastError();
}

// ---- fill (graph-safe replacement for a memset) -------------------------------------------------
__global__ void fill_u32_kernel(uint32_t* p, size_t n, uint32_t v) {
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) p[i] = v;
}

hipError_t launch_fill_u32(uint32_t* p, size_t n, uint32_t v, hipStream_t st) {
    const int blocks = (int)((n + 255) / 256 < 1024 ? (n + 255) / 256 : 1024);
    hipLaunchKernelGGL(fill_u32_kernel, dim3(blocks > 0 ? blocks : 1), dim3(256), 0, st, p, n, v);
    return hipGetLastError();
}

// ---- row copies ----------------------------------------------------------------------------
__global__ void gather_last_kernel(const float* x, int d, SeqTable seqs, float* out) {
    const int b = blockIdx.x;
    const float* src = x + (size_t)(seqs.cu[b + 1] - 1) * d;
    for (int k = threadIdx.x; k < d; k += blockDim.x) out[(size_t)b * d + k] = src[k];
}

hipError_t launch_gather_rows(const float* x, int d, const SeqTable& seqs, float* out, hipStream_t st) {
    hipLaunchKernelGGL(gather_last_kernel, dim3(seqs.n), dim3(256), 0, st, x, d, seqs, out);
    return hipGetLastError();
}

template <bool F32>
__global__ void act_to_f32_kernel(const void* src, size_t n, float* dst) {
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x)
        dst[i] = ld_act<F32>(src, i);
}

hipError_t launch_act_to_f32(int wdtype, const void* src, int rows, int d, float* dst, hipStream_t st) {
    const size_t n = (size_t)rows * d;
    const int blocks = (int)((n + 255) / 256 < 4096 ? (n + 255) / 256 : 4096);
    if (wdtype == FTTS_F32) hipLaunchKernelGGL(act_to_f32_kernel<true>, dim3(blocks), dim3(256), 0, st, src, n, dst);
    else hipLaunchKernelGGL(act_to_f32_kernel<false>, dim3(blocks), dim3(256), 0, st, src, n, dst);
    return hipGetLastError();
}

// ---- prefill input assembly -----------------------------------------------------------------
// One workgroup per assembled row.  Text ids outside [0, text_vocab) read as a
// zero token row (only the position embedding remains); no access leaves the tables.
template <bool F32>
__global__ __launch_bounds__(256) void assemble_prefix_kernel(const AssembleArgs a) {
    const int r = blockIdx.x;
    int lo = 0, hi = a.seqs.n - 1;  // the sequence holding row r
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (a.seqs.cu[mid] <= r) lo = mid;
        else hi = mid - 1;
    }
    const int j = r - a.seqs.cu[lo], nc = a.cond_cu[lo + 1] - a.cond_cu[lo];
    float* xr = a.x + (size_t)r * a.d;
    if (j < nc) {
        const size_t src = (size_t)(a.cond_cu[lo] + j) * a.d;
        for (int k = threadIdx.x; k < a.d; k += blockDim.x) xr[k] = ld_act<F32>(a.cond, src + k);
        return;
    }
    const int i = j - nc;                                 // text position within the sequence
    const int id = a.text_ids[a.seqs.cu[lo] - a.cond_cu[lo] + i];
    const bool ok = id >= 0 && id < a.text_vocab;
    const size_t tr = (size_t)(a.vocab + (ok ? id : 0)) * a.d, pr = (size_t)(a.text_pos0 + i) * a.d;
    for (int k = threadIdx.x; k < a.d; k += blockDim.x)
        xr[k] = (ok ? ld_act<F32>(a.tok_emb, tr + k) : 0.f) + ld_act<F32>(a.pos_emb, pr + k);
}

hipError_t launch_assemble_prefix(int wdtype, const AssembleArgs& a, int rows, hipStream_t st) {
    if (wdtype == FTTS_F32) hipLaunchKernelGGL(assemble_prefix_kernel<true>, dim3(rows), dim3(256), 0, st, a);
    else hipLaunchKernelGGL(assemble_prefix_kernel<false>, dim3(rows), dim3(256), 0, st, a);
    return hipGetLastError();
}

// ---- sampler ------------------------------------------------------------------------------
// One 256-thread workgroup per sequence; thread t holds the tempered logits of
// indices t, t + 256, ... in registers.  Order is by (value, index): the larger
// value first, the lower index on ties.  NaN logits count as -inf.
//
// Top-k without k sequential block reductions: each wave finds the k-th largest
// of its 64 lane maxima, t_w; at least k entries are >= t_w, so with t = max_w t_w
// every one of the k best entries is >= t.  The entries >= t (typically a few
// times k) are compacted into LDS and each is ranked by counting the candidates
// that beat it; ranks below k fill the ordered top-k list.  Rows with more than
// kSampCand candidates (massive exact ties) take k rounds of block argmax instead.
constexpr int kSampThreads = 256, kSampWaves = kSampThreads / kWave, kSampPer = 64;  // vocab <= 16384
constexpr int kSampCand = 1024;

__device__ __forceinline__ bool beats(float v, int i, float bv, int bi) {
    return v > bv || (v == bv && i < bi);
}

template <int CTRL>
__device__ __forceinline__ int dpp_mov_int(int v) {
    return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xF, 0xF, false);
}
__device__ __forceinline__ int wave_min_int(int v) {
    v = min(v, dpp_mov_int<kDppQuadSwap1>(v));
    v = min(v, dpp_mov_int<kDppQuadSwap2>(v));
    v = min(v, dpp_mov_int<kDppHalfMirror>(v));
    v = min(v, dpp_mov_int<kDppMirror>(v));
    {
        const auto r = __builtin_amdgcn_permlane16_swap((unsigned)v, (unsigned)v, false, false);
        v = min((int)r[0], (int)r[1]);
    }
    {
        const auto r = __builtin_amdgcn_permlane32_swap((unsigned)v, (unsigned)v, false, false);
        v = min((int)r[0], (int)r[1]);
    }
    return v;
}

// Best (value, index) of the wave, in every lane: the largest value, then the
// lowest index holding it.  Lanes with nothing to offer pass (-inf, INT_MAX).
__device__ __forceinline__ void wave_best(float& v, int& i) {
    const float m = wave_max(v);
    i = wave_min_int(v == m ? i : INT_MAX);
    v = m;
}

// Best untaken entry of this lane (indices increase with the slot, so the
// first of equal values wins).
__device__ __forceinline__ void lane_best(const float (&z)[kSampPer], uint64_t taken, float& bv, int& bi) {
    bv = -INFINITY;
    bi = INT_MAX;
#pragma unroll
    for (int j = 0; j < kSampPer; ++j)
        if (!((taken >> j) & 1u) && (z[j] > bv || bi == INT_MAX)) {
            bv = z[j];
            bi = (int)threadIdx.x + kSampThreads * j;
        }
}

// Block-wide best; every thread receives it.
__device__ __forceinline__ void block_best(float& v, int& i, float* rv, int* ri) {
    wave_best(v, i);
    const int w = threadIdx.x / kWave;
    if ((threadIdx.x & (kWave - 1)) == 0) {
        rv[w] = v;
        ri[w] = i;
    }
    __syncthreads();
    v = rv[0];
    i = ri[0];
    for (int j = 1; j < kSampWaves; ++j)
        if (beats(rv[j], ri[j], v, i)) {
            v = rv[j];
            i = ri[j];
        }
    __syncthreads();
}

__global__ __launch_bounds__(kSampThreads) void sample_kernel(const float* logits, int V, float temperature,
                                                              int top_k, float top_p, const float* uniforms,
                                                              const int32_t* active, int32_t* out) {
    __shared__ float cand_v[kSampCand];
    __shared__ int cand_i[kSampCand];
    __shared__ float selv[FTTS_MAX_TOP_K];
    __shared__ int seli[FTTS_MAX_TOP_K];
    __shared__ float rv[kSampWaves];
    __shared__ int ri[kSampWaves];
    __shared__ int s_cnt[kSampWaves];
    const int b = blockIdx.x, tid = threadIdx.x, wave = tid / kWave, lane = tid & (kWave - 1);
    const float* row = logits + (size_t)b * V;
    const bool greedy = top_k == 1;
    // the row, the draw and the activity flag are requested together
    float z[kSampPer];
#pragma unroll
    for (int j = 0; j < kSampPer; ++j) {
        const int i = tid + kSampThreads * j;
        z[j] = i < V ? row[i] : -INFINITY;
    }
    const float u = greedy ? 0.f : uniforms[b];
    if (active && !active[b]) {
        if (tid == 0) out[b] = -1;
        return;
    }
#pragma unroll
    for (int j = 0; j < kSampPer; ++j) {
        const float v = greedy ? z[j] : z[j] / temperature;
        z[j] = v != v ? -INFINITY : v;
    }
    if (greedy) {
        float bv;
        int bi;
        lane_best(z, 0, bv, bi);
        block_best(bv, bi, rv, ri);
        if (tid == 0) out[b] = bi < V ? bi : 0;
        return;
    }
    // wave threshold: the k-th largest lane maximum (ties: lower lane first)
    float lm = -INFINITY;
#pragma unroll
    for (int j = 0; j < kSampPer; ++j) lm = fmaxf(lm, z[j]);
    int rank = 0;
#pragma unroll
    for (int l = 0; l < kWave; ++l) {
        const float o = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(lm), l));
        rank += (o > lm || (o == lm && l < lane)) ? 1 : 0;
    }
    const uint64_t hit = __ballot(rank == top_k - 1);
    const float tw = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(lm), (int)__builtin_ctzll(hit)));
    if (lane == 0) rv[wave] = tw;
    __syncthreads();
    float t = rv[0];
    for (int w = 1; w < kSampWaves; ++w) t = fmaxf(t, rv[w]);
    // candidates: count, exclusive offsets (wave scan, then wave totals), compaction
    int cnt = 0;
#pragma unroll
    for (int j = 0; j < kSampPer; ++j) cnt += z[j] >= t ? 1 : 0;
    int incl = cnt;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        const int u = __shfl_up(incl, o, kWave);
        incl += lane >= o ? u : 0;
    }
    if (lane == kWave - 1) s_cnt[wave] = incl;
    __syncthreads();
    int off = incl - cnt, total = 0;
    for (int w = 0; w < kSampWaves; ++w) {
        off += w < wave ? s_cnt[w] : 0;
        total += s_cnt[w];
    }
    if (total <= kSampCand) {
#pragma unroll
        for (int j = 0; j < kSampPer; ++j)
            if (z[j] >= t) {
                cand_v[off] = z[j];
                cand_i[off] = tid + kSampThreads * j;
                ++off;
            }
        __syncthreads();
        for (int c = tid; c < total; c += kSampThreads) {
            const float cv = cand_v[c];
            const int ci = cand_i[c];
            int r = 0;
            for (int c2 = 0; c2 < total; ++c2) r += beats(cand_v[c2], cand_i[c2], cv, ci) ? 1 : 0;
            if (r < top_k) {
                selv[r] = cv;
                seli[r] = ci;
            }
        }
        __syncthreads();
    } else {
        uint64_t taken = 0;
        float bv;
        int bi;
        lane_best(z, taken, bv, bi);
        for (int r = 0; r < top_k; ++r) {
            float wv = bv;
            int wi = bi;
            block_best(wv, wi, rv, ri);
            if (tid == 0) {
                selv[r] = wv;
                seli[r] = wi;
            }
            if (wi == bi && (wi - tid) % kSampThreads == 0) {  // this thread held the winner
                taken |= 1ull << ((wi - tid) / kSampThreads);
                lane_best(z, taken, bv, bi);
            }
        }
        __syncthreads();
    }
    if (wave != 0) return;
    // fp32 tail in wave 0, lane i holding rank i: the weights exp(z_i - z_1) side
    // by side, then the running sums in rank order (the same additions as a
    // sequential loop), the nucleus cut and the inverse-CDF draw by ballot.
    const bool in = lane < top_k;
    const float e = in ? expf(selv[lane] - selv[0]) : 0.f;
    float acc = 0.f, cum = 0.f;
    for (int i = 0; i < top_k; ++i) {
        acc = acc + __int_as_float(__builtin_amdgcn_readlane(__float_as_int(e), i));
        cum = lane == i ? acc : cum;
    }
    const float thresh = top_p * acc;
    const uint64_t ge = __ballot(in && cum >= thresh);
    const int n = ge ? (int)__builtin_ctzll(ge) + 1 : top_k;
    const float rr = u * __int_as_float(__builtin_amdgcn_readlane(__float_as_int(cum), n - 1));
    const uint64_t gt = __ballot(lane < n && cum > rr);
    const int j = gt ? (int)__builtin_ctzll(gt) : n - 1;
    if (lane == 0) out[b] = seli[j] < V ? seli[j] : 0;
}

hipError_t launch_sample(const float* logits, int B, int V, const ftts_sampling& s, const float* uniforms,
                         const int32_t* active, int32_t* out, hipStream_t st) {
    if (V > kSampThreads * kSampPer || s.top_k < 1 || s.top_k > FTTS_MAX_TOP_K) return hipErrorInvalidValue;
    hipLaunchKernelGGL(sample_kernel, dim3(B), dim3(kSampThreads), 0, st, logits, V, s.temperature, s.top_k,
                       s.top_p, uniforms, active, out);
    return hipGetLastError();
}

// ---- generation-loop bookkeeping -----------------------------------------------------------
__global__ __launch_bounds__(1024) void advance_kernel(int32_t* tokens, int32_t* positions, int32_t* seq_lens,
                                                       int32_t* sampled, int32_t* remaining, int32_t stop_token,
                                                       bool retire_on_stop, int32_t* history, int32_t* step_counter,
                                                       int max_steps, int B) {
    const int step = step_counter ? *step_counter : 0;
    // this thread's first row, requested with the counter (a row is read and
    // written by its own thread only)
    const int b0 = threadIdx.x;
    const int tok0 = b0 < B ? tokens[b0] : -1, smp0 = b0 < B ? sampled[b0] : -1;
    __syncthreads();  // every thread has read the counter before it moves
    for (int b = threadIdx.x; b < B; b += blockDim.x) {
        int h = -1;
        if ((b == b0 ? tok0 : tokens[b]) >= 0) {
            seq_lens[b] += 1;
            positions[b] += 1;
            int next = b == b0 ? smp0 : sampled[b];
            bool retire = retire_on_stop && next == stop_token;  // the model's own stop code
            if (remaining) {
                const int r = remaining[b] - 1;
                remaining[b] = r;
                if (r <= 0) {  // the budget's last step: forced stop code
                    next = stop_token;
                    sampled[b] = stop_token;
                    retire = true;
                }
            }
            tokens[b] = retire ? -1 : next;
            h = next;
        }
        if (history && step < max_steps) history[(size_t)step * B + b] = h;
    }
    if (step_counter && threadIdx.x == 0) *step_counter = step + 1;
}

hipError_t launch_advance(int32_t* tokens, int32_t* positions, int32_t* seq_lens, int32_t* sampled,
                          int32_t* remaining, int32_t stop_token, bool retire_on_stop, int32_t* history,
                          int32_t* step_counter, int max_steps, int B, hipStream_t st) {
    hipLaunchKernelGGL(advance_kernel, dim3(1), dim3(B < 64 ? 64 : (B + 63) / 64 * 64), 0, st, tokens, positions,
                       seq_lens, sampled, remaining, stop_token, retire_on_stop, history, step_counter, max_steps,
                       B);
    return hipGetLastError();
}

// ---- weight quantiser ----------------------------------------------------------------------
// W8A16: one block per row.  s = bf16(amax / 127) (1 if 0); code = clamp(rint(w / s), -127, 127).
__global__ __launch_bounds__(256) void quant_w8_kernel(const float* w, int64_t K, int8_t* codes,
                                                       uint16_t* scales) {
    __shared__ float red[4];
    const int64_t n = blockIdx.x;
    const float* wr = w + n * K;
    float m = 0.f;
    for (int64_t k = threadIdx.x; k < K; k += 256) m = fmaxf(m, fabsf(wr[k]));
    m = wave_max(m);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
    __syncthreads();
    const float amax = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
    uint16_t sb = f32_to_bf16(amax / 127.0f);
    if ((sb & 0x7FFF) == 0) sb = 0x3F80;  // zero scale -> 1
    const float s = bf16_to_f32(sb);
    if (threadIdx.x == 0) scales[n] = sb;
    for (int64_t k = threadIdx.x; k < K; k += 256) {
        const float q = fminf(fmaxf(rintf(wr[k] / s), -127.f), 127.f);
        codes[n * K + k] = (int8_t)q;
    }
}

// W4A16: one block of `group` threads per (row, group).  The range [min(0, mn), max(0, mx)]
// sets s = bf16((mx - mn) / 15) (1 if 0) and z = clamp(rint(-mn / s), 0, 15);
// code = clamp(rint(w / s) + z, 0, 15), packed eight to an int32, low nibble first.
__global__ __launch_bounds__(128) void quant_w4_kernel(const float* w, int64_t K, int group, int32_t* codes,
                                                       uint16_t* scales, uint16_t* zeros) {
    __shared__ float rmin[2], rmax[2];
    __shared__ uint8_t q8[128];
    const int g = blockIdx.x;
    const int64_t n = blockIdx.y;
    const int t = threadIdx.x;
    const float v = w[n * K + (int64_t)g * group + t];
    float mn = v, mx = v;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        mn = fminf(mn, __shfl_xor(mn, o, kWave));
        mx = fmaxf(mx, __shfl_xor(mx, o, kWave));
    }
    if ((t & 63) == 0) {
        rmin[t >> 6] = mn;
        rmax[t >> 6] = mx;
    }
    __syncthreads();
    mn = fminf(fminf(rmin[0], rmin[1]), 0.f);
    mx = fmaxf(fmaxf(rmax[0], rmax[1]), 0.f);
    uint16_t sb = f32_to_bf16((mx - mn) / 15.0f);
    if ((sb & 0x7FFF) == 0) sb = 0x3F80;
    const float s = bf16_to_f32(sb);
    const float z = fminf(fmaxf(rintf(-mn / s), 0.f), 15.f);
    const float q = fminf(fmaxf(rintf(v / s) + z, 0.f), 15.f);
    q8[t] = (uint8_t)q;
    __syncthreads();
    const int n_groups = (int)(K / group);
    if (t == 0) {
        scales[n * n_groups + g] = sb;
        zeros[n * n_groups + g] = f32_to_bf16(z);
    }
    if (t < group / 8) {
        uint32_t word = 0;
#pragma unroll
        for (int j = 0; j < 8; ++j) word |= (uint32_t)q8[t * 8 + j] << (4 * j);
        codes[n * (K / 8) + (int64_t)g * (group / 8) + t] = (int32_t)word;
    }
}

hipError_t launch_quantize(int wdtype, const float* w, int64_t N, int64_t K, int group, void* codes,
                           uint16_t* scales, uint16_t* zeros, hipStream_t st) {
    if (wdtype == FTTS_W8A16) {
        hipLaunchKernelGGL(quant_w8_kernel, dim3((unsigned)N), dim3(256), 0, st, w, K, (int8_t*)codes, scales);
    } else {
        hipLaunchKernelGGL(quant_w4_kernel, dim3((unsigned)(K / group), (unsigned)N), dim3(group), 0, st, w, K,
                           group, (int32_t*)codes, scales, zeros);
    }
    return hipGetLastError();
}

}  // namespace ftts
