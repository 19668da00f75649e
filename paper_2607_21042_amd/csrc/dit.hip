// Small kernels around one guided Euler step of the flow-matching DiT (Sec. II-A:
// the Semantic-to-Mel module integrates a learned velocity field with an Euler
// solver under classifier-free guidance).  The dense work of the step -- every
// linear and the attention -- runs on the prefill GEMM and the matrix-core
// attention; these kernels only build the step's inputs and combine its outputs:
//
//   dit_time_hidden / dit_time_out   e(t) = W_t2 silu(W_t1 s(t) + b_t1) + b_t2
//   dit_prepare                      h rows <- e(t); bf16 input rows [x | c] and
//                                    [x | 0]; zero the velocity accumulator and the
//                                    split-K counters
//   dit_guide                        v = v_u + w (v_c - v_u); x' = x + dt v
//
// Both guidance branches run as one batch of 2T rows: rows 0 .. T-1 carry the
// conditioning, rows T .. 2T-1 a zero conditioning.
#include <algorithm>

#include "ftts_internal.hpp"

namespace ftts {

namespace {

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

// One wave per output row r of W [N][K] bf16 (row-major) times the fp32 vector u [K].
__device__ __forceinline__ float row_dot(const uint16_t* W, int K, int r, const float* u, int lane) {
    const uint16_t* wr = W + (size_t)r * K;
    float acc = 0.f;
    for (int k = lane; k < K; k += 64) acc += bf16_to_f32(wr[k]) * u[k];
    return wave_sum(acc);
}

// Sinusoidal time features in LDS (in double, then rounded once), then
// u = silu(W_t1 s + b_t1), one wave per row of W_t1.
__global__ __launch_bounds__(256) void dit_time_hidden_kernel(float t, const void* w1, const void* b1, int D,
                                                              int t_dim, float* u) {
    __shared__ float s[1024];
    const int half = t_dim / 2;
    for (int i = threadIdx.x; i < t_dim; i += blockDim.x) {
        const int j = i < half ? i : i - half;
        const double ph = 1000.0 * (double)t * exp(-log(10000.0) * (double)j / (double)half);
        s[i] = (float)(i < half ? cos(ph) : sin(ph));
    }
    __syncthreads();
    const int lane = threadIdx.x & 63, r = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (r >= D) return;
    const float y = row_dot(reinterpret_cast<const uint16_t*>(w1), t_dim, r, s, lane) +
                    bf16_to_f32(reinterpret_cast<const uint16_t*>(b1)[r]);
    if (lane == 0) u[r] = y / (1.f + expf(-y));
}

// e = W_t2 u + b_t2, one wave per row.
__global__ __launch_bounds__(256) void dit_time_out_kernel(const void* w2, const void* b2, int D, const float* u,
                                                           float* e) {
    const int lane = threadIdx.x & 63, r = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (r >= D) return;
    const float y = row_dot(reinterpret_cast<const uint16_t*>(w2), D, r, u, lane) +
                    bf16_to_f32(reinterpret_cast<const uint16_t*>(b2)[r]);
    if (lane == 0) e[r] = y;
}

// The four things the step starts from, one row of each per loop iteration
// (rows m of the 2T-row batch; columns strided over the workgroup):
//   input row m: x[m mod T] (bf16), then cond[m] or zeros
//   h[m][j] = e[j]
//   velocity accumulator row m <- 0
// and the split-K arrival counters <- 0 (first workgroup).
__global__ __launch_bounds__(256) void dit_prepare_kernel(const DitPrepareArgs a) {
    const int M = 2 * a.T, Kin = a.n_mel + a.d_cond;
    uint16_t* inp = reinterpret_cast<uint16_t*>(a.inp);
    const uint16_t* cond = reinterpret_cast<const uint16_t*>(a.cond);
    if (blockIdx.x == 0)
        for (size_t i = threadIdx.x; i < a.n_count; i += blockDim.x) a.count[i] = 0u;
    for (int m = blockIdx.x; m < M; m += gridDim.x) {
        const bool guided = m < a.T;
        const int f = guided ? m : m - a.T;  // frame of this row
        const float* xr = a.x + (size_t)f * a.n_mel;
        const uint16_t* cr = cond + (size_t)f * a.d_cond;
        uint16_t* ir = inp + (size_t)m * Kin;
        for (int c = threadIdx.x; c < a.n_mel; c += blockDim.x) ir[c] = f32_to_bf16(xr[c]);
        for (int c = threadIdx.x; c < a.d_cond; c += blockDim.x) ir[a.n_mel + c] = guided ? cr[c] : (uint16_t)0;
        float* hr = a.h + (size_t)m * a.d_model;
        for (int c = threadIdx.x; c < a.d_model; c += blockDim.x) hr[c] = a.e[c];
        float* vr = a.vel + (size_t)m * a.n_mel;
        for (int c = threadIdx.x; c < a.n_mel; c += blockDim.x) vr[c] = 0.f;
    }
}

__global__ __launch_bounds__(256) void dit_guide_kernel(const float* vel, int T, int n_mel, float w, float dt,
                                                        const float* x, float* x_out, float* v_out) {
    const size_t n = (size_t)T * n_mel;
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
        const float vc = vel[i], vu = vel[n + i];
        const float v = vu + w * (vc - vu);
        const float xi = x[i];
        if (v_out) v_out[i] = v;
        x_out[i] = xi + dt * v;
    }
}

unsigned flat_grid(size_t n) {
    const size_t g = (n + 255) / 256;
    return (unsigned)std::min<size_t>(std::max<size_t>(g, 1), 4096);
}

}  // namespace

hipError_t launch_dit_time(float t, const void* w1, const void* b1, const void* w2, const void* b2, int D, int t_dim,
                           float* u, float* e, hipStream_t st) {
    if (t_dim < 2 || t_dim > 1024 || t_dim % 2) return hipErrorInvalidValue;
    const dim3 g((D + 3) / 4);
    hipLaunchKernelGGL(dit_time_hidden_kernel, g, dim3(256), 0, st, t, w1, b1, D, t_dim, u);
    hipLaunchKernelGGL(dit_time_out_kernel, g, dim3(256), 0, st, w2, b2, D, u, e);
    return hipGetLastError();
}

hipError_t launch_dit_prepare(const DitPrepareArgs& a, hipStream_t st) {
    const unsigned rows = 2u * (unsigned)a.T;
    hipLaunchKernelGGL(dit_prepare_kernel, dim3(std::min(rows, 8192u)), dim3(256), 0, st, a);
    return hipGetLastError();
}

hipError_t launch_dit_guide(const float* vel, int T, int n_mel, float w, float dt, const float* x, float* x_out,
                            float* v_out, hipStream_t st) {
    hipLaunchKernelGGL(dit_guide_kernel, dim3(flat_grid((size_t)T * n_mel)), dim3(256), 0, st, vel, T, n_mel, w, dt,
                       x, x_out, v_out);
    return hipGetLastError();
}

}  // namespace ftts
