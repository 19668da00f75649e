// One 64-token page of a head's keys or values as held by one lane of a wave:
// 8 chunks, chunk i holding dims (lane%8)*8 .. +7 of token i*8 + lane/8, so a
// page is 8 fully coalesced 1 KB wave loads.
#pragma once
#include "ftts_internal.hpp"

namespace ftts {

// One page of K or V as seen by one lane: 8 chunks, each 8 consecutive dims of one token.
template <bool F32> struct PageRegs;
template <> struct PageRegs<false> { uint4 k[8], v[8]; };
template <> struct PageRegs<true> { float4 k[16], v[16]; };

template <bool F32>
__device__ __forceinline__ void load_page(const void* base, size_t kbase, size_t vbase, int lane, PageRegs<F32>& r) {
    if constexpr (F32) {
        const float4* K = reinterpret_cast<const float4*>(reinterpret_cast<const float*>(base) + kbase);
        const float4* V = reinterpret_cast<const float4*>(reinterpret_cast<const float*>(base) + vbase);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            r.k[2 * i] = K[(i * 64 + lane) * 2];
            r.k[2 * i + 1] = K[(i * 64 + lane) * 2 + 1];
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            r.v[2 * i] = V[(i * 64 + lane) * 2];
            r.v[2 * i + 1] = V[(i * 64 + lane) * 2 + 1];
        }
    } else {
        const uint4* K = reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(base) + kbase);
        const uint4* V = reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(base) + vbase);
#pragma unroll
        for (int i = 0; i < 8; ++i) r.k[i] = K[i * 64 + lane];
#pragma unroll
        for (int i = 0; i < 8; ++i) r.v[i] = V[i * 64 + lane];
    }
}

template <bool F32>
__device__ __forceinline__ void unpack8(const PageRegs<F32>& r, bool is_v, int i, float (&x)[8]) {
    if constexpr (F32) {
        const float4 a = is_v ? r.v[2 * i] : r.k[2 * i];
        const float4 b = is_v ? r.v[2 * i + 1] : r.k[2 * i + 1];
        x[0] = a.x; x[1] = a.y; x[2] = a.z; x[3] = a.w; x[4] = b.x; x[5] = b.y; x[6] = b.z; x[7] = b.w;
    } else {
        const uint4 w = is_v ? r.v[i] : r.k[i];
        x[0] = bf16lo(w.x); x[1] = bf16hi(w.x); x[2] = bf16lo(w.y); x[3] = bf16hi(w.y);
        x[4] = bf16lo(w.z); x[5] = bf16hi(w.z); x[6] = bf16lo(w.w); x[7] = bf16hi(w.w);
    }
}

}  // namespace ftts
