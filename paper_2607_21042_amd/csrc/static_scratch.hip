// ftts_decode_step_static: the decode step with its scratch in a static device
// array of this library instead of a caller workspace, for callers that cannot
// allocate device memory.
//
// `scratch` is a file-scope __device__ array: every GPU the library runs on
// holds its own copy, at its own address, until the process ends.  Host code
// never passes the array's name to a kernel (on the host it is only a stand-in
// symbol): the first call on each device looks up that device's address with
// hipGetSymbolAddress, with the device current, and every kernel argument,
// fill and copy uses the address found.
#include <mutex>

#include "decode_entry.hpp"

namespace {

constexpr size_t kScratchBytes = FTTS_STATIC_SCRATCH_BYTES;
__device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
void* g_ptr[kMaxDevices];     // device address of `scratch`, per device
bool g_cleared[kMaxDevices];  // its control words have been cleared once

// Epochs of the persistent step are (step << 8) | event in 32 bits.
constexpr uint32_t kStepWrap = 1u << 24;

// Runs before every step on the scratch: after a step that gave up (abort word
// set), or before the step counter would leave the epoch space, clear the
// control words and exchange buffers, so the next step starts as after a
// prefill.  One workgroup, so that every thread decides on the same words.
__global__ __launch_bounds__(1024) void static_recover_kernel(uint32_t* ctl, size_t words) {
    const bool reset = ctl[1] != 0 || ctl[0] >= kStepWrap - 1;
    __syncthreads();
    if (!reset) return;
    for (size_t i = threadIdx.x; i < words; i += blockDim.x) ctl[i] = 0;
}

int device_scratch(void** out, int* dev_out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return ftts::set_error(FTTS_E_HIP, "hipGetDevice: %s", hipGetErrorString(e));
    if (dev < 0 || dev >= kMaxDevices) return ftts::set_error(FTTS_E_UNSUPPORTED, "device %d out of range", dev);
    std::lock_guard<std::mutex> lock(g_mu);
    if (!g_ptr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return ftts::set_error(FTTS_E_HIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
        g_ptr[dev] = p;
    }
    *out = g_ptr[dev];
    *dev_out = dev;
    return FTTS_OK;
}

// Called by the decode step once every argument has been validated.
int prepare_static(void* ws, hipStream_t st) {
    int dev = -1;
    (void)hipGetDevice(&dev);
    uint32_t* ctl = reinterpret_cast<uint32_t*>(ws);
    const size_t words = ftts::decode_control_bytes() / 4;
    {
        std::lock_guard<std::mutex> lock(g_mu);
        if (dev >= 0 && dev < kMaxDevices && !g_cleared[dev]) {
            const hipError_t e = ftts::launch_fill_u32(ctl, words, 0u, st);
            if (e != hipSuccess) return ftts::set_error(FTTS_E_HIP, "scratch clear: %s", hipGetErrorString(e));
            g_cleared[dev] = true;
        }
    }
    hipLaunchKernelGGL(static_recover_kernel, dim3(1), dim3(1024), 0, st, ctl, words);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return ftts::set_error(FTTS_E_HIP, "scratch recovery: %s", hipGetErrorString(e));
    return FTTS_OK;
}

}  // namespace

extern "C" int ftts_decode_step_static(const ftts_weights* w, const int32_t* tokens, const int32_t* positions,
                                       const ftts_page_table* pt, const ftts_kv_pool* kv, float* logits_out,
                                       int32_t* sampled_out, const float* uniforms, const ftts_sampling* samp,
                                       int32_t B, void* stream) {
    if (w) {
        const size_t need = ftts_workspace_bytes(&w->cfg, B, 0);
        if (need > kScratchBytes)
            return ftts::set_error(FTTS_E_WORKSPACE,
                                   "this model and batch need %zu bytes of scratch, more than the static scratch's "
                                   "%zu (use ftts_decode_step with a workspace)",
                                   need, kScratchBytes);
    }
    void* ptr = nullptr;
    int dev = -1;
    const int rc = device_scratch(&ptr, &dev);
    if (rc != FTTS_OK) return rc;
    return ftts::decode_step(w, tokens, positions, pt, kv, logits_out, nullptr, sampled_out, uniforms, samp, B, ptr,
                             kScratchBytes, stream, prepare_static);
}
