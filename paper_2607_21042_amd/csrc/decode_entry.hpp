// The decode step behind ftts_decode_step, shared with the entry point that
// runs it on a static scratch array instead of a caller workspace.
#pragma once

#include "ftts_internal.hpp"

namespace ftts {

// Sets the calling thread's ftts_last_error message; returns code.
int set_error(int code, const char* fmt, ...);

// Bytes at the start of a decode workspace that hold the persistent step's
// control words (step counter, abort word) and its exchange buffers.
size_t decode_control_bytes();

// One decode step on workspace `ws`; `prepare`, when not null, is called once
// every argument has been validated and before anything is enqueued on `stream`
// (it may enqueue work of its own there); a non-zero return is passed back.
int decode_step(const ftts_weights* w, const int32_t* tokens, const int32_t* positions, const ftts_page_table* pt,
                const ftts_kv_pool* kv, float* logits_out, float* hidden_out, int32_t* sampled_out,
                const float* uniforms, const ftts_sampling* samp, int32_t B, void* ws, size_t ws_bytes, void* stream,
                int (*prepare)(void* ws, hipStream_t st));

}  // namespace ftts
