// Internal interface between the C-ABI layer (xdit_api.cpp) and the HIP
// kernels.  Shapes have been validated before any of these is called.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace xdit {

// One attention launch: chunk attention (fresh_k == nullptr) or a fused
// PipeFusion patch step (K/V rows [off, off+len) come from fresh_k/fresh_v and
// are written back into the buffer planes wk/wv).
struct AttnParams {
    const void* q;        // [B, Nq, H, D]
    const void* k;        // [B, Nk, H, D]  (patch: K plane of the buffer)
    const void* v;        // [B, Nk, H, D]  (patch: V plane of the buffer)
    const void* fresh_k;  // [B, len, H, D] or nullptr
    const void* fresh_v;
    void* wk;             // patch write-back target planes (== k / v) or nullptr
    void* wv;
    void* out;            // [B, Nq, H, D]
    float* lse;           // [B, H, Nq] or nullptr
    int B, H, Nq, Nk, D;
    int off, len;         // patch slice; len == 0 for chunk attention
};

struct MergeParams {
    const void* const* outs;  // host array of n device pointers
    const float* const* lses; // host array of n device pointers
    int n;
    void* out;
    float* lse_out;           // or nullptr
    int B, Nq, H, D;
};

struct UpdateParams {
    void* kv_buf;             // [2, B, N, H, D]
    const void* fresh_k;      // [B, len, H, D]
    const void* fresh_v;
    int B, N, H, D, off, len;
    int esize;                // bytes per element
};

constexpr int kMaxPartials = 64;

hipError_t launch_attn_bf16(const AttnParams& p, hipStream_t s);
hipError_t launch_attn_f32(const AttnParams& p, hipStream_t s);
hipError_t launch_merge_bf16(const MergeParams& p, hipStream_t s);
hipError_t launch_merge_f32(const MergeParams& p, hipStream_t s);
hipError_t launch_kv_update(const UpdateParams& p, hipStream_t s);

}  // namespace xdit
