// Internal interface between the C-ABI layer (xdit_api.cpp) and the HIP
// kernels.  Shapes have been validated before any of these is called.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace xdit {

// One attention launch: chunk attention (fresh_k == nullptr) or a fused
// PipeFusion patch step: K/V rows in the fresh ranges [off0, off0+len0) and
// [off1, off1+len1) come from fresh_k/fresh_v (rows 0..len0-1, then
// len0..len0+len1-1) and are written back into the buffer planes wk/wv.
struct AttnParams {
    const void* q;        // [B, Nq, H, D]
    const void* k;        // [B, Nk, H, D]  (patch: K plane of the buffer)
    const void* v;        // [B, Nk, H, D]  (patch: V plane of the buffer)
    const void* fresh_k;  // [B, len0 + len1, H, D] or nullptr
    const void* fresh_v;
    void* wk;             // patch write-back target planes (== k / v) or nullptr
    void* wv;
    void* out;            // [B, Nq, H, D]
    float* lse;           // [B, H, Nq] or nullptr
    int B, H, Nq, Nk, D;
    int off0, len0;       // first fresh range
    int off1, len1;       // second fresh range (len1 == 0: none); disjoint from the first
    int accum;            // merge into the running (out, lse) instead of overwriting them
    // Work partition (bf16 only; 128-row query tiles).  parts = 0: one
    // workgroup per query tile.  parts > 0: `whole` workgroups (a multiple
    // of 8) sweep the first `whole` query tiles whole, and the (query tile,
    // K/V tile) units of the others are cut into `parts` contiguous ranges,
    // one workgroup each; partials of cut sweeps go to `part`
    // (kPartSlotRows * (D + 1) floats per slot; slots 0..parts-1, and
    // parts..2*parts-1 when ranges may cross query tiles) and a fix-up
    // launch merges them.
    int64_t whole, parts;
    float* part;
};

struct MergeParams {
    const void* const* outs;  // host array of n device pointers
    const float* const* lses; // host array of n device pointers
    int n;
    void* out;
    float* lse_out;           // or nullptr
    int B, Nq, H, D;
};

// Copy fresh rows [fbase, fbase+len) of fresh_k/fresh_v [B, frows, H, D]
// into rows [off, off+len) of both buffer planes.
struct UpdateParams {
    void* kv_buf;             // [2, B, N, H, D]
    const void* fresh_k;      // [B, frows, H, D]
    const void* fresh_v;
    int B, N, H, D, off, len;
    int frows, fbase;
    int esize;                // bytes per element
};

constexpr int kMaxPartials = 64;
constexpr int kPartSlotRows = 128;  // query rows of a partitioned launch's tile
constexpr int kMaxSweepParts = 17;  // most partition ranges one sweep may meet

hipError_t launch_attn_bf16(const AttnParams& p, hipStream_t s);
// The second launch of a partitioned bf16 attention (128-row query tiles,
// sweeps of T K/V tiles): merges the partials of the cut sweeps into out
// and lse.
hipError_t launch_attn_fixup(const AttnParams& p, int q_tiles, int T, hipStream_t s);
// bf16 attention with 64 query rows per wave and one wave per SIMD (head
// dim 128); hipErrorNotSupported for shapes it does not take.
hipError_t launch_attn_w64(const AttnParams& p, hipStream_t s);
hipError_t launch_attn_f32(const AttnParams& p, hipStream_t s);
hipError_t launch_merge_bf16(const MergeParams& p, hipStream_t s);
hipError_t launch_merge_f32(const MergeParams& p, hipStream_t s);
hipError_t launch_kv_update(const UpdateParams& p, hipStream_t s);

}  // namespace xdit
