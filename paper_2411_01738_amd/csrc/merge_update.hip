// HBM-bound kernels of the hot path:
//   * the log-sum-exp merge of chunk partials (Section 4.1.1: SP-Ring's
//     per-chunk partial attentions recombine into the serial result), and
//   * the stand-alone K/V-slice update of the PipeFusion buffer
//     (Section 4.1.2; Section 4.1.4 stores communicated K/V the same way).
// Both move 16 bytes per lane per access, consecutive lanes on consecutive
// addresses.
#include "kernels.h"

#include <math.h>

namespace xdit {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;

struct MergeArgs {
    const void* outs[kMaxPartials];
    const float* lses[kMaxPartials];
    void* out;
    float* lse_out;
    int n, Nq, H, chunks;  // chunks = 16-byte chunks per (b, i, h) row
    int64_t total;         // B * Nq * H * chunks
};

__device__ __forceinline__ float bf16lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }
// Two floats to a packed bf16 pair (round to nearest even): one v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    typedef float f32x2_t __attribute__((ext_vector_type(2)));
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t{lo, hi}), bf16x2_t));
}

// One lane merges one 16-byte chunk of one output row: 8 bf16 or 4 float
// elements.  Weights w_r = exp(lse_r - M) / sum_r' exp(lse_r' - M), which
// equals exp(lse_r - L) with L the merged log-sum-exp.  The partials' loads
// of a lane are issued in groups of kGroup before any is used: with one load
// in flight per lane the merge ran at about half the HBM rate, bound by
// memory latency.
constexpr int kGroup = 8;

// NP > 0: exactly NP partials, known at compile time: every load of a lane
// (its NP LSEs and NP chunks) is issued before any is used, one memory round
// trip per lane.  NP = 0: any n, the partials in groups of kGroup.
template <bool BF16, int NP>
__global__ __launch_bounds__(kThreads) void merge_kernel(MergeArgs a) {
    const int64_t g = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (g >= a.total) return;
    const int cc = (int)(g % a.chunks);
    const int64_t row = g / a.chunks;  // (b * Nq + i) * H + h
    const int h = (int)(row % a.H);
    const int64_t bi = row / a.H;
    const int i = (int)(bi % a.Nq);
    const int64_t b = bi / a.Nq;
    const int64_t lidx = (b * a.H + h) * a.Nq + i;
    constexpr float kLog2e = 1.4426950408889634f;
    const int64_t off = row * a.chunks + cc;  // in 16-byte units
    constexpr int EPC = BF16 ? 8 : 4;
    float acc[EPC];
#pragma unroll
    for (int e = 0; e < EPC; ++e) acc[e] = 0.f;
    float L = -INFINITY;

    if constexpr (NP > 0) {
        u32x4 x[NP];
        float l[NP];
#pragma unroll
        for (int r = 0; r < NP; ++r) {
            l[r] = a.lses[r][lidx];
            x[r] = ((const u32x4*)a.outs[r])[off];
        }
        float M = l[0];
#pragma unroll
        for (int r = 1; r < NP; ++r) M = fmaxf(M, l[r]);
        if (M != -INFINITY) {
            // (lse_r - M) is exactly 0 for the largest partial, so its weight
            // is exactly 1 before normalisation and n = 1 reproduces the partial
            float w[NP], sum = 0.f;
#pragma unroll
            for (int r = 0; r < NP; ++r) {
                w[r] = exp2f((l[r] - M) * kLog2e);
                sum += w[r];
            }
            const float inv = 1.f / sum;
            L = M + logf(sum);
#pragma unroll
            for (int r = 0; r < NP; ++r) {
                const float wr = w[r] * inv;
                if constexpr (BF16) {
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        acc[2 * e] = __builtin_fmaf(wr, bf16lo(x[r][e]), acc[2 * e]);
                        acc[2 * e + 1] = __builtin_fmaf(wr, bf16hi(x[r][e]), acc[2 * e + 1]);
                    }
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e) acc[e] = __builtin_fmaf(wr, __uint_as_float(x[r][e]), acc[e]);
                }
            }
        }
    } else {
        float M = -INFINITY;
        for (int r = 0; r < a.n; ++r) M = fmaxf(M, a.lses[r][lidx]);
        if (M != -INFINITY) {
            // (lse_r - M) is exactly 0 for the largest partial, so its weight is
            // exactly 1 before normalisation and n = 1 reproduces the partial.
            float sum = 0.f;
            for (int r = 0; r < a.n; ++r) sum += exp2f((a.lses[r][lidx] - M) * kLog2e);
            const float inv = 1.f / sum;
            L = M + logf(sum);
            for (int r0 = 0; r0 < a.n; r0 += kGroup) {
                u32x4 x[kGroup];
                float w[kGroup];
#pragma unroll
                for (int j = 0; j < kGroup; ++j)
                    if (r0 + j < a.n) {
                        x[j] = ((const u32x4*)a.outs[r0 + j])[off];
                        w[j] = a.lses[r0 + j][lidx];
                    }
#pragma unroll
                for (int j = 0; j < kGroup; ++j)
                    if (r0 + j < a.n) {
                        const float wj = exp2f((w[j] - M) * kLog2e) * inv;
                        if constexpr (BF16) {
#pragma unroll
                            for (int e = 0; e < 4; ++e) {
                                acc[2 * e] = __builtin_fmaf(wj, bf16lo(x[j][e]), acc[2 * e]);
                                acc[2 * e + 1] = __builtin_fmaf(wj, bf16hi(x[j][e]), acc[2 * e + 1]);
                            }
                        } else {
#pragma unroll
                            for (int e = 0; e < 4; ++e) acc[e] = __builtin_fmaf(wj, __uint_as_float(x[j][e]), acc[e]);
                        }
                    }
            }
        }
    }
    u32x4 y;
    if constexpr (BF16) {
#pragma unroll
        for (int e = 0; e < 4; ++e) y[e] = pack_bf16x2(acc[2 * e], acc[2 * e + 1]);
    } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) y[e] = __float_as_uint(acc[e]);
    }
    ((u32x4*)a.out)[off] = y;
    if (a.lse_out && cc == 0) a.lse_out[lidx] = L;
}

template <bool BF16>
hipError_t launch_merge(const MergeParams& p, hipStream_t s) {
    MergeArgs a;
    for (int r = 0; r < kMaxPartials; ++r) {
        a.outs[r] = r < p.n ? p.outs[r] : nullptr;
        a.lses[r] = r < p.n ? p.lses[r] : nullptr;
    }
    a.out = p.out;
    a.lse_out = p.lse_out;
    a.n = p.n;
    a.Nq = p.Nq;
    a.H = p.H;
    a.chunks = p.D * (BF16 ? 2 : 4) / 16;
    a.total = (int64_t)p.B * p.Nq * p.H * a.chunks;
    if (a.total == 0) return hipSuccess;
    const int64_t blocks = (a.total + kThreads - 1) / kThreads;
    const dim3 grid((unsigned)blocks), block(kThreads);
    switch (p.n) {
        case 1: hipLaunchKernelGGL((merge_kernel<BF16, 1>), grid, block, 0, s, a); break;
        case 2: hipLaunchKernelGGL((merge_kernel<BF16, 2>), grid, block, 0, s, a); break;
        case 3: hipLaunchKernelGGL((merge_kernel<BF16, 3>), grid, block, 0, s, a); break;
        case 4: hipLaunchKernelGGL((merge_kernel<BF16, 4>), grid, block, 0, s, a); break;
        case 6: hipLaunchKernelGGL((merge_kernel<BF16, 6>), grid, block, 0, s, a); break;
        case 8: hipLaunchKernelGGL((merge_kernel<BF16, 8>), grid, block, 0, s, a); break;
        default: hipLaunchKernelGGL((merge_kernel<BF16, 0>), grid, block, 0, s, a); break;
    }
    return hipGetLastError();
}

struct UpdateArgs {
    u32x4* kv;            // buffer base
    const u32x4* fk;      // fresh rows, already offset to row fbase of batch 0
    const u32x4* fv;
    int64_t plane_vecs;   // B * N * H * D * esize / 16
    int64_t batch_vecs;   // N * H * D * esize / 16
    int64_t off_vecs;     // off * H * D * esize / 16
    int64_t slice_vecs;   // len * H * D * esize / 16 (per batch)
    int64_t fbatch_vecs;  // frows * H * D * esize / 16
    int B;
};

// blockIdx.y = plane * B + b; the slice of one (plane, batch) is contiguous.
// A lane copies kUpd vectors per pass, all loads issued before the stores.
constexpr int kUpd = 4;

__global__ __launch_bounds__(kThreads) void kv_update_kernel(UpdateArgs a) {
    const int plane = blockIdx.y / a.B, b = blockIdx.y % a.B;
    const u32x4* src = (plane ? a.fv : a.fk) + (int64_t)b * a.fbatch_vecs;
    u32x4* dst = a.kv + plane * a.plane_vecs + (int64_t)b * a.batch_vecs + a.off_vecs;
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    for (int64_t v0 = (int64_t)blockIdx.x * kThreads + threadIdx.x; v0 < a.slice_vecs; v0 += kUpd * stride) {
        u32x4 x[kUpd];
#pragma unroll
        for (int u = 0; u < kUpd; ++u)
            if (v0 + u * stride < a.slice_vecs) x[u] = src[v0 + u * stride];
#pragma unroll
        for (int u = 0; u < kUpd; ++u)
            if (v0 + u * stride < a.slice_vecs) dst[v0 + u * stride] = x[u];
    }
}

}  // namespace

hipError_t launch_merge_bf16(const MergeParams& p, hipStream_t s) { return launch_merge<true>(p, s); }
hipError_t launch_merge_f32(const MergeParams& p, hipStream_t s) { return launch_merge<false>(p, s); }

hipError_t launch_kv_update(const UpdateParams& p, hipStream_t s) {
    const int64_t row_vecs = (int64_t)p.H * p.D * p.esize / 16;
    UpdateArgs a;
    a.kv = (u32x4*)p.kv_buf;
    a.fk = (const u32x4*)p.fresh_k + (int64_t)p.fbase * row_vecs;
    a.fv = (const u32x4*)p.fresh_v + (int64_t)p.fbase * row_vecs;
    a.fbatch_vecs = (int64_t)p.frows * row_vecs;
    a.batch_vecs = (int64_t)p.N * row_vecs;
    a.plane_vecs = (int64_t)p.B * a.batch_vecs;
    a.off_vecs = (int64_t)p.off * row_vecs;
    a.slice_vecs = (int64_t)p.len * row_vecs;
    a.B = p.B;
    if (a.slice_vecs == 0 || p.B == 0) return hipSuccess;
    int64_t bx = (a.slice_vecs + kThreads * kUpd - 1) / (kThreads * kUpd);  // one pass of kUpd vectors per lane
    if (bx < 1) bx = 1;
    if (bx > 65535) bx = 65535;
    hipLaunchKernelGGL(kv_update_kernel, dim3((unsigned)bx, (unsigned)(2 * p.B)), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

}  // namespace xdit
