// float32 attention (chunk attention with O and LSE, and the fused PipeFusion
// patch step) with float32 products throughout.  This path exists for the
// exactness check at float32 I/O; it is not a throughput path.
//
// One workgroup = one wave = 64 query rows of one (batch, head), one query per
// lane.  K/V are swept in tiles of 32 rows staged through LDS (every lane
// reads the same row: an LDS broadcast).  Per tile: 32 scores per lane, one
// rescale of the running output by exp(m_old - m_new), then the weighted sum.
#include "kernels.h"

#include <math.h>

namespace xdit {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kFBM = 64;  // queries per workgroup
constexpr int kFBN = 32;  // keys per tile

struct Args {
    const float* q;
    const float* k;
    const float* v;
    const float* fk;
    const float* fv;
    float* wk;
    float* wv;
    float* out;
    float* lse;
    int B, H, Nq, Nk, q_tiles;
    int off0, len0, off1, len1;  // fresh ranges (fresh rows: range 0's, then range 1's)
    float scale;
    int accum;  // merge into the running (out, lse) instead of overwriting them
};

__device__ __forceinline__ int xcd_remap(int pid, int total) {
    const int per = total >> 3, rem = total & 7;
    const int xcd = pid & 7, loc = pid >> 3;
    return xcd * per + (xcd < rem ? xcd : rem) + loc;
}

template <int D, bool PATCH>
__global__ __launch_bounds__(kFBM) void attn_f32_kernel(Args a) {
    __shared__ __attribute__((aligned(16))) float Ks[kFBN * D];
    __shared__ __attribute__((aligned(16))) float Vs[kFBN * D];
    constexpr int C4 = D / 4;  // 16-byte chunks per row

    const int tid = threadIdx.x;
    const int logical = xcd_remap(blockIdx.x, gridDim.x);
    const int qt = logical % a.q_tiles;
    const int bh = logical / a.q_tiles;
    const int hh = bh % a.H, b = bh / a.H;
    const int64_t rs = (int64_t)a.H * D;
    const bool writeback = PATCH && qt == 0;

    const int qrow = qt * kFBM + tid;
    const bool qvalid = qrow < a.Nq;
    float qv[D], o[D];
    {
        const float* qp = a.q + ((int64_t)b * a.Nq + qrow) * rs + (int64_t)hh * D;
#pragma unroll
        for (int c = 0; c < D; ++c) {
            qv[c] = qvalid ? qp[c] : 0.f;
            o[c] = 0.f;
        }
    }
    float m = -INFINITY, l = 0.f;

    // row of the fresh tensors that holds buffer row j, or -1
    const int F = a.len0 + a.len1;
    auto fresh_row = [&](int j) -> int {
        if (!PATCH) return -1;
        if ((unsigned)(j - a.off0) < (unsigned)a.len0) return j - a.off0;
        if ((unsigned)(j - a.off1) < (unsigned)a.len1) return a.len0 + j - a.off1;
        return -1;
    };

    const int ntiles = (a.Nk + kFBN - 1) / kFBN;
    for (int t = 0; t < ntiles; ++t) {
        __syncthreads();  // the previous tile has been consumed
        for (int e = tid; e < kFBN * C4; e += kFBM) {
            const int r = e / C4, cc = e % C4, j = t * kFBN + r;
            f32x4 kx = {0.f, 0.f, 0.f, 0.f}, vx = {0.f, 0.f, 0.f, 0.f};
            if (j < a.Nk) {
                const float *kp, *vp;
                const int fr = fresh_row(j);
                if (fr >= 0) {
                    const int64_t o2 = ((int64_t)b * F + fr) * rs + (int64_t)hh * D + 4 * cc;
                    kp = a.fk + o2;
                    vp = a.fv + o2;
                } else {
                    const int64_t o2 = ((int64_t)b * a.Nk + j) * rs + (int64_t)hh * D + 4 * cc;
                    kp = a.k + o2;
                    vp = a.v + o2;
                }
                kx = *(const f32x4*)kp;
                vx = *(const f32x4*)vp;
                if (writeback && fr >= 0) {
                    const int64_t o3 = ((int64_t)b * a.Nk + j) * rs + (int64_t)hh * D + 4 * cc;
                    *(f32x4*)(a.wk + o3) = kx;
                    *(f32x4*)(a.wv + o3) = vx;
                }
            }
            *(f32x4*)(Ks + r * D + 4 * cc) = kx;
            *(f32x4*)(Vs + r * D + 4 * cc) = vx;
        }
        __syncthreads();

        float s[kFBN];
        float mt = -INFINITY;
#pragma unroll
        for (int r = 0; r < kFBN; ++r) {
            float dot = 0.f;
#pragma unroll
            for (int c = 0; c < D; ++c) dot = __builtin_fmaf(qv[c], Ks[r * D + c], dot);
            s[r] = (t * kFBN + r < a.Nk) ? dot * a.scale : -INFINITY;
            mt = fmaxf(mt, s[r]);
        }
        const float m_new = fmaxf(m, mt);
        const float alpha = expf(m - m_new);
        m = m_new;
        l *= alpha;
#pragma unroll
        for (int c = 0; c < D; ++c) o[c] *= alpha;
#pragma unroll
        for (int r = 0; r < kFBN; ++r) {
            const float p = expf(s[r] - m_new);
            l += p;
#pragma unroll
            for (int c = 0; c < D; ++c) o[c] = __builtin_fmaf(p, Vs[r * D + c], o[c]);
        }
    }

    if (qvalid) {
        const float inv = l > 0.f ? 1.f / l : 0.f;
        const float lse_new = l > 0.f ? m + logf(l) : -INFINITY;
        const int64_t lidx = ((int64_t)b * a.H + hh) * a.Nq + qrow;
        // merge into a running (out, lse): see the bf16 kernel
        float w_prev = 0.f, w_new = inv, lse_out = lse_new;
        if (a.accum) {
            const float lse_prev = a.lse[lidx];
            if (lse_prev != -INFINITY) {
                if (lse_new == -INFINITY) {
                    w_prev = 1.f;
                    w_new = 0.f;
                    lse_out = lse_prev;
                } else {
                    const float M = fmaxf(lse_prev, lse_new);
                    const float e1 = expf(lse_prev - M), e2 = expf(lse_new - M);
                    w_prev = e1 / (e1 + e2);
                    w_new = e2 / (e1 + e2) * inv;
                    lse_out = M + logf(e1 + e2);
                }
            }
        }
        float* op = a.out + ((int64_t)b * a.Nq + qrow) * rs + (int64_t)hh * D;
#pragma unroll
        for (int c = 0; c < D; c += 4) {
            f32x4 y = {o[c] * w_new, o[c + 1] * w_new, o[c + 2] * w_new, o[c + 3] * w_new};
            if (w_prev != 0.f) {
                const f32x4 x = *(const f32x4*)(op + c);
                y = f32x4{__builtin_fmaf(w_prev, x[0], y[0]), __builtin_fmaf(w_prev, x[1], y[1]),
                          __builtin_fmaf(w_prev, x[2], y[2]), __builtin_fmaf(w_prev, x[3], y[3])};
            }
            *(f32x4*)(op + c) = y;
        }
        if (a.lse) a.lse[lidx] = lse_out;
    }
}

template <int D, bool PATCH>
hipError_t launch(const AttnParams& p, hipStream_t s) {
    Args a;
    a.q = (const float*)p.q;
    a.k = (const float*)p.k;
    a.v = (const float*)p.v;
    a.fk = (const float*)p.fresh_k;
    a.fv = (const float*)p.fresh_v;
    a.wk = (float*)p.wk;
    a.wv = (float*)p.wv;
    a.out = (float*)p.out;
    a.lse = p.lse;
    a.B = p.B;
    a.H = p.H;
    a.Nq = p.Nq;
    a.Nk = p.Nk;
    a.off0 = p.off0;
    a.len0 = p.len0;
    a.off1 = p.off1;
    a.len1 = p.len1;
    a.q_tiles = (p.Nq + kFBM - 1) / kFBM;
    a.scale = (float)(1.0 / sqrt((double)D));
    a.accum = p.accum;
    const int64_t blocks = (int64_t)a.q_tiles * p.H * p.B;
    if (blocks == 0) return hipSuccess;
    hipLaunchKernelGGL((attn_f32_kernel<D, PATCH>), dim3((unsigned)blocks), dim3(kFBM), 0, s, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_attn_f32(const AttnParams& p, hipStream_t s) {
    const bool patch = p.fresh_k != nullptr;
    switch (p.D) {
        case 64: return patch ? launch<64, true>(p, s) : launch<64, false>(p, s);
        case 72: return patch ? launch<72, true>(p, s) : launch<72, false>(p, s);
        case 128: return patch ? launch<128, true>(p, s) : launch<128, false>(p, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace xdit
