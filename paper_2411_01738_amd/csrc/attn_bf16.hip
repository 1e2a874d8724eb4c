// bf16 attention on the gfx950 matrix cores: chunk attention with O and LSE,
// and the fused PipeFusion patch step (K/V-slice update + attention over the
// fresh/stale buffer).
//
// What is computed (Section 2 and Sections 4.1.1/4.1.2 of arXiv 2411.01738):
//   out_i = sum_j softmax_j(s_ij) v_j,  s_ij = (q_i . k_j) / sqrt(d),
//   lse_i = ln sum_j exp(s_ij),
// full (non-causal) attention per (batch, head).  In patch mode K/V row j is
// taken from the fresh rows when off <= j < off+len and from the buffer
// otherwise, and the fresh rows are written into the buffer.
//
// Work decomposition
//   * one workgroup = 4 waves = 128 query rows of one (batch, head); each
//     wave owns 32 query rows for the whole K/V sweep;
//   * K/V are swept in tiles of BN rows staged through LDS (double buffered,
//     one barrier per tile); the global loads of tile t+1 are in flight while
//     tile t is computed.  Loads go through buffer resources: a row past the
//     end, or a row served by the other source in patch mode, gets an
//     out-of-range offset and reads as zero, so no lane branches;
//   * scores are computed transposed, S^T = K Q^T, with
//     v_mfma_f32_32x32x16_bf16: A = K rows from LDS, B = the wave's Q rows
//     held in registers for the whole sweep.  In the 32x32 accumulator layout
//     each lane then holds 16 keys of ONE query, so the row max is in-lane
//     except for one exchange between the two 32-lane halves;
//   * online softmax in the log2 domain (scale*log2(e) folded into one FMA
//     before v_exp_f32).  The reference max is only raised when a row's tile
//     max exceeds it by more than 2^8 in weight, so the running output is
//     rescaled rarely; weights up to 2^8 are exact enough in bf16/float32 and
//     the final normalisation uses the same reference, so the result does not
//     depend on when rescales happen;
//   * O^T = V^T P^T on the same instruction: P^T comes straight from the
//     score accumulators (no data movement) because the K index order of an
//     MFMA contraction is free as long as A and B agree; V is transposed into
//     LDS while staging, with the key order permuted to match P's register
//     order, so each A operand is one 16-byte LDS read;
//   * where the output rows are padded (d = 72 -> 96), one padding row of V^T
//     holds ones, so the same MFMA also produces the row sums of the bf16
//     weights (the exact normaliser of the bf16 numerator);
//   * LDS pitches are padded so the 16-byte operand reads of 16 lanes hit
//     distinct bank groups.
// Workgroups are renumbered so that all query tiles of one (batch, head) run
// on the same XCD and share its L2 for K/V (the hardware deals workgroup ids
// round-robin over the 8 XCDs).
#include "kernels.h"

#include <math.h>

namespace xdit {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kThreads = 256;  // 4 waves
constexpr int kBM = 128;       // query rows per workgroup
constexpr uint32_t kOOB = 0x80000000u;       // offset past any buffer's range: reads 0, writes dropped
constexpr int kRsrcFlags = 0x00020000;       // raw buffer, 32-bit data format
constexpr float kRescaleLog2 = 8.0f;         // raise the reference max only beyond 2^8 growth

template <int D, int BN>
struct Cfg {
    static constexpr int DK = (D + 15) / 16 * 16;  // QK^T contraction length, padded to 16
    static constexpr int DV = (D + 31) / 32 * 32;  // PV output rows, padded to 32
    static constexpr int KSTEPS = DK / 16;
    static constexpr int DBLK = DV / 32;
    static constexpr int CH = D / 8;               // 16-byte chunks per K/V row
    static constexpr int KP = DK + 8;              // K tile row pitch (elements)
    static constexpr int VP = BN + 8;              // V^T tile row pitch (elements)
    static constexpr int K_ELEMS = BN * KP;
    static constexpr int V_ELEMS = DV * VP;
    static constexpr int STAGE = K_ELEMS + V_ELEMS;
    static constexpr int K_CHUNKS = BN * CH;
    static constexpr int K_LOADS = (K_CHUNKS + kThreads - 1) / kThreads;
    static constexpr int V_BLOCKS = (BN / 4) * CH;  // 4 rows x 8 dims per block
    static constexpr int V_LOADS = (V_BLOCKS + kThreads - 1) / kThreads;
    static constexpr int NKB = BN / 32;              // 32-key blocks of S^T
    static constexpr int NKS = BN / 16;              // 16-key PV steps
    static constexpr bool SUM_BY_MFMA = DV > D;      // a padding row of V^T holds ones
    static_assert(DK - D == 0 || DK - D == 8, "K padding is at most one 16-byte chunk");
};

struct Args {
    const uint16_t* q;
    const uint16_t* k;
    const uint16_t* v;
    const uint16_t* fk;
    const uint16_t* fv;
    uint16_t* wk;
    uint16_t* wv;
    uint16_t* out;
    float* lse;
    int B, H, Nq, Nk, off, len, q_tiles;
    float c2;  // softmax scale * log2(e)
};

typedef __amdgpu_buffer_rsrc_t Rsrc;

__device__ __forceinline__ Rsrc rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, kRsrcFlags);
}
__device__ __forceinline__ u32x4 bload(Rsrc r, uint32_t off) {
    return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
}
__device__ __forceinline__ void bstore(Rsrc r, uint32_t off, u32x4 x) {
    __builtin_amdgcn_raw_buffer_store_b128(x, r, off, 0, 0);
}

__device__ __forceinline__ int xcd_remap(int pid, int total) {
    const int per = total >> 3, rem = total & 7;
    const int xcd = pid & 7, loc = pid >> 3;
    return xcd * per + (xcd < rem ? xcd : rem) + loc;
}

// Position of key `key` (within a tile) in the V^T LDS rows: bits 2 and 3 of
// the index are swapped inside each group of 16 keys, so that the 8 keys a
// lane contributes to one PV k-step are contiguous.
__device__ __forceinline__ int vpos(int key) {
    return (key & ~15) | (key & 3) | ((key & 4) << 1) | ((key & 8) >> 1);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    const __bf16 a = (__bf16)lo, b = (__bf16)hi;
    return (uint32_t)__builtin_bit_cast(uint16_t, a) |
           ((uint32_t)__builtin_bit_cast(uint16_t, b) << 16);
}

// x combined with its value in the other 32-lane half (lane l <-> l ^ 32);
// the result is bit-identical in both lanes of a pair.
__device__ __forceinline__ float halves_max(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float halves_sum(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

template <int D, int BN, bool PATCH>
__global__ __launch_bounds__(kThreads, 2) void attn_bf16_kernel(Args a) {
    using C = Cfg<D, BN>;
    __shared__ __attribute__((aligned(16))) uint16_t lds[2 * C::STAGE];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int c = lane & 31, hf = lane >> 5;

    const int logical = xcd_remap(blockIdx.x, gridDim.x);
    const int qt = logical % a.q_tiles;
    const int bh = logical / a.q_tiles;
    const int hh = bh % a.H, b = bh / a.H;
    const uint32_t rowb = (uint32_t)a.H * D * 2;  // bytes between consecutive rows
    const uint32_t headb = (uint32_t)hh * D * 2;  // byte offset of this head in a row
    const bool writeback = PATCH && qt == 0;

    const int64_t kvbatch = (int64_t)b * a.Nk * a.H * D;
    const Rsrc rk = rsrc(a.k + kvbatch, (uint32_t)a.Nk * rowb);
    const Rsrc rv = rsrc(a.v + kvbatch, (uint32_t)a.Nk * rowb);
    Rsrc rfk = rk, rfv = rv, rwk = rk, rwv = rv;
    if constexpr (PATCH) {
        const int64_t fbatch = (int64_t)b * a.len * a.H * D;
        rfk = rsrc(a.fk + fbatch, (uint32_t)a.len * rowb);
        rfv = rsrc(a.fv + fbatch, (uint32_t)a.len * rowb);
        rwk = rsrc(a.wk + kvbatch, (uint32_t)a.Nk * rowb);
        rwv = rsrc(a.wv + kvbatch, (uint32_t)a.Nk * rowb);
    }

    // Padding of both stages, written once (tile stores never touch it):
    // K columns [D, DK) are zero; V^T rows [D, DV) are zero except row D,
    // which holds ones when the row sums are taken on the matrix cores.
    if constexpr (C::DK > D) {
        for (int e = tid; e < 2 * BN; e += kThreads) {
            const int s = e / BN, r = e % BN;
            *(u32x4*)(lds + s * C::STAGE + r * C::KP + D) = u32x4{0, 0, 0, 0};
        }
    }
    if constexpr (C::DV > D) {
        constexpr int PR = C::DV - D, CPR = BN / 8;
        for (int e = tid; e < 2 * PR * CPR; e += kThreads) {
            const int s = e / (PR * CPR), rem = e % (PR * CPR);
            const int r = D + rem / CPR, cc = rem % CPR;
            const uint32_t fill = r == D ? 0x3f803f80u : 0u;  // bf16 1.0 pairs
            *(u32x4*)(lds + s * C::STAGE + C::K_ELEMS + r * C::VP + 8 * cc) = u32x4{fill, fill, fill, fill};
        }
    }

    // The wave's 32 query rows, as B operands (lane: query c, dims 16kk+8hf..+7).
    const int qrow = qt * kBM + wave * 32 + c;
    const bool qvalid = qrow < a.Nq;
    const Rsrc rq = rsrc(a.q + (int64_t)b * a.Nq * a.H * D, (uint32_t)a.Nq * rowb);
    const Rsrc ro = rsrc(a.out + (int64_t)b * a.Nq * a.H * D, (uint32_t)a.Nq * rowb);
    bf16x8 qf[C::KSTEPS];
#pragma unroll
    for (int kk = 0; kk < C::KSTEPS; ++kk) {
        const int col = 16 * kk + 8 * hf;
        const uint32_t o = (qvalid && col < D) ? (uint32_t)qrow * rowb + headb + 2 * col : kOOB;
        qf[kk] = __builtin_bit_cast(bf16x8, bload(rq, o));
    }

    // Per-thread (row, byte column) of the chunks it stages; independent of
    // the tile.  A thread without a chunk gets column kOOB: row offsets stay
    // below 2^31 (checked by the host), so row + kOOB never wraps into range.
    int krow[C::K_LOADS];
    uint32_t kcol[C::K_LOADS];
#pragma unroll
    for (int i = 0; i < C::K_LOADS; ++i) {
        const int e = tid + i * kThreads;
        const bool ok = e < C::K_CHUNKS;
        krow[i] = ok ? e / C::CH : 0;
        kcol[i] = ok ? headb + 16 * (e % C::CH) : kOOB;
    }
    int vrg[C::V_LOADS];
    uint32_t vcol[C::V_LOADS];
#pragma unroll
    for (int i = 0; i < C::V_LOADS; ++i) {
        const int e = tid + i * kThreads;
        const bool ok = e < C::V_BLOCKS;
        vrg[i] = ok ? e / C::CH : 0;
        vcol[i] = ok ? headb + 16 * (e % C::CH) : kOOB;
    }

    auto in_slice = [&](int j) -> bool { return (unsigned)(j - a.off) < (unsigned)a.len; };
    // Byte offset of row j in the buffer source (out of range for fresh rows)
    // and in the fresh source (out of range for every other row).
    auto buf_off = [&](int j, uint32_t col) -> uint32_t {
        return (PATCH && in_slice(j)) ? kOOB : (uint32_t)j * rowb + col;
    };
    auto fresh_off = [&](int j, uint32_t col) -> uint32_t {
        return in_slice(j) ? (uint32_t)(j - a.off) * rowb + col : kOOB;
    };

    // Staged rows of the next tile: from the buffer / chunk source, and (patch
    // mode) from the fresh source.  Each row comes from exactly one of them;
    // the other reads as zero.  They are combined only when stored to LDS, so
    // no wait on the loads happens before the current tile is computed.
    u32x4 kreg[C::K_LOADS], vreg[4 * C::V_LOADS];
    u32x4 kfr[PATCH ? C::K_LOADS : 1], vfr[PATCH ? 4 * C::V_LOADS : 1];

    // Which sources a tile touches (uniform across the workgroup).
    auto tile_needs = [&](int t, bool& need_buf, bool& need_fresh) {
        const int lo = t * BN, hi = lo + BN;
        need_fresh = PATCH && a.len > 0 && lo < a.off + a.len && a.off < hi;
        need_buf = !PATCH || !(a.off <= lo && hi <= a.off + a.len);
    };

    auto load_tile = [&](int t) {
        bool need_buf, need_fresh;
        tile_needs(t, need_buf, need_fresh);
        const int base = t * BN;
#pragma unroll
        for (int i = 0; i < C::K_LOADS; ++i) kreg[i] = u32x4{0, 0, 0, 0};
#pragma unroll
        for (int i = 0; i < 4 * C::V_LOADS; ++i) vreg[i] = u32x4{0, 0, 0, 0};
        if (need_buf) {
#pragma unroll
            for (int i = 0; i < C::K_LOADS; ++i) kreg[i] = bload(rk, buf_off(base + krow[i], kcol[i]));
#pragma unroll
            for (int i = 0; i < C::V_LOADS; ++i)
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    vreg[4 * i + r] = bload(rv, buf_off(base + 4 * vrg[i] + r, vcol[i]));
        }
        if constexpr (PATCH) {
#pragma unroll
            for (int i = 0; i < C::K_LOADS; ++i) kfr[i] = u32x4{0, 0, 0, 0};
#pragma unroll
            for (int i = 0; i < 4 * C::V_LOADS; ++i) vfr[i] = u32x4{0, 0, 0, 0};
            if (need_fresh) {
#pragma unroll
                for (int i = 0; i < C::K_LOADS; ++i) kfr[i] = bload(rfk, fresh_off(base + krow[i], kcol[i]));
#pragma unroll
                for (int i = 0; i < C::V_LOADS; ++i)
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        vfr[4 * i + r] = bload(rfv, fresh_off(base + 4 * vrg[i] + r, vcol[i]));
            }
        }
    };

    auto store_tile = [&](int stage, int t) {
        uint16_t* Ks = lds + stage * C::STAGE;
        uint16_t* Vt = Ks + C::K_ELEMS;
        if constexpr (PATCH) {
#pragma unroll
            for (int i = 0; i < C::K_LOADS; ++i) kreg[i] |= kfr[i];
#pragma unroll
            for (int i = 0; i < 4 * C::V_LOADS; ++i) vreg[i] |= vfr[i];
        }
#pragma unroll
        for (int i = 0; i < C::K_LOADS; ++i) {
            const int e = tid + i * kThreads;
            if (C::K_CHUNKS % kThreads == 0 || e < C::K_CHUNKS)
                *(u32x4*)(Ks + krow[i] * C::KP + (e % C::CH) * 8) = kreg[i];
        }
#pragma unroll
        for (int i = 0; i < C::V_LOADS; ++i) {
            const int e = tid + i * kThreads;
            if (C::V_BLOCKS % kThreads == 0 || e < C::V_BLOCKS) {
                const int cc = e % C::CH;
                const u32x4 r0 = vreg[4 * i], r1 = vreg[4 * i + 1];
                const u32x4 r2 = vreg[4 * i + 2], r3 = vreg[4 * i + 3];
                const int pos = vpos(4 * vrg[i]);
#pragma unroll
                for (int w = 0; w < 4; ++w) {
                    // dims 8cc+2w (low halves) and 8cc+2w+1 (high halves) of the 4 rows
                    const u32x2 even = {(r0[w] & 0xffffu) | (r1[w] << 16),
                                        (r2[w] & 0xffffu) | (r3[w] << 16)};
                    const u32x2 odd = {(r0[w] >> 16) | (r1[w] & 0xffff0000u),
                                       (r2[w] >> 16) | (r3[w] & 0xffff0000u)};
                    *(u32x2*)(Vt + (8 * cc + 2 * w) * C::VP + pos) = even;
                    *(u32x2*)(Vt + (8 * cc + 2 * w + 1) * C::VP + pos) = odd;
                }
            }
        }
        if constexpr (PATCH) {
            bool need_buf, need_fresh;
            tile_needs(t, need_buf, need_fresh);
            if (writeback && need_fresh) {  // the fresh rows also go into the buffer
                const int base = t * BN;
#pragma unroll
                for (int i = 0; i < C::K_LOADS; ++i) {
                    const int j = base + krow[i];
                    bstore(rwk, in_slice(j) ? (uint32_t)j * rowb + kcol[i] : kOOB, kreg[i]);
                }
#pragma unroll
                for (int i = 0; i < C::V_LOADS; ++i)
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int j = base + 4 * vrg[i] + r;
                        bstore(rwv, in_slice(j) ? (uint32_t)j * rowb + vcol[i] : kOOB, vreg[4 * i + r]);
                    }
            }
        }
    };

    // Make sure the query registers are complete before the loop, so the
    // loop body never waits on memory operations other than the staged tile.
#pragma unroll
    for (int kk = 0; kk < C::KSTEPS; ++kk) asm volatile("" ::"v"(qf[kk]));

    f32x16 oacc[C::DBLK];
#pragma unroll
    for (int db = 0; db < C::DBLK; ++db) oacc[db] = f32x16{};
    float m_ref = -INFINITY;  // reference max of the raw dot products
    float l_run = 0.f;        // this lane's share of the running sum (VALU-summed case)
    const float thr = kRescaleLog2 / a.c2;

    const int ntiles = (a.Nk + BN - 1) / BN;
    if (ntiles > 0) {
        load_tile(0);
        store_tile(0, 0);
    }
    __syncthreads();

    for (int t = 0; t < ntiles; ++t) {
        if (t + 1 < ntiles) load_tile(t + 1);

        const uint16_t* Ks = lds + (t & 1) * C::STAGE;
        const uint16_t* Vt = Ks + C::K_ELEMS;

        // S^T for BN keys x 32 queries: sacc[kb][i] = score of key
        // 32kb + 8(i/4) + 4hf + (i%4) against query c.
        f32x16 sacc[C::NKB];
#pragma unroll
        for (int kb = 0; kb < C::NKB; ++kb) sacc[kb] = f32x16{};
#pragma unroll
        for (int kk = 0; kk < C::KSTEPS; ++kk) {
#pragma unroll
            for (int kb = 0; kb < C::NKB; ++kb) {
                const bf16x8 ka = *(const bf16x8*)(Ks + (32 * kb + c) * C::KP + 16 * kk + 8 * hf);
                sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qf[kk], sacc[kb], 0, 0, 0);
            }
        }

        if ((t + 1) * BN > a.Nk) {  // ragged last tile: keys past the end get -inf
#pragma unroll
            for (int kb = 0; kb < C::NKB; ++kb)
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const int key = t * BN + 32 * kb + 8 * (i >> 2) + 4 * hf + (i & 3);
                    if (key >= a.Nk) sacc[kb][i] = -INFINITY;
                }
        }

        float mx = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < C::NKB; ++kb)
#pragma unroll
            for (int i = 0; i < 16; ++i) mx = fmaxf(mx, sacc[kb][i]);
        mx = halves_max(mx);
        if (__builtin_amdgcn_ballot_w64(mx > m_ref + thr) != 0) {
            const float m_new = fmaxf(m_ref, mx);
            const float alpha = __builtin_amdgcn_exp2f((m_ref - m_new) * a.c2);
            m_ref = m_new;
            l_run *= alpha;
#pragma unroll
            for (int db = 0; db < C::DBLK; ++db) oacc[db] *= alpha;
        }
        const float mc = m_ref * a.c2;

#pragma unroll
        for (int kb = 0; kb < C::NKB; ++kb)
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[kb][i], a.c2, -mc));
                sacc[kb][i] = p;
                if constexpr (!C::SUM_BY_MFMA) l_run += p;
            }

        // O^T += V^T P^T over BN/16 k-steps of 16 keys.
#pragma unroll
        for (int ks = 0; ks < C::NKS; ++ks) {
            const int kb = ks >> 1, i0 = 8 * (ks & 1);
            u32x4 pw;
#pragma unroll
            for (int w = 0; w < 4; ++w) pw[w] = pack_bf16x2(sacc[kb][i0 + 2 * w], sacc[kb][i0 + 2 * w + 1]);
            const bf16x8 pb = __builtin_bit_cast(bf16x8, pw);
#pragma unroll
            for (int db = 0; db < C::DBLK; ++db) {
                const bf16x8 va = *(const bf16x8*)(Vt + (32 * db + c) * C::VP + 16 * ks + 8 * hf);
                oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb, oacc[db], 0, 0, 0);
            }
        }

        if (t + 1 < ntiles) store_tile((t + 1) & 1, t + 1);
        __syncthreads();
    }

    float l_tot;
    if constexpr (C::SUM_BY_MFMA) {
        // row D of O^T: block D/32, local row lr held by lanes of half (lr/4)&1
        constexpr int lr = D % 32, idx = 4 * (lr / 8) + (lr % 4), owner = (lr / 4) & 1;
        l_tot = __shfl(oacc[D / 32][idx], c + 32 * owner);
    } else {
        l_tot = halves_sum(l_run);
    }
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
#pragma unroll
    for (int db = 0; db < C::DBLK; ++db)
#pragma unroll
        for (int g = 0; g < 4; g += 2) {
            // dims 32db + 8g + 4hf .. +3 and 32db + 8(g+1) + 4hf .. +3
            const int dim = 32 * db + 8 * g + 4 * hf;
            if (dim < D) {
                const u32x2 w0 = {pack_bf16x2(oacc[db][4 * g] * inv, oacc[db][4 * g + 1] * inv),
                                  pack_bf16x2(oacc[db][4 * g + 2] * inv, oacc[db][4 * g + 3] * inv)};
                const uint32_t o = qvalid ? (uint32_t)qrow * rowb + headb + 2 * dim : kOOB;
                __builtin_amdgcn_raw_buffer_store_b64(w0, ro, o, 0, 0);
            }
            if (dim + 8 < D) {
                const int h2 = g + 1;
                const u32x2 w1 = {pack_bf16x2(oacc[db][4 * h2] * inv, oacc[db][4 * h2 + 1] * inv),
                                  pack_bf16x2(oacc[db][4 * h2 + 2] * inv, oacc[db][4 * h2 + 3] * inv)};
                const uint32_t o = qvalid ? (uint32_t)qrow * rowb + headb + 2 * (dim + 8) : kOOB;
                __builtin_amdgcn_raw_buffer_store_b64(w1, ro, o, 0, 0);
            }
        }
    if (a.lse && hf == 0 && qvalid) {
        const float lse = l_tot > 0.f ? (m_ref * a.c2 + __log2f(l_tot)) * 0.69314718055994531f : -INFINITY;
        a.lse[((int64_t)b * a.H + hh) * a.Nq + qrow] = lse;
    }
}

template <int D, int BN, bool PATCH>
hipError_t launch(const AttnParams& p, hipStream_t s) {
    Args a;
    a.q = (const uint16_t*)p.q;
    a.k = (const uint16_t*)p.k;
    a.v = (const uint16_t*)p.v;
    a.fk = (const uint16_t*)p.fresh_k;
    a.fv = (const uint16_t*)p.fresh_v;
    a.wk = (uint16_t*)p.wk;
    a.wv = (uint16_t*)p.wv;
    a.out = (uint16_t*)p.out;
    a.lse = p.lse;
    a.B = p.B;
    a.H = p.H;
    a.Nq = p.Nq;
    a.Nk = p.Nk;
    a.off = p.off;
    a.len = p.len;
    a.q_tiles = (p.Nq + kBM - 1) / kBM;
    a.c2 = (float)(1.4426950408889634 / sqrt((double)D));
    const int64_t blocks = (int64_t)a.q_tiles * p.H * p.B;
    if (blocks == 0) return hipSuccess;
    hipLaunchKernelGGL((attn_bf16_kernel<D, BN, PATCH>), dim3((unsigned)blocks), dim3(kThreads), 0, s, a);
    return hipGetLastError();
}

constexpr int kBN = 64;

}  // namespace

hipError_t launch_attn_bf16(const AttnParams& p, hipStream_t s) {
    const bool patch = p.fresh_k != nullptr;
    switch (p.D) {
        case 64: return patch ? launch<64, kBN, true>(p, s) : launch<64, kBN, false>(p, s);
        case 72: return patch ? launch<72, kBN, true>(p, s) : launch<72, kBN, false>(p, s);
        case 128: return patch ? launch<128, kBN, true>(p, s) : launch<128, kBN, false>(p, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace xdit
