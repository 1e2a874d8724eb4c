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
// Work decomposition (one workgroup = one query tile of one (batch, head))
//   * QB x KS waves: QB blocks of 32 query rows, and for each block KS waves
//     that split every K/V tile between them (each takes KW keys of the
//     BN = KS*KW-key tile).  The KS waves of a query block keep separate
//     running (max, sum, output) and are merged through LDS at the end, like
//     the chunk partials of the sequence-parallel merge.  Two or more waves
//     per SIMD let one wave's matrix work overlap another's softmax;
//   * K/V tiles are staged through LDS (double buffered, one barrier per
//     tile); the global loads of tile t+1 are in flight while tile t is
//     computed.  Loads go through buffer resources: a row past the end, or a
//     row served by the other source in patch mode, gets an out-of-range
//     offset and reads as zero, so no lane branches;
//   * scores are computed transposed, S^T = K Q^T, with
//     v_mfma_f32_32x32x16_bf16: A = K rows from LDS, B = the wave's Q rows
//     held in registers for the whole sweep.  In the 32x32 accumulator layout
//     each lane then holds 16 keys of ONE query, so the row max is in-lane
//     except for one exchange between the two 32-lane halves;
//   * online softmax in the log2 domain (scale*log2(e) folded into one FMA
//     before v_exp_f32).  The reference max is only raised when a row's tile
//     max exceeds it by more than 2^8 in weight, so the running output is
//     rescaled rarely; weights up to 2^8 lose nothing in bf16/float32 and the
//     final normalisation uses the same reference, so the result does not
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
#include <stdlib.h>
#include <string.h>

namespace xdit {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr uint32_t kOOB = 0x80000000u;  // offset past any buffer's range: reads 0, writes dropped
constexpr int kRsrcFlags = 0x00020000;  // raw buffer, 32-bit data format
constexpr float kRescaleLog2 = 8.0f;    // raise the reference max only beyond 2^8 growth

template <int D, int QB_, int KS_, int KW_>
struct Cfg {
    static constexpr int QB = QB_, KS = KS_, KW = KW_;
    static constexpr int NW = QB * KS;               // waves per workgroup
    static constexpr int THREADS = 64 * NW;
    static constexpr int BM = 32 * QB;               // query rows per workgroup
    static constexpr int BN = KS * KW;               // keys per tile
    static constexpr int DK = (D + 15) / 16 * 16;    // QK^T contraction length, padded to 16
    static constexpr int DV = (D + 31) / 32 * 32;    // PV output rows, padded to 32
    static constexpr int KSTEPS = DK / 16;
    static constexpr int DBLK = DV / 32;
    static constexpr int CH = D / 8;                 // 16-byte chunks per K/V row
    static constexpr int KP = DK + 8;                // K tile row pitch (elements)
    static constexpr int VP = BN + 8;                // V^T tile row pitch (elements)
    static constexpr int K_ELEMS = BN * KP;
    static constexpr int V_ELEMS = DV * VP;
    static constexpr int STAGE = K_ELEMS + V_ELEMS;
    static constexpr int K_CHUNKS = BN * CH;
    static constexpr int K_LOADS = (K_CHUNKS + THREADS - 1) / THREADS;
    static constexpr int V_BLOCKS = (BN / 4) * CH;   // 4 rows x 8 dims per block
    static constexpr int V_LOADS = (V_BLOCKS + THREADS - 1) / THREADS;
    static constexpr int NKB = KW / 32;              // 32-key blocks of S^T per wave
    static constexpr int NKS = KW / 16;              // 16-key PV steps per wave
    static constexpr bool SUM_BY_MFMA = DV > D;      // a padding row of V^T holds ones
    // end-of-sweep exchange: one slot (m, l, O^T accumulators) per partial wave
    static constexpr int XSLOT = 64 * (2 + 16 * DBLK);         // floats
    static constexpr int X_ELEMS = 2 * QB * (KS - 1) * XSLOT;  // in 2-byte units
    static constexpr int LDS_ELEMS = 2 * STAGE > X_ELEMS ? 2 * STAGE : X_ELEMS;
    static_assert(DK - D == 0 || DK - D == 8, "K padding is at most one 16-byte chunk");
    static_assert(KW % 32 == 0, "a wave takes whole 32-key blocks");
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

// Two floats to a packed bf16 pair (round to nearest even): one v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    typedef float f32x2_t __attribute__((ext_vector_type(2)));
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t{lo, hi}), bf16x2_t));
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

template <int D, int QB, int KS, int KW, bool PATCH>
__global__ __launch_bounds__(64 * QB * KS) void attn_bf16_kernel(Args a) {
    using C = Cfg<D, QB, KS, KW>;
    constexpr int NT = C::THREADS, BN = C::BN;
    __shared__ __attribute__((aligned(16))) uint16_t lds[C::LDS_ELEMS];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int c = lane & 31, hf = lane >> 5;
    const int qb = wave % QB, kh = wave / QB;  // query block, key split

    const int logical = xcd_remap(blockIdx.x, gridDim.x);
    const int qt = logical % a.q_tiles;
    const int bh = logical / a.q_tiles;
    const int hh = bh % a.H, b = bh / a.H;
    const uint32_t rowb = (uint32_t)a.H * D * 2;  // bytes between consecutive rows
    const uint32_t headb = (uint32_t)hh * D * 2;  // byte offset of this head in a row
    const bool writeback = PATCH && qt == 0;

    // Row 0 of this (batch, head) in each source; per-thread offsets are
    // then row * rowb + 16-byte column, and each tile gets its own buffer
    // resource (scalar work only) whose range ends at the source's last row,
    // so rows past the end read as zero and writes to them are dropped.
    const int64_t headoff = (int64_t)hh * D;
    const uint16_t* kbase = a.k + (int64_t)b * a.Nk * a.H * D + headoff;
    const uint16_t* vbase = a.v + (int64_t)b * a.Nk * a.H * D + headoff;
    const uint16_t* fkbase = PATCH ? a.fk + (int64_t)b * a.len * a.H * D + headoff : nullptr;
    const uint16_t* fvbase = PATCH ? a.fv + (int64_t)b * a.len * a.H * D + headoff : nullptr;
    // resource over rows [row0, rows) of a source starting at `base`
    auto rows_rsrc = [&](const uint16_t* base, int row0, int rows) -> Rsrc {
        return rsrc(base + (int64_t)row0 * a.H * D, (uint32_t)(rows - row0) * rowb - headb);
    };

    // LDS: two K stages then two V^T stages.  K tile t lives in K stage t%2
    // and V tile t in V stage t%2; K runs one tile ahead of V (see the loop).
    auto kstage = [&](int s) -> uint16_t* { return lds + s * C::K_ELEMS; };
    auto vstage = [&](int s) -> uint16_t* { return lds + 2 * C::K_ELEMS + s * C::V_ELEMS; };

    // Padding of every stage, written once (tile stores never touch it):
    // K columns [D, DK) are zero; V^T rows [D, DV) are zero except row D,
    // which holds ones when the row sums are taken on the matrix cores.
    if constexpr (C::DK > D) {
        for (int e = tid; e < 2 * BN; e += NT) {
            const int st = e / BN, r = e % BN;
            *(u32x4*)(kstage(st) + r * C::KP + D) = u32x4{0, 0, 0, 0};
        }
    }
    if constexpr (C::DV > D) {
        constexpr int PR = C::DV - D, CPR = BN / 8;
        for (int e = tid; e < 2 * PR * CPR; e += NT) {
            const int st = e / (PR * CPR), rem = e % (PR * CPR);
            const int r = D + rem / CPR, cc = rem % CPR;
            const uint32_t fill = r == D ? 0x3f803f80u : 0u;  // bf16 1.0 pairs
            *(u32x4*)(vstage(st) + r * C::VP + 8 * cc) = u32x4{fill, fill, fill, fill};
        }
    }

    // The block's 32 query rows, as B operands (lane: query c, dims 16kk+8hf..+7).
    const int qrow = qt * C::BM + qb * 32 + c;
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

    // Per-thread chunks it stages, independent of the tile: K chunk i is row
    // krow[i], 16-byte column kcol[i]; V block i is rows 4*vrg[i]..+3, column
    // vcc[i].  koff / voff are the byte offsets from the tile's first row; a
    // thread without a chunk gets kOOB, which no resource range reaches (row
    // offsets stay below 2^31, checked by the host).
    int krow[C::K_LOADS];
    uint32_t kcol[C::K_LOADS], koff[C::K_LOADS];
#pragma unroll
    for (int i = 0; i < C::K_LOADS; ++i) {
        const int e = tid + i * NT;
        const bool ok = e < C::K_CHUNKS;
        krow[i] = ok ? e / C::CH : 0;
        kcol[i] = 16 * (e % C::CH);
        koff[i] = ok ? (uint32_t)krow[i] * rowb + kcol[i] : kOOB;
    }
    // V blocks go row-group fastest across lanes: the transposed LDS writes
    // of a block land 8 rows apart per 16-byte column, so lanes that differed
    // in column would all hit the same banks.
    constexpr int RG = BN / 4;  // row groups per tile
    int vrg[C::V_LOADS], vcc[C::V_LOADS];
    uint32_t voff[C::V_LOADS];
#pragma unroll
    for (int i = 0; i < C::V_LOADS; ++i) {
        const int e = tid + i * NT;
        const bool ok = e < C::V_BLOCKS;
        vrg[i] = ok ? e % RG : 0;
        vcc[i] = ok ? e / RG : 0;
        voff[i] = ok ? (uint32_t)(4 * vrg[i]) * rowb + 16 * vcc[i] : kOOB;
    }

    auto in_slice = [&](int j) -> bool { return (unsigned)(j - a.off) < (unsigned)a.len; };

    // Where a tile's rows come from (uniform across the workgroup): all from
    // the buffer (or the chunk), all from the fresh rows, or both.
    enum { kBuf = 0, kFresh = 1, kMixed = 2 };
    auto tile_kind = [&](int t) -> int {
        if constexpr (!PATCH) return kBuf;
        const int lo = t * BN, hi = min(lo + BN, a.Nk);
        if (hi <= a.off || lo >= a.off + a.len) return kBuf;
        if (a.off <= lo && hi <= a.off + a.len) return kFresh;
        return kMixed;
    };

    u32x4 kreg[C::K_LOADS], vreg[4 * C::V_LOADS];

    // Global -> registers for K tile t.  A whole-tile source needs no
    // per-lane selects; a tile straddling a slice boundary (at most two per
    // sweep) reads each row from its own source, the other read returning
    // zero, and waits for its loads at once.
    auto load_k = [&](int t) {
        const int kind = tile_kind(t), lo = t * BN;
        if (kind != kMixed) {
            const Rsrc r = kind == kBuf ? rows_rsrc(kbase, lo, a.Nk) : rows_rsrc(fkbase, lo - a.off, a.len);
#pragma unroll
            for (int i = 0; i < C::K_LOADS; ++i) kreg[i] = bload(r, koff[i]);
        } else {
            const Rsrc rb = rows_rsrc(kbase, lo, a.Nk), rf = rows_rsrc(fkbase, 0, a.len);
#pragma unroll
            for (int i = 0; i < C::K_LOADS; ++i) {
                const int j = lo + krow[i];
                const bool f = in_slice(j) && koff[i] != kOOB;
                kreg[i] = bload(rb, f ? kOOB : koff[i]) |
                          bload(rf, f ? (uint32_t)(j - a.off) * rowb + kcol[i] : kOOB);
            }
        }
    };
    auto load_v = [&](int t) {
        const int kind = tile_kind(t), lo = t * BN;
        if (kind != kMixed) {
            const Rsrc r = kind == kBuf ? rows_rsrc(vbase, lo, a.Nk) : rows_rsrc(fvbase, lo - a.off, a.len);
#pragma unroll
            for (int i = 0; i < C::V_LOADS; ++i)
#pragma unroll
                for (int q = 0; q < 4; ++q) vreg[4 * i + q] = bload(r, voff[i] == kOOB ? kOOB : voff[i] + q * rowb);
        } else {
            const Rsrc rb = rows_rsrc(vbase, lo, a.Nk), rf = rows_rsrc(fvbase, 0, a.len);
#pragma unroll
            for (int i = 0; i < C::V_LOADS; ++i)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int j = lo + 4 * vrg[i] + q;
                    const bool f = in_slice(j) && voff[i] != kOOB;
                    const uint32_t o = voff[i] == kOOB ? kOOB : voff[i] + q * rowb;
                    vreg[4 * i + q] = bload(rb, f ? kOOB : o) |
                                      bload(rf, f ? (uint32_t)(j - a.off) * rowb + 16 * vcc[i] : kOOB);
                }
        }
    };

    // Registers -> LDS stage, plus (patch mode, first query tile only) the
    // fresh rows into the buffer.
    auto store_k = [&](int st, int t) {
        uint16_t* Ks = kstage(st);
#pragma unroll
        for (int i = 0; i < C::K_LOADS; ++i) {
            const int e = tid + i * NT;
            if (C::K_CHUNKS % NT == 0 || e < C::K_CHUNKS)
                *(u32x4*)(Ks + krow[i] * C::KP + kcol[i] / 2) = kreg[i];
        }
        if constexpr (PATCH) {
            const int kind = tile_kind(t), lo = t * BN;
            if (writeback && kind != kBuf) {
                const Rsrc rw = rows_rsrc(a.wk + (kbase - a.k), lo, a.Nk);
#pragma unroll
                for (int i = 0; i < C::K_LOADS; ++i) {
                    const bool f = kind == kFresh || in_slice(lo + krow[i]);
                    bstore(rw, f ? koff[i] : kOOB, kreg[i]);
                }
            }
        }
    };
    auto store_v = [&](int st, int t) {
        uint16_t* Vt = vstage(st);
#pragma unroll
        for (int i = 0; i < C::V_LOADS; ++i) {
            const int e = tid + i * NT;
            if (C::V_BLOCKS % NT == 0 || e < C::V_BLOCKS) {
                const int cc = vcc[i];
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
            const int kind = tile_kind(t), lo = t * BN;
            if (writeback && kind != kBuf) {
                const Rsrc rw = rows_rsrc(a.wv + (vbase - a.v), lo, a.Nk);
#pragma unroll
                for (int i = 0; i < C::V_LOADS; ++i)
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const bool f = kind == kFresh || in_slice(lo + 4 * vrg[i] + q);
                        const uint32_t o = voff[i] == kOOB ? kOOB : voff[i] + q * rowb;
                        bstore(rw, f ? o : kOOB, vreg[4 * i + q]);
                    }
            }
        }
    };

    const int kw0 = kh * KW;  // this wave's first key within a tile

    // S^T for this wave's KW keys of K tile in stage st x its 32 queries:
    // S[kb][i] = score of key kw0 + 32kb + 8(i/4) + 4hf + (i%4) against query c.
    auto qk = [&](int st, f32x16 (&S)[C::NKB]) {
        const uint16_t* Ks = kstage(st);
#pragma unroll
        for (int kb = 0; kb < C::NKB; ++kb) S[kb] = f32x16{};
#pragma unroll
        for (int kk = 0; kk < C::KSTEPS; ++kk)
#pragma unroll
            for (int kb = 0; kb < C::NKB; ++kb) {
                const bf16x8 ka = *(const bf16x8*)(Ks + (kw0 + 32 * kb + c) * C::KP + 16 * kk + 8 * hf);
                S[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qf[kk], S[kb], 0, 0, 0);
            }
    };
    // Keys of tile t past the end get -inf; the row max of the rest.
    auto mask_max = [&](int t, f32x16 (&S)[C::NKB]) -> float {
        if ((t + 1) * BN > a.Nk) {
#pragma unroll
            for (int kb = 0; kb < C::NKB; ++kb)
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const int key = t * BN + kw0 + 32 * kb + 8 * (i >> 2) + 4 * hf + (i & 3);
                    if (key >= a.Nk) S[kb][i] = -INFINITY;
                }
        }
        float mx = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < C::NKB; ++kb)
#pragma unroll
            for (int i = 0; i < 16; ++i) mx = fmaxf(mx, S[kb][i]);
        return halves_max(mx);
    };

    // Make sure the query registers are complete before the loop, so the
    // loop body never waits on memory operations other than the staged tiles.
#pragma unroll
    for (int kk = 0; kk < C::KSTEPS; ++kk) asm volatile("" ::"v"(qf[kk]));

    f32x16 oacc[C::DBLK];
#pragma unroll
    for (int db = 0; db < C::DBLK; ++db) oacc[db] = f32x16{};
    float m_ref = -INFINITY;  // reference max of the raw dot products (this wave's keys)
    float l_run = 0.f;        // this lane's share of the running sum (VALU-summed case)
    const float thr = kRescaleLog2 / a.c2;

    // Software pipeline over tiles.  Iteration t computes the weights of tile
    // t while the scores of tile t+1 run on the matrix cores, then P(t) V(t)
    // while the row max of tile t+1 and the staging of K(t+2), V(t+1) run on
    // the vector units.  So K tile t+1 and V tile t are read during iteration
    // t, and K(t+2) / V(t+1) are written into the stages that K(t) / V(t-1)
    // left free at the previous barrier: two stages each, one barrier per tile.
    const int ntiles = (a.Nk + BN - 1) / BN;
    f32x16 SA[C::NKB], SB[C::NKB];
    float mx = -INFINITY;
    if (ntiles > 0) {
        load_k(0);
        load_v(0);
        store_k(0, 0);
        store_v(0, 0);
        if (ntiles > 1) {
            load_k(1);
            store_k(1, 1);
        }
    }
    __syncthreads();
    if (ntiles > 0) {
        qk(0, SA);
        mx = mask_max(0, SA);
    }
    __syncthreads();  // K stage 0 is rewritten in iteration 0

    auto step = [&](int t, f32x16 (&S)[C::NKB], f32x16 (&Sn)[C::NKB]) {
        if (t + 2 < ntiles) load_k(t + 2);
        if (t + 1 < ntiles) load_v(t + 1);

        if (__builtin_amdgcn_ballot_w64(mx > m_ref + thr) != 0) {
            const float m_new = fmaxf(m_ref, mx);
            // m_new = -inf only while a wave has seen no valid key: keep alpha finite
            const float alpha = m_new == -INFINITY ? 1.f : __builtin_amdgcn_exp2f((m_ref - m_new) * a.c2);
            m_ref = m_new;
            l_run *= alpha;
#pragma unroll
            for (int db = 0; db < C::DBLK; ++db) oacc[db] *= alpha;
        }
        // with no valid key yet every score is -inf and any finite shift gives 0
        const float mc = m_ref == -INFINITY ? 0.f : m_ref * a.c2;

        // scores of tile t+1 (a tile past the end computes garbage that is
        // never used) || weights of tile t, packed as PV B operands
        qk((t + 1) & 1, Sn);
        bf16x8 pb[C::NKS];
#pragma unroll
        for (int ks = 0; ks < C::NKS; ++ks) {
            const int kb = ks >> 1, i0 = 8 * (ks & 1);
            float p[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                p[e] = __builtin_amdgcn_exp2f(__builtin_fmaf(S[kb][i0 + e], a.c2, -mc));
                if constexpr (!C::SUM_BY_MFMA) l_run += p[e];
            }
            u32x4 pw;
#pragma unroll
            for (int w = 0; w < 4; ++w) pw[w] = pack_bf16x2(p[2 * w], p[2 * w + 1]);
            pb[ks] = __builtin_bit_cast(bf16x8, pw);
        }

        // O^T += V^T P^T over KW/16 k-steps of 16 keys || row max of tile t+1
        const uint16_t* Vt = vstage(t & 1);
#pragma unroll
        for (int ks = 0; ks < C::NKS; ++ks)
#pragma unroll
            for (int db = 0; db < C::DBLK; ++db) {
                const bf16x8 va = *(const bf16x8*)(Vt + (32 * db + c) * C::VP + kw0 + 16 * ks + 8 * hf);
                oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb[ks], oacc[db], 0, 0, 0);
            }
        mx = mask_max(t + 1, Sn);

        if (t + 2 < ntiles) store_k(t & 1, t + 2);
        if (t + 1 < ntiles) store_v((t + 1) & 1, t + 1);
        __syncthreads();
    };
    for (int t = 0; t < ntiles; t += 2) {
        step(t, SA, SB);
        if (t + 1 < ntiles) step(t + 1, SB, SA);
    }

    // Merge the KS partial sweeps of each query block (the K/V stages are no
    // longer read: the loop ended with a barrier).  Slots are lane-major so
    // the exchange is free of bank conflicts.
    if constexpr (KS > 1) {
        float* xs = (float*)lds;
        if (kh > 0) {
            float* slot = xs + ((kh - 1) * QB + qb) * C::XSLOT;
            slot[lane] = m_ref;
            slot[64 + lane] = l_run;
#pragma unroll
            for (int db = 0; db < C::DBLK; ++db)
#pragma unroll
                for (int i = 0; i < 16; ++i) slot[(2 + 16 * db + i) * 64 + lane] = oacc[db][i];
        }
        __syncthreads();
        if (kh == 0) {
            float M = m_ref;
#pragma unroll
            for (int k2 = 1; k2 < KS; ++k2) M = fmaxf(M, xs[((k2 - 1) * QB + qb) * C::XSLOT + lane]);
            const float mM = M == -INFINITY ? 0.f : M;
            const float a0 = m_ref == -INFINITY ? 0.f : __builtin_amdgcn_exp2f((m_ref - mM) * a.c2);
            l_run *= a0;
#pragma unroll
            for (int db = 0; db < C::DBLK; ++db) oacc[db] *= a0;
#pragma unroll
            for (int k2 = 1; k2 < KS; ++k2) {
                const float* slot = xs + ((k2 - 1) * QB + qb) * C::XSLOT;
                const float mk = slot[lane];
                const float ak = mk == -INFINITY ? 0.f : __builtin_amdgcn_exp2f((mk - mM) * a.c2);
                l_run = __builtin_fmaf(ak, slot[64 + lane], l_run);
#pragma unroll
                for (int db = 0; db < C::DBLK; ++db)
#pragma unroll
                    for (int i = 0; i < 16; ++i)
                        oacc[db][i] = __builtin_fmaf(ak, slot[(2 + 16 * db + i) * 64 + lane], oacc[db][i]);
            }
            m_ref = M;
        }
    }
    if (kh != 0) return;

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
        for (int g = 0; g < 4; ++g) {
            // dims 32db + 8g + 4hf .. +3
            const int dim = 32 * db + 8 * g + 4 * hf;
            if (dim < D) {
                const u32x2 w = {pack_bf16x2(oacc[db][4 * g] * inv, oacc[db][4 * g + 1] * inv),
                                 pack_bf16x2(oacc[db][4 * g + 2] * inv, oacc[db][4 * g + 3] * inv)};
                const uint32_t o = qvalid ? (uint32_t)qrow * rowb + headb + 2 * dim : kOOB;
                __builtin_amdgcn_raw_buffer_store_b64(w, ro, o, 0, 0);
            }
        }
    if (a.lse && hf == 0 && qvalid) {
        const float lse = l_tot > 0.f ? (m_ref * a.c2 + __log2f(l_tot)) * 0.69314718055994531f : -INFINITY;
        a.lse[((int64_t)b * a.H + hh) * a.Nq + qrow] = lse;
    }
}

template <int D, int QB, int KS, int KW, bool PATCH>
hipError_t launch(const AttnParams& p, hipStream_t s) {
    using C = Cfg<D, QB, KS, KW>;
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
    a.q_tiles = (p.Nq + C::BM - 1) / C::BM;
    a.c2 = (float)(1.4426950408889634 / sqrt((double)D));
    const int64_t blocks = (int64_t)a.q_tiles * p.H * p.B;
    if (blocks == 0) return hipSuccess;
    hipLaunchKernelGGL((attn_bf16_kernel<D, QB, KS, KW, PATCH>), dim3((unsigned)blocks), dim3(C::THREADS),
                       0, s, a);
    return hipGetLastError();
}

// Two shapes of 8-wave workgroup: 128 query rows x 2 key splits of 64 keys,
// or 64 query rows x 4 key splits of 32 keys for query counts whose 128-row
// tiles would leave many of the 256 CUs idle.
constexpr int kCUs = 256;

double fill(int64_t blocks) {
    const int64_t rounds = (blocks + kCUs - 1) / kCUs;
    return rounds ? (double)blocks / (double)(rounds * kCUs) : 1.0;
}

// XDIT_ATTN_TILE=wide|narrow forces one shape (tuning and tests); anything
// else, or unset, picks by the fill estimate below.
int forced_shape() {
    const char* e = getenv("XDIT_ATTN_TILE");
    if (e == nullptr) return 0;
    if (strcmp(e, "wide") == 0) return 1;
    if (strcmp(e, "narrow") == 0) return 2;
    return 0;
}

template <int D, bool PATCH>
hipError_t dispatch(const AttnParams& p, hipStream_t s) {
    const int forced = forced_shape();
    if (forced == 1) return launch<D, 4, 2, 64, PATCH>(p, s);
    if (forced == 2) return launch<D, 2, 4, 32, PATCH>(p, s);
    // at d = 128 the wide shape's two score tiles do not fit in registers
    if constexpr (D > 96) return launch<D, 2, 4, 32, PATCH>(p, s);
    const int64_t bh = (int64_t)p.B * p.H;
    const int64_t wide = (p.Nq + 127) / 128 * bh, narrow = (p.Nq + 63) / 64 * bh;
    const double qfill_w = (double)p.Nq / ((p.Nq + 127) / 128 * 128.0);
    const double qfill_n = (double)p.Nq / ((p.Nq + 63) / 64 * 64.0);
    if (fill(narrow) * qfill_n > 1.1 * fill(wide) * qfill_w) return launch<D, 2, 4, 32, PATCH>(p, s);
    return launch<D, 4, 2, 64, PATCH>(p, s);
}

}  // namespace

hipError_t launch_attn_bf16(const AttnParams& p, hipStream_t s) {
    const bool patch = p.fresh_k != nullptr;
    switch (p.D) {
        case 64: return patch ? dispatch<64, true>(p, s) : dispatch<64, false>(p, s);
        case 72: return patch ? dispatch<72, true>(p, s) : dispatch<72, false>(p, s);
        case 128: return patch ? dispatch<128, true>(p, s) : dispatch<128, false>(p, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace xdit
