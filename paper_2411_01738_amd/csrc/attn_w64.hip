// bf16 attention with 64 query rows per wave and one wave per SIMD (head dim
// 128): the same operation as attn_bf16.hip (chunk attention with O and LSE,
// the fused PipeFusion patch step, the merge-into form and partitioned
// launches; Sections 4.1.1, 4.1.2 and 4.1.4 of arXiv 2411.01738), with a work
// decomposition that halves the LDS operand traffic per matrix product.
//
// Why: with 32 query rows per wave every 32x32x16 product reads a 1 KB K or
// V^T operand from LDS, so the operand reads of a tile take about as long as
// its products and the matrix pipes idle on LDS latency.  Here a wave holds
// two 32-row query blocks, and each K and V^T operand it reads feeds one
// product per block.
//
// Work decomposition (one workgroup = one 128-row query tile of one
// (batch, head), 4 waves, one per SIMD):
//   * waves = 2 query groups of 64 rows x 2 key splits; a K/V tile is 64
//     keys, each wave takes 32 of them;
//   * scores S^T = K Q^T on v_mfma_f32_32x32x16_bf16 with the K operand from
//     LDS and the wave's Q rows in registers (two blocks of 32), as in
//     attn_bf16.hip; the score accumulators stay in VGPRs;
//   * the output accumulators O^T (2 blocks x 128 dims x 32 queries = 128
//     registers per lane) live in AGPRs: the PV products are written as
//     inline assembly with AGPR accumulators, so the 256 VGPRs hold the
//     operands, scores and weights;
//   * every LDS operand read is issued by hand, several k-steps before its
//     product, with explicit lgkmcnt waits (LDS reads complete in issue
//     order), and the loop is ordered by hand in groups separated by
//     scheduling barriers (one wave per SIMD has no second wave to cover a
//     stall):
//       G1  QK products of tile t+1, under the weights (exps) of the second
//           half of tile t's keys; the V^T reads of tile t issued between
//           them;
//       G2a PV products of the first half of tile t's keys, under the row
//           max of tile t+1 and the reference-max update;
//       barrier; loads of tile t+4 into the stage tile t used; K reads of
//           tile t+2;
//       G2b PV products of the second half of tile t's keys (covering the K
//           reads' latency), under the weights of the first half of tile
//           t+1's keys;
//   * online softmax in base 2 with the lazy reference max of attn_bf16.hip;
//     row sums of the bf16 weights by v_dot2 with ones.
// Hazards the compiler cannot see in inline assembly are covered by explicit
// s_nop: a VALU read of an AGPR accumulator (rescale, epilogue) waits for the
// last PV product, and a PV product waits two cycles after the VALU writes of
// its weights.
#include "kernels.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <type_traits>

namespace xdit {
namespace {

#include "attn_common.h"

template <int D>
struct W64 {
    static_assert(D == 128, "this decomposition is built for head dim 128");
    static constexpr int QG = 2, KS = 2, KW = 32;  // query groups x key splits; keys per wave and tile
    static constexpr int NW = QG * KS, THREADS = 64 * NW;
    static constexpr int BM = 128;                 // query rows per workgroup (two blocks of 32 per wave)
    static constexpr int BN = KS * KW;             // keys per tile
    static constexpr int KSTEPS = D / 16;          // QK^T k-steps
    static constexpr int DBLK = D / 32;            // 32-row blocks of O^T
    static constexpr int CH = D / 8, ROWB = 16 * CH;
    // LDS row layout as in attn_bf16.hip at d = 128: chunk c of row r sits in
    // slot c ^ (r & 15), and the keys of every 16-key block are ordered by
    // krow so that the transposing V reads are free of bank conflicts; the
    // two half k-steps of a V^T read are 2 rows apart.
    static constexpr int E_ROWS = 2;
    __device__ static constexpr int swz(int r) { return r & 15; }
    static constexpr int TILE_BYTES = BN * ROWB;   // 16 KiB
    static constexpr int CONST_OFF = 2 * TILE_BYTES;
    static constexpr int STAGE_BYTES = 2 * TILE_BYTES + 32;
    static constexpr int NST = 4;
    static constexpr int DMA_PER_TILE = TILE_BYTES / 1024;
    static constexpr int DMA_PER_WAVE = DMA_PER_TILE / NW;  // loads of one K (or V) tile per wave
    static constexpr int Q_PIECES = BM * ROWB / 1024;
    static constexpr int Q_PER_WAVE = Q_PIECES / NW;
    static constexpr int NKS = KW / 16;            // PV k-steps per wave and tile
    // end-of-sweep exchange: per lane m, l of both blocks, then O^T
    static constexpr int XSLOT = 64 * (4 + 2 * 16 * DBLK);  // floats per wave
    static constexpr int LDS_BYTES = NST * STAGE_BYTES;
    static constexpr int SLOT_FLOATS = BM * (D + 1);
    static_assert(DMA_PER_TILE % NW == 0 && Q_PIECES % NW == 0, "even load shares");
    static_assert(BM * ROWB <= CONST_OFF, "the query tile fits a stage");
    static_assert(NST * STAGE_BYTES <= kLdsBytes, "LDS budget");
    static_assert(4 * QG * XSLOT <= LDS_BYTES, "exchange fits the stages");
    static_assert(BM == kPartSlotRows, "partial slots of 128 rows");
};

// Key of S^T row x (0..31) of a 32-key block: x = 16a + 8e + 4h + j is key
// 16a + 4j + 2e + h (the key order of attn_bf16.hip at d = 128).
__device__ __forceinline__ int krow128(int x) {
    return (x & 16) + 4 * (x & 3) + 2 * ((x >> 3) & 1) + ((x >> 2) & 1);
}

// LDS reads issued without a wait (the caller waits with lgkm_wait): a
// transposing 8-byte read at byte address a + OFF (lds_b128 of
// attn_common.h is the 16-byte one).
// the same into AGPRs (the query operands, read only by inline assembly)
__device__ __forceinline__ u32x4 lds_b128_agpr(uint32_t a) {
    u32x4 r;
    asm volatile("ds_read_b128 %0, %1" : "=a"(r) : "v"(a));
    return r;
}
template <int OFF>
__device__ __forceinline__ u32x2 lds_tr64(uint32_t a) {
    static_assert(OFF >= 0 && OFF < 65536, "ds offset range");
    u32x2 r;
    asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(r) : "v"(a), "i"(OFF));
    return r;
}
// Wait until at most N LDS operations of this wave are in flight, then mark
// the given registers as written after the wait, so that no use of them
// moves above it.
template <typename T>
__device__ __forceinline__ void hold(T& r) {
    asm volatile("" : "+v"(r));
}
template <int N, typename... R>
__device__ __forceinline__ void lgkm_wait(R&... r) {
    static_assert(N >= 0 && N <= 15, "lgkmcnt range");
    asm volatile("s_waitcnt lgkmcnt(%0)" ::"n"(N));
    (hold(r), ...);
}

// O^T += V^T P^T on the matrix cores with the accumulator in AGPRs.
__device__ __forceinline__ void mfma_acc(f32x16& acc, const u32x4& a, const bf16x8& b) {
    asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+a"(acc) : "v"(a), "v"(b));
}
// A VALU access of the accumulators waits out the last PV product that
// wrote them (18 wait states after a 16-pass product; one more for margin);
// every block passes through the statement, so that no read of any of them
// is placed above it.  The next PV product reading a block after a VALU
// write waits 2 more (acc_written).
__device__ __forceinline__ void acc_ready(f32x16 (&o)[2][4]) {
    asm volatile("s_nop 15\n\ts_nop 2"
                 : "+a"(o[0][0]), "+a"(o[0][1]), "+a"(o[0][2]), "+a"(o[0][3]), "+a"(o[1][0]), "+a"(o[1][1]),
                   "+a"(o[1][2]), "+a"(o[1][3]));
}
__device__ __forceinline__ void acc_written(f32x16& acc) {
    asm volatile("s_nop 3" : "+a"(acc));
}
// S^T (+)= K Q^T with the query operand in AGPRs (held there for the whole
// sweep) and the scores in VGPRs; FIRST starts from zero.  The scores may not
// share registers with the K operand.
// (The query operand is passed read-write: each of its definitions is then an
// AGPR one, and the register allocator keeps it there rather than in VGPRs
// copied over before every product.)
template <bool FIRST>
__device__ __forceinline__ void mfma_qk(f32x16& s, const u32x4& k, u32x4& q) {
    if constexpr (FIRST)
        asm volatile("v_mfma_f32_32x32x16_bf16 %0, %2, %1, 0" : "=&v"(s), "+a"(q) : "v"(k));
    else
        asm volatile("v_mfma_f32_32x32x16_bf16 %0, %2, %1, %0" : "+v"(s), "+a"(q) : "v"(k));
}
// A VALU read of scores waits out the last QK product that wrote them (18
// wait states after a 16-pass product; one more for margin).
__device__ __forceinline__ void scores_ready(f32x16 (&s)[2]) {
    asm volatile("s_nop 15\n\ts_nop 2" : "+v"(s[0]), "+v"(s[1]));
}

__device__ __forceinline__ void sched_fence() { __builtin_amdgcn_sched_barrier(0); }

// One segment: K/V tiles [tile0, tile0 + nt) of the sweep of pair `pair`;
// pslot: where its partial goes, nullptr for a whole sweep.
template <int D, bool PATCH, bool PARTS>
__device__ __forceinline__ void w64_segment(const Args& a, unsigned char* lds, int pair, int tile0, int nt,
                                            float* pslot) {
    using C = W64<D>;
    constexpr int NT = C::THREADS, BN = C::BN, NST = C::NST, KSTEPS = C::KSTEPS, DBLK = C::DBLK;

    int tid = threadIdx.x;
    if constexpr (PARTS) asm volatile("" : "+v"(tid));
    const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int c = lane & 31, hf = lane >> 5;
    const int qg = wave % C::QG, kh = wave / C::QG;  // query group, key split

    const int qt = pair % a.q_tiles, bh = pair / a.q_tiles;
    const int all_tiles = (a.Nk + BN - 1) / BN;
    const int tb = tile0;
    const int ntiles = max(0, min(nt, all_tiles - tile0));
    const int hh = bh % a.H, b = bh / a.H;
    const uint32_t rowb = (uint32_t)a.H * D * 2;
    const uint32_t headb = (uint32_t)hh * D * 2;
    const int64_t headoff = (int64_t)hh * D;
    const uint16_t* kbase = a.k + (int64_t)b * a.Nk * a.H * D + headoff;
    const uint16_t* vbase = a.v + (int64_t)b * a.Nk * a.H * D + headoff;
    const int F = a.len0 + a.len1;
    const uint16_t* fkbase = PATCH ? a.fk + (int64_t)b * F * a.H * D + headoff : nullptr;
    const uint16_t* fvbase = PATCH ? a.fv + (int64_t)b * F * a.H * D + headoff : nullptr;
    auto rows_rsrc = [&](const uint16_t* base, int row0, int rows) -> Rsrc {
        return rsrc(base + (int64_t)row0 * a.H * D, rows > row0 ? (uint32_t)(rows - row0) * rowb - headb : 0u);
    };
    auto stage = [&](int s) -> unsigned char* { return lds + s * C::STAGE_BYTES; };
    const uint32_t lds_u32 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) unsigned char*)lds;

    // the query tile goes to stage NST-1, which no K/V tile uses before the
    // first step; rows past Nq read as zero
    {
        const Rsrc rq = rows_rsrc(a.q + (int64_t)b * a.Nq * a.H * D + headoff, qt * C::BM, a.Nq);
#pragma unroll
        for (int n = 0; n < C::Q_PER_WAVE; ++n) {
            const int ins = wave + n * C::NW;
            const int p = 64 * ins + lane, r = p / C::CH;
            dma16(rq, stage(NST - 1) + 1024 * ins, (uint32_t)r * rowb + 16 * ((p % C::CH) ^ C::swz(r)));
        }
    }
    uint32_t dma_off[C::DMA_PER_WAVE];
#pragma unroll
    for (int n = 0; n < C::DMA_PER_WAVE; ++n) {
        const int p = 64 * (wave + n * C::NW) + lane;
        const int r = p / C::CH, pc = p % C::CH;
        dma_off[n] = (uint32_t)r * rowb + 16 * (pc ^ C::swz(r));
    }
    // loads of K and V tile t into stage s: the short path for tiles of
    // buffer (or chunk) rows, the long one for the few tiles of a patch that
    // hold fresh rows
    auto load_tile = [&](int t, int s) {
        const int gt = tb + t, lo = gt * BN;
        unsigned char* kdst = stage(s);
        unsigned char* vdst = stage(s) + C::TILE_BYTES;
        auto issue = [&](Rsrc rk, Rsrc rv) {
#pragma unroll
            for (int n = 0; n < C::DMA_PER_WAVE; ++n) {
                const int ins = wave + n * C::NW;
                dma16(rk, kdst + 1024 * ins, dma_off[n]);
                dma16(rv, vdst + 1024 * ins, dma_off[n]);
            }
        };
        // (chunk launches take the same test, whose ranges are empty: with
        // the loads on one straight path the compiler's register allocation
        // of this loop spilled)
        const bool plain = (unsigned)(gt - a.sa0) >= (unsigned)a.sn0 && (unsigned)(gt - a.sa1) >= (unsigned)a.sn1;
        if (__builtin_expect(plain, 1)) {
            issue(rows_rsrc(kbase, lo, a.Nk), rows_rsrc(vbase, lo, a.Nk));
            return;
        }
        const int hi = min(lo + BN, a.Nk);
        const bool all0 = a.off0 <= lo && hi <= a.off0 + a.len0;
        const bool all1 = a.off1 <= lo && hi <= a.off1 + a.len1;
        if (all0 || all1) {
            const int fbase = all0 ? -a.off0 : a.len0 - a.off1;
            const int fend = all0 ? a.len0 : F;
            issue(rows_rsrc(fkbase, lo + fbase, fend), rows_rsrc(fvbase, lo + fbase, fend));
            return;
        }
        const Rsrc rk = rows_rsrc(kbase, lo, a.Nk), rv = rows_rsrc(vbase, lo, a.Nk);
        const Rsrc fk = rows_rsrc(fkbase, 0, F), fv = rows_rsrc(fvbase, 0, F);
#pragma unroll
        for (int n = 0; n < C::DMA_PER_WAVE; ++n) {
            const int ins = wave + n * C::NW;
            const int r = (64 * ins + lane) / C::CH;
            const int j = lo + r;
            const bool in0 = (unsigned)(j - a.off0) < (unsigned)a.len0;
            const bool in1 = (unsigned)(j - a.off1) < (unsigned)a.len1;
            if (in0 || in1) {
                const int fr = in0 ? j - a.off0 : a.len0 + j - a.off1;
                const uint32_t o = dma_off[n] + (uint32_t)(fr - r) * rowb;
                dma16(fk, kdst + 1024 * ins, o);
                dma16(fv, vdst + 1024 * ins, o);
            } else {
                dma16(rk, kdst + 1024 * ins, dma_off[n]);
                dma16(rv, vdst + 1024 * ins, dma_off[n]);
            }
        }
    };
    // every wave issues 2 * DMA_PER_WAVE loads per tile (twice as many for a
    // tile that straddles a fresh range's edge, which only makes a wait
    // stricter)
    constexpr int LPT = 2 * C::DMA_PER_WAVE;

    // LDS byte offsets (within a stage) of this lane's operand reads.
    //  K: row kw0 + krow(c), logical chunk 2kk + hf.
    //  V^T: in each 16-lane group, lane 4j+q reads dims d0+4q..+3 of key
    //  kw0 + 16ks + krow(8e + 4hf + j), d0 = 32db + 16(group & 1), e the
    //  half k-step; lane i of the group then holds dim d0 + i of four keys in
    //  the order of the weights P (the S^T rows).
    const int kw0 = kh * C::KW;
    uint32_t kaddr[KSTEPS];
    {
        const int r = kw0 + krow128(c);
#pragma unroll
        for (int kk = 0; kk < KSTEPS; ++kk) kaddr[kk] = r * C::ROWB + 16 * ((2 * kk + hf) ^ C::swz(r));
    }
    const int gi = lane & 15, grp = lane >> 4;
    uint32_t vaddr[DBLK][2];
    {
        const int vkey0 = kw0 + krow128(4 * hf + (gi >> 2));
#pragma unroll
        for (int db = 0; db < DBLK; ++db) {
            const int dim = 32 * db + 16 * (grp & 1) + 4 * (gi & 3);
#pragma unroll
            for (int e = 0; e < 2; ++e) {
                const int r = vkey0 + C::E_ROWS * e;
                vaddr[db][e] = C::TILE_BYTES + r * C::ROWB + 16 * ((dim >> 3) ^ C::swz(r)) + 2 * (dim & 7);
            }
        }
    }

    // O^T accumulators (AGPRs): oacc[qb][db] = dims 32db.. of query block qb
    f32x16 oacc[2][DBLK];
#pragma unroll
    for (int qb = 0; qb < 2; ++qb)
#pragma unroll
        for (int db = 0; db < DBLK; ++db) oacc[qb][db] = f32x16{};
    float m_ref[2] = {-INFINITY, -INFINITY};  // reference max of the raw dot products
    float l_run[2] = {0.f, 0.f};              // this lane's share of the running sums
    float mc[2] = {0.f, 0.f};                 // m_ref * c2
    const float thr = kRescaleLog2 / a.c2;

    // The query operands: block qb of this wave's group, read from LDS after
    // the prologue's barrier
    u32x4 qf[2][KSTEPS];

    // K reads of tile t: kr[kk] = the A operand of k-step kk, issued
    // KAHEAD k-steps ahead of their products
    constexpr int KAHEAD = 4;
    u32x4 kr[KSTEPS];
    auto k_stage = [&](int t) -> uint32_t { return lds_u32 + (uint32_t)((t % NST) * C::STAGE_BYTES); };
    auto read_k = [&](uint32_t st, auto kc) {
        constexpr int kk = decltype(kc)::value;
        kr[kk] = lds_b128<0>(st + kaddr[kk]);
    };
    // keys past the end of a ragged last tile get -inf
    auto mask = [&](int t, f32x16 (&s)[2]) {
        if ((tb + t + 1) * BN > a.Nk) {
#pragma unroll
            for (int qb = 0; qb < 2; ++qb)
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const int key = (tb + t) * BN + kw0 + krow128(8 * (i >> 2) + 4 * hf + (i & 3));
                    if (key >= a.Nk) s[qb][i] = -INFINITY;
                }
        }
    };
    auto row_max = [&](const f32x16& s) -> float {
        f32x16 x = s;
        asm volatile("" : "+v"(x));
        float mx = -INFINITY;
#pragma unroll
        for (int i = 0; i < 16; ++i) mx = fmaxf(mx, x[i]);
        mx = halves_max(mx);
        asm volatile("" : "+v"(mx));
        return mx;
    };
    // Weights of block qb, keys 16ks+2w, 16ks+2w+1 of the wave's 32 (score
    // registers 8ks+2w, +1): a packed bf16 pair, element w of the B operand
    // of PV k-step ks.  The row sums of the bf16 weights go to l_run by
    // v_dot2 with ones.
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    typedef float f32x2_t __attribute__((ext_vector_type(2)));
    // The scores enter and the packed pair leaves through empty volatile
    // asm statements, which keep their order with the other volatile
    // statements of the loop: the compiler can then move this arithmetic
    // neither above the unit it is written in nor below it (scheduling
    // barriers alone do not stop code motion before instruction selection).
    auto weight_pair = [&](const f32x16& s, int qb, int ks, int w) -> uint32_t {
        const bf16x2_t ones = {(__bf16)1.0f, (__bf16)1.0f};
        float x0 = s[8 * ks + 2 * w], x1 = s[8 * ks + 2 * w + 1];
        asm volatile("" : "+v"(x0), "+v"(x1));
        const float p0 = __builtin_amdgcn_exp2f(__builtin_fmaf(x0, a.c2, -mc[qb]));
        const float p1 = __builtin_amdgcn_exp2f(__builtin_fmaf(x1, a.c2, -mc[qb]));
        const bf16x2_t pp = __builtin_convertvector((f32x2_t{p0, p1}), bf16x2_t);
        l_run[qb] = __builtin_amdgcn_fdot2_f32_bf16(pp, ones, l_run[qb], false);
        uint32_t r = __builtin_bit_cast(uint32_t, pp);
        asm volatile("" : "+v"(r), "+v"(l_run[qb]));
        return r;
    };
    auto weights = [&](const f32x16& s, int qb, int ks) -> bf16x8 {
        u32x4 pw;
#pragma unroll
        for (int w = 0; w < 4; ++w) pw[w] = weight_pair(s, qb, ks, w);
        return __builtin_bit_cast(bf16x8, pw);
    };

    // Raise the reference max if a block's tile max exceeds it by more than
    // 2^8 in weight; returns whether the O accumulators must be rescaled
    // (by alpha, applied by the caller once the tile's PV products are in)
    float alpha[2] = {1.f, 1.f};
    auto update_max = [&](float mx0, float mx1) -> bool {
        const bool up = __builtin_amdgcn_ballot_w64(mx0 > m_ref[0] + thr || mx1 > m_ref[1] + thr) != 0;
        if (up) {
            const float mx[2] = {mx0, mx1};
#pragma unroll
            for (int qb = 0; qb < 2; ++qb) {
                const float m_new = fmaxf(m_ref[qb], mx[qb]);
                alpha[qb] = m_new == -INFINITY ? 1.f : __builtin_amdgcn_exp2f((m_ref[qb] - m_new) * a.c2);
                m_ref[qb] = m_new;
                l_run[qb] *= alpha[qb];
            }
        }
#pragma unroll
        for (int qb = 0; qb < 2; ++qb) mc[qb] = m_ref[qb] == -INFINITY ? 0.f : m_ref[qb] * a.c2;
        return up;
    };
    // O *= alpha (rare), one accumulator block at a time
    auto rescale_o = [&]() {
        acc_ready(oacc);
#pragma unroll
        for (int qb = 0; qb < 2; ++qb)
#pragma unroll
            for (int db = 0; db < DBLK; ++db) {
                oacc[qb][db] *= alpha[qb];
                acc_written(oacc[qb][db]);
                sched_fence();
            }
    };

    // V^T operands of tile t: vr[ks][db] (two transposing reads each)
    u32x2 vr[C::NKS][DBLK][2];
    bf16x8 pb0[2], pb1[2];  // weights of the first / second half of the wave's keys
    u32x4 pw[2];            // pairs of weights being assembled

    // One step t: PV of tile t, QK of tile t+1 (NEXT), K reads of tile t+2
    // (issued after the barrier when it exists).  On entry: sc = S of tile
    // t, pb0 = its first-half weights, kr = K reads of tile t+1 in flight
    // (NEXT), no other LDS read in flight.
    const bool ragged = ntiles > 0 && (tb + ntiles) * BN > a.Nk;
    auto step = [&](int t, f32x16 (&sc)[2], f32x16 (&sn)[2], auto next_c) {
        constexpr bool NEXT = decltype(next_c)::value;
        const uint32_t vst = lds_u32 + (uint32_t)((t % NST) * C::STAGE_BYTES);
        // ---- G1: QK of tile t+1 | second-half weights of tile t | V^T reads of tile t
        // LDS reads in issue order over a step: K reads 0..KAHEAD-1 of tile
        // t+1 (issued before G2b of the previous step); in G1 unit u, the K
        // read u + KAHEAD and the V^T read u of the first half; in G2a unit
        // db, the V^T reads 2db, 2db+1 of the second half.  Reads complete
        // in issue order, so a wait for one read is a wait until at most
        // the reads issued after it are in flight:
        //   K read kk at G1 unit kk: the later K reads issued so far and the
        //   V^T reads issued after it;
        constexpr auto g1_after = [](int kk) {
            const int kmax = KAHEAD - 1 + kk < KSTEPS - 1 ? KAHEAD - 1 + kk : KSTEPS - 1;
            return (kmax - kk) + (kk < KAHEAD ? kk : KAHEAD);
        };
        static_assert(KSTEPS == 2 * DBLK, "one first-half V^T read per QK k-step");
        const uint32_t kst = k_stage(t + 1);
        static_for<0, KSTEPS>([&](auto kc) {
            constexpr int kk = decltype(kc)::value;
            if constexpr (NEXT) {
                lgkm_wait<g1_after(kk)>(kr[kk]);
                mfma_qk<kk == 0>(sn[0], kr[kk], qf[0][kk]);
                mfma_qk<kk == 0>(sn[1], kr[kk], qf[1][kk]);
                if constexpr (kk + KAHEAD < KSTEPS) read_k(kst, std::integral_constant<int, kk + KAHEAD>{});
            }
            // V^T read kk of the first half: block db = kk / 2, half step e = kk % 2
            vr[0][kk / 2][kk % 2] = lds_tr64<0>(vst + vaddr[kk / 2][kk % 2]);
            // one pair of the second half's weights: block kk / 4, pair kk % 4
            pw[kk / 4][kk % 4] = weight_pair(sc[kk / 4], kk / 4, 1, kk % 4);
            if constexpr (kk % 4 == 3) pb1[kk / 4] = __builtin_bit_cast(bf16x8, pw[kk / 4]);
            sched_fence();
        });
        // ---- G2a: PV of the first half | row max of tile t+1, max update
        float mx[2] = {0.f, 0.f};
        bool rescale = false;
        static_for<0, DBLK>([&](auto dc) {
            constexpr int db = decltype(dc)::value;
            // V^T reads 2db, 2db+1 of the first half: issued after them, the
            // first half's 6 - 2db later ones and the second half's 2db
            lgkm_wait<6>(vr[0][db][0], vr[0][db][1]);
            const u32x4 v4 = {vr[0][db][0][0], vr[0][db][0][1], vr[0][db][1][0], vr[0][db][1][1]};
            mfma_acc(oacc[0][db], v4, pb0[0]);
            mfma_acc(oacc[1][db], v4, pb0[1]);
            vr[1][db][0] = lds_tr64<16 * C::ROWB>(vst + vaddr[db][0]);
            vr[1][db][1] = lds_tr64<16 * C::ROWB>(vst + vaddr[db][1]);
            if constexpr (NEXT && db == 0) scores_ready(sn);
            if constexpr (NEXT) {
                if constexpr (db == 0)
                    if (ragged && t + 2 == ntiles) mask(t + 1, sn);
                if constexpr (db == 1) mx[0] = row_max(sn[0]);
                if constexpr (db == 2) mx[1] = row_max(sn[1]);
                if constexpr (db == DBLK - 1) rescale = update_max(mx[0], mx[1]);
            }
            sched_fence();
        });
        // ---- barrier; loads of tile t+4 into this tile's stage; K reads of tile t+2
        const bool k2 = t + 2 < ntiles;
        if (k2) {
            // V^T reads of tile t are all in registers before its stage is refilled
            lgkm_wait<0>(vr[1][0][0], vr[1][0][1], vr[1][1][0], vr[1][1][1], vr[1][2][0], vr[1][2][1],
                         vr[1][3][0], vr[1][3][1]);
            // tile t+2 must have landed; tile t+3 (issued at step t-1, or
            // not at all at step 0) may still be in flight
            if (t >= 1 && t + 3 < ntiles) wait_vmem<LPT>();
            else wait_vmem<0>();
            asm volatile("" ::: "memory");
            __builtin_amdgcn_s_barrier();
            asm volatile("" ::: "memory");
            if (t == 0 && 3 < ntiles) load_tile(3, 3);  // stage 3 held the query tile until now
            if (t + 4 < ntiles) load_tile(t + 4, t % NST);
            const uint32_t st2 = k_stage(t + 2);
            static_for<0, KAHEAD>([&](auto kc) { read_k(st2, kc); });
        }
        sched_fence();
        // ---- G2b: PV of the second half | first-half weights of tile t+1
        static_for<0, DBLK>([&](auto dc) {
            constexpr int db = decltype(dc)::value;
            // (after the barrier the second half's reads have all landed)
            if (!k2) lgkm_wait<2 * DBLK - 2 * (db + 1)>(vr[1][db][0], vr[1][db][1]);
            const u32x4 v4 = {vr[1][db][0][0], vr[1][db][0][1], vr[1][db][1][0], vr[1][db][1][1]};
            mfma_acc(oacc[0][db], v4, pb1[0]);
            mfma_acc(oacc[1][db], v4, pb1[1]);
            if constexpr (NEXT) {
                // two pairs of the first half's weights of tile t+1 per unit
                constexpr int qb = db / 2, w0 = 2 * (db % 2);
                pw[qb][w0] = weight_pair(sn[qb], qb, 0, w0);
                pw[qb][w0 + 1] = weight_pair(sn[qb], qb, 0, w0 + 1);
                if constexpr (db % 2 == 1) pb0[qb] = __builtin_bit_cast(bf16x8, pw[qb]);
            }
            sched_fence();
        });
        if (rescale) rescale_o();
        sched_fence();
    };
    using T_ = std::true_type;
    using F_ = std::false_type;

    // Prologue: the query tile and tiles 0..2 load; tiles 0 and 1 (and the
    // query tile) must land, tile 2 may still be in flight.
#pragma unroll
    for (int t = 0; t < NST - 1; ++t) load_tile(t, t);
    wait_vmem<LPT>();
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    {
        // by hand, as the operand reads: a compiler-issued LDS read would wait
        // for the tile loads in flight, whose LDS bytes it cannot tell apart
        const uint32_t qst = lds_u32 + (uint32_t)((NST - 1) * C::STAGE_BYTES);
        static_for<0, 2>([&](auto qc) {
            constexpr int qb = decltype(qc)::value;
            const int r = qg * 64 + qb * 32 + c;
            static_for<0, KSTEPS>([&](auto kc) {
                constexpr int kk = decltype(kc)::value;
                qf[qb][kk] = lds_b128_agpr(qst + 16 * (r * C::CH + ((2 * kk + hf) ^ C::swz(r))));
            });
        });
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
        for (int qb = 0; qb < 2; ++qb)
#pragma unroll
            for (int kk = 0; kk < KSTEPS; ++kk) asm volatile("" : "+a"(qf[qb][kk]));
    }
    f32x16 sA[2], sB[2];
    if (ntiles > 0) {
        // S of tile 0, its max, its first-half weights; the first K reads
        // of tile 1
        const uint32_t st0 = k_stage(0);
        static_for<0, KSTEPS>([&](auto kc) { read_k(st0, kc); });
        static_for<0, KSTEPS>([&](auto kc) {
            constexpr int kk = decltype(kc)::value;
            lgkm_wait<KSTEPS - 1 - kk>(kr[kk]);
            mfma_qk<kk == 0>(sA[0], kr[kk], qf[0][kk]);
            mfma_qk<kk == 0>(sA[1], kr[kk], qf[1][kk]);
        });
        scores_ready(sA);
        if (ntiles > 1) {
            const uint32_t st1 = k_stage(1);
            static_for<0, KAHEAD>([&](auto kc) { read_k(st1, kc); });
        }
        mask(0, sA);
        update_max(row_max(sA[0]), row_max(sA[1]));
        pb0[0] = weights(sA[0], 0, 0);
        pb0[1] = weights(sA[1], 1, 0);
    }
    sched_fence();
    // steps with a next tile in pairs (the score buffers swap roles), then
    // the last tile's PV alone
    int t = 0;
    for (;;) {
        if (t + 1 >= ntiles) break;
        step(t, sA, sB, T_{});
        ++t;
        if (t + 1 >= ntiles) {
            sA[0] = sB[0];
            sA[1] = sB[1];
            break;
        }
        step(t, sB, sA, T_{});
        ++t;
    }
    if (t < ntiles) step(t, sA, sB, F_{});
    // no tile load in flight (fewer than three tiles leave prologue loads
    // outstanding), every wave done with the stages
    wait_vmem<0>();
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    __syncthreads();

    // Patch mode: this workgroup's share of the fresh rows goes into the
    // buffer (as in attn_bf16.hip: the share of this segment's units)
    constexpr int CU = 4;
    const int64_t hu = (int64_t)a.q_tiles * a.T, u0 = (int64_t)qt * a.T + tile0;
    const int cr0 = (int)((int64_t)F * u0 / hu);
    const int cn = ((int)((int64_t)F * (u0 + nt) / hu) - cr0) * C::CH;
    uint32_t cd[CU];
    u32x4 ck[CU], cv[CU];
    auto copy_load = [&](int e0) {
        const Rsrc fk = rows_rsrc(fkbase, 0, F), fv = rows_rsrc(fvbase, 0, F);
#pragma unroll
        for (int u = 0; u < CU; ++u) {
            const int e = e0 + tid + u * NT;
            const int fr = cr0 + e / C::CH, cc = 16 * (e % C::CH);
            const int j = fr < a.len0 ? a.off0 + fr : a.off1 + fr - a.len0;
            const uint32_t cs = e < cn ? (uint32_t)fr * rowb + cc : kOOB;
            cd[u] = e < cn ? (uint32_t)j * rowb + cc : kOOB;
            ck[u] = bload(fk, cs);
            cv[u] = bload(fv, cs);
        }
    };
    auto copy_rest = [&]() {
        const Rsrc wk = rows_rsrc(a.wk + (kbase - a.k), 0, a.Nk);
        const Rsrc wv = rows_rsrc(a.wv + (vbase - a.v), 0, a.Nk);
        for (int e0 = 0;;) {
#pragma unroll
            for (int u = 0; u < CU; ++u) {
                bstore(wk, cd[u], ck[u]);
                bstore(wv, cd[u], cv[u]);
            }
            e0 += CU * NT;
            if (e0 >= cn) break;
            copy_load(e0);
        }
    };
    if constexpr (PATCH) copy_load(0);


    // Merge the two key splits of each query group through LDS (lane-major
    // slots: no bank conflicts)
    acc_ready(oacc);
    {
        float* xs = (float*)lds;
        float* slot = xs + qg * C::XSLOT;
        if (kh == 1) {
#pragma unroll
            for (int qb = 0; qb < 2; ++qb) {
                slot[(2 * qb) * 64 + lane] = m_ref[qb];
                slot[(2 * qb + 1) * 64 + lane] = l_run[qb];
#pragma unroll
                for (int db = 0; db < DBLK; ++db)
#pragma unroll
                    for (int i = 0; i < 16; ++i) slot[(4 + (qb * DBLK + db) * 16 + i) * 64 + lane] = oacc[qb][db][i];
            }
        }
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
        if (kh == 0) {
#pragma unroll
            for (int qb = 0; qb < 2; ++qb) {
                const float mk = slot[(2 * qb) * 64 + lane];
                const float M = fmaxf(m_ref[qb], mk);
                const float mM = M == -INFINITY ? 0.f : M;
                const float a0 = m_ref[qb] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f((m_ref[qb] - mM) * a.c2);
                const float a1 = mk == -INFINITY ? 0.f : __builtin_amdgcn_exp2f((mk - mM) * a.c2);
                l_run[qb] = __builtin_fmaf(a1, slot[(2 * qb + 1) * 64 + lane], l_run[qb] * a0);
#pragma unroll
                for (int db = 0; db < DBLK; ++db)
#pragma unroll
                    for (int i = 0; i < 16; ++i)
                        oacc[qb][db][i] = __builtin_fmaf(a1, slot[(4 + (qb * DBLK + db) * 16 + i) * 64 + lane],
                                                         oacc[qb][db][i] * a0);
                m_ref[qb] = M;
            }
        }
    }
    if (kh != 0) {
        if constexpr (PATCH) copy_rest();
        return;
    }

    const Rsrc ro = rsrc(a.out + (int64_t)b * a.Nq * a.H * D, (uint32_t)a.Nq * rowb);
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
        const int r = qg * 64 + qb * 32 + c;  // row within the tile
        const int qrow = qt * C::BM + r;
        const bool qvalid = qrow < a.Nq;
        const float l_tot = halves_sum(l_run[qb]);
        const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
        constexpr float kLn2 = 0.69314718055994531f;
        const float lse_new = l_tot > 0.f ? (m_ref[qb] * a.c2 + __log2f(l_tot)) * kLn2 : -INFINITY;
        if (pslot != nullptr) {
            // partial sweep: normalised O and the LSE in float32 for the
            // fix-up; chunk k4 (dims 4k4..4k4+3) of tile row r at float4 k4*BM + r
            f32x4* po = (f32x4*)pslot;
#pragma unroll
            for (int db = 0; db < DBLK; ++db)
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const f32x4 y = {oacc[qb][db][4 * g] * inv, oacc[qb][db][4 * g + 1] * inv,
                                     oacc[qb][db][4 * g + 2] * inv, oacc[qb][db][4 * g + 3] * inv};
                    po[(8 * db + 2 * g + hf) * C::BM + r] = y;
                }
            if (hf == 0) pslot[C::BM * D + r] = lse_new;
            continue;
        }
        const int64_t lidx = ((int64_t)b * a.H + hh) * a.Nq + qrow;
        float w_prev = 0.f, w_new = inv, lse_out = lse_new;
        if (a.accum) {
            const float lse_prev = qvalid ? a.lse[lidx] : -INFINITY;
            if (lse_prev != -INFINITY) {
                if (lse_new == -INFINITY) {
                    w_prev = 1.f;
                    w_new = 0.f;
                    lse_out = lse_prev;
                } else {
                    const float M = fmaxf(lse_prev, lse_new);
                    const float e1 = __expf(lse_prev - M), e2 = __expf(lse_new - M);
                    const float rs = 1.f / (e1 + e2);
                    w_prev = e1 * rs;
                    w_new = e2 * rs * inv;
                    lse_out = M + __logf(e1 + e2);
                }
            }
        }
#pragma unroll
        for (int db = 0; db < DBLK; ++db)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int dim = 32 * db + 8 * g + 4 * hf;
                const uint32_t o = qvalid ? (uint32_t)qrow * rowb + headb + 2 * dim : kOOB;
                float y[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) y[e] = oacc[qb][db][4 * g + e] * w_new;
                if (w_prev != 0.f) {
                    const u32x2 pv = __builtin_amdgcn_raw_buffer_load_b64(ro, o, 0, 0);
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const uint32_t h = pv[e >> 1];
                        const float x = __uint_as_float((e & 1) ? (h & 0xffff0000u) : (h << 16));
                        y[e] = __builtin_fmaf(w_prev, x, y[e]);
                    }
                }
                const u32x2 w = {pack_bf16x2(y[0], y[1]), pack_bf16x2(y[2], y[3])};
                __builtin_amdgcn_raw_buffer_store_b64(w, ro, o, 0, 0);
            }
        if (a.lse && hf == 0 && qvalid) a.lse[lidx] = lse_out;
    }
    if constexpr (PATCH) copy_rest();
}

template <int D, bool PATCH, bool PARTS>
__global__ __launch_bounds__(W64<D>::THREADS) void attn_w64_kernel(Args a) {
    using C = W64<D>;
    __shared__ __attribute__((aligned(1024))) unsigned char lds[C::LDS_BYTES];
    if constexpr (!PARTS) {
        w64_segment<D, PATCH, false>(a, lds, xcd_remap(blockIdx.x, gridDim.x), 0, a.T, nullptr);
        return;
    }
    const int G2 = gridDim.x - a.G1;
    int64_t ub, ue;
    int j = 0;
    if ((int)blockIdx.x < a.G1) {
        ub = (int64_t)xcd_remap(blockIdx.x, a.G1) * a.T;
        ue = ub + a.T;
    } else {
        j = xcd_remap(blockIdx.x - a.G1, G2);
        const int64_t base = (int64_t)a.G1 * a.T, rem = a.units - base;
        ub = base + rem * j / G2;
        ue = base + rem * (j + 1) / G2;
    }
    for (int64_t u = ub; u < ue;) {
        const int pair = (int)(u / a.T);
        const int t0 = (int)(u - (int64_t)pair * a.T);
        const int nt = (int)min((int64_t)(a.T - t0), ue - u);
        float* slot = t0 == 0 && nt == a.T ? nullptr : a.part + (int64_t)(u == ub ? j : G2 + j) * C::SLOT_FLOATS;
        if (u != ub) __syncthreads();
        w64_segment<D, PATCH, true>(a, lds, pair, t0, nt, slot);
        u += nt;
    }
}

template <int D, bool PATCH>
hipError_t launch(const AttnParams& p, hipStream_t s) {
    using C = W64<D>;
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
    a.off0 = p.off0;
    a.len0 = p.len0;
    a.off1 = p.off1;
    a.len1 = p.len1;
    a.sa0 = p.len0 > 0 ? p.off0 / C::BN : 0;
    a.sn0 = p.len0 > 0 ? (p.off0 + p.len0 + C::BN - 1) / C::BN - a.sa0 : 0;
    a.sa1 = p.len1 > 0 ? p.off1 / C::BN : 0;
    a.sn1 = p.len1 > 0 ? (p.off1 + p.len1 + C::BN - 1) / C::BN - a.sa1 : 0;
    a.q_tiles = (p.Nq + C::BM - 1) / C::BM;
    a.c2 = (float)(1.4426950408889634 / sqrt((double)D));
    a.accum = p.accum;
    a.T = max(1, (p.Nk + C::BN - 1) / C::BN);
    const int64_t pairs = (int64_t)a.q_tiles * p.H * p.B;
    a.units = pairs * a.T;
    a.G1 = (int)p.whole;
    a.part = p.part;
    if (pairs == 0) return hipSuccess;
    if (p.parts <= 0) {
        hipLaunchKernelGGL((attn_w64_kernel<D, PATCH, false>), dim3((unsigned)pairs), dim3(C::THREADS), 0, s, a);
        return hipGetLastError();
    }
    if (p.whole < 0 || p.whole > pairs || p.whole % 8 != 0) return hipErrorInvalidValue;
    hipLaunchKernelGGL((attn_w64_kernel<D, PATCH, true>), dim3((unsigned)(p.whole + p.parts)), dim3(C::THREADS), 0,
                       s, a);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_attn_fixup(p, a.q_tiles, a.T, s);
}

}  // namespace

hipError_t launch_attn_w64(const AttnParams& p, hipStream_t s) {
    if (p.D != 128) return hipErrorNotSupported;
    return p.fresh_k != nullptr ? launch<128, true>(p, s) : launch<128, false>(p, s);
}

}  // namespace xdit
