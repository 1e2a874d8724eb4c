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
//     the chunk partials of the sequence-parallel merge.  Two waves per SIMD
//     let one wave's matrix work overlap another's softmax.  Shapes: 8
//     waves of 128 rows x 2 splits or 64 rows x 4 splits over 128-key tiles
//     (d <= 72, one workgroup per CU); 4 waves of 128 rows over 64-key (d
//     <= 72) or 32-key (d = 128) tiles, two workgroups per CU;
//   * K/V tiles go from memory straight into LDS (buffer loads with an LDS
//     destination: no registers, no LDS store instructions), NSTAGE tiles
//     deep, so the loads of the next tiles are in flight while tile t is
//     computed; one barrier per tile.  A row past the end of its source reads
//     as zero.  Both tiles are stored row-major as loaded, 16-byte chunks
//     XOR-swizzled by row where a row has a power-of-two chunk count, so the
//     operand reads below are free of bank conflicts;
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
//     MFMA contraction is free as long as A and B agree; the V^T operand is
//     read from the row-major V tile with ds_read_b64_tr_b16, which hands
//     each lane one head dimension of four keys, the keys chosen to match
//     P's register order;
//   * at d = 72 dims 64..71 run as one 16-row tail block on
//     v_mfma_f32_16x16x32_bf16, whose padding lanes read a constant chunk in
//     LDS: dimension 72 reads ones, so the same product also yields the row
//     sums of the bf16 weights (the exact normaliser of the bf16
//     numerator), the rest read zeros.
// Workgroups are renumbered so that all query tiles of one (batch, head) run
// on the same XCD and share its L2 for K/V (the hardware deals workgroup ids
// round-robin over the 8 XCDs).
#include "kernels.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <type_traits>

namespace xdit {
namespace {

#include "attn_common.h"


template <int D, int QB_, int KS_, int KW_>
struct Cfg {
    static constexpr int QB = QB_, KS = KS_, KW = KW_;
    static constexpr int NW = QB * KS;               // waves per workgroup
    static constexpr int THREADS = 64 * NW;
    static constexpr int BM = 32 * QB;               // query rows per workgroup
    static constexpr int BN = KS * KW;               // keys per tile
    static constexpr int DK = (D + 15) / 16 * 16;    // QK^T contraction length, padded to 16
    // PV output rows: DBLK full 32-row blocks; the rest (d = 72: dims 64..71)
    // goes to one 16-row tail block, rows TB..TB+15, on the 16x16x32
    // instruction
    static constexpr int DBLK = D / 32;
    static constexpr bool TAIL = D % 32 != 0;
    static constexpr int TB = 32 * DBLK;             // first dim of the tail block
    static constexpr int KSTEPS = DK / 16;
    static constexpr int CH = D / 8;                 // 16-byte chunks per K/V row
    static constexpr int ROWB = 16 * CH;             // bytes per row in LDS
    // LDS layout of a row: logical chunk c sits in slot c ^ swz(row).  Both
    // this swizzle and the key order krow (PERM) are chosen so that the
    // operand reads of a tile hit distinct banks (64 banks of 4 bytes; a
    // 16-byte read serves 16 lanes per cycle, an 8-byte transposing read
    // 32).  The V reads of the two half k-steps are E_ROWS rows apart, and
    // those of successive k-steps 16: swz ignores both offsets.
    //  d = 72 (9 chunks, rows 36 banks apart): no swizzle; krow puts the
    //    four keys of a transposing read four rows apart.
    //  d = 64 (8 chunks, two rows per bank cycle): rows in order, swizzle
    //    of row bits 1..3.
    //  d = 128 (16 chunks, one row per bank cycle): krow as for d = 72,
    //    swizzle of row bits 0..3.
    // Where the swizzle differs between the two half k-steps (E_SPLIT),
    // each has its own V read address.
    static constexpr bool PERM = CH != 8;
    static constexpr int E_ROWS = PERM ? 2 : 8;  // rows between the two half k-steps
    __device__ static constexpr int swz(int r) {
        if constexpr (CH == 8) return (((r >> 1) & 1) << 2) | ((r >> 2) & 3);
        else if constexpr (CH == 16) return r & 15;
        else return 0;
    }
    static constexpr bool E_SPLIT = CH == 8 || CH == 16;
    static constexpr bool SWIZZLED = CH == 8 || CH == 16;  // swz is not identically zero
    static constexpr int TILE_BYTES = BN * ROWB;     // one K or V tile
    // LDS layout: the K regions of the stages, then their V regions; a
    // region is one tile, then 16 zero bytes and the ones chunk (read by
    // the lanes of padding dims).  With K and V apart, every operand read
    // of a stage known at compile time is one per-lane base register plus
    // an immediate offset (all below 64 KiB), with no address arithmetic
    // per read.
    static constexpr int REGION = TILE_BYTES + 32;
    static constexpr int CONST_OFF = TILE_BYTES;      // within a region
    static constexpr int STAGE_BYTES = 2 * REGION;
    // Iteration t reads V of tile t and K of tile t+1 while the tiles after
    // them load: three stages at least, four where they fit (in half the
    // LDS for workgroups of 4 waves, which run two per CU).
    static constexpr int LDS_BUDGET = NW == 4 ? kLdsBytes / 2 : kLdsBytes;
    static constexpr int NSTAGE = LDS_BUDGET / STAGE_BYTES >= 4 ? 4 : 3;
    static constexpr int VBASE = NSTAGE * REGION;     // the first V region
    static constexpr int DMA_PER_TILE = TILE_BYTES / 1024;  // 64 lanes x 16 bytes per load
    static constexpr int DMA_PER_WAVE = (DMA_PER_TILE + NW - 1) / NW;
    static constexpr int DMA_MIN_PER_WAVE = 2 * (DMA_PER_TILE / NW);  // K and V, fewest by any wave
    static constexpr int Q_PIECES = BM * ROWB / 1024;  // 64-lane loads of the query tile
    static constexpr int Q_PER_WAVE = (Q_PIECES + NW - 1) / NW;
    // the query tile is staged through LDS where it fits the K and V tiles
    // of stage NSTAGE-1 (rows 0..BN-1 in its K region, the rest in its V
    // region); otherwise (128 rows of d = 128 over 32-key tiles) each wave
    // loads its rows straight into registers
    static constexpr bool Q_LDS = BM * ROWB <= 2 * TILE_BYTES;
    static constexpr int NKB = KW / 32;              // 32-key blocks of S^T per wave
    static constexpr int NKS = KW / 16;              // 16-key PV steps per wave
    static constexpr bool SUM_BY_MFMA = TAIL;        // a padding row of V^T holds ones
    // end-of-sweep exchange: one slot (m, l, O^T accumulators) per query
    // block of each partial wave
    static constexpr int XSLOT = 64 * (2 + 16 * DBLK + (TAIL ? 8 : 0));  // floats
    static constexpr int X_BYTES = 4 * QB * (KS - 1) * XSLOT;
    static constexpr int LDS_BYTES = NSTAGE * STAGE_BYTES > X_BYTES ? NSTAGE * STAGE_BYTES : X_BYTES;
    // partial (O, LSE) of one query tile: O as float4 chunks [D/4][BM],
    // then the LSE of the BM rows
    static constexpr int SLOT_FLOATS = BM * (D + 1);
    static_assert(DK - D == 0 || DK - D == 8, "K padding is at most one 16-byte chunk");
    static_assert(!TAIL || (D - TB <= 15 && D - TB > 0 && KW % 32 == 0), "tail block: dims TB..D-1, then the ones row");
    static_assert(KW % 32 == 0, "a wave takes whole 32-key blocks");
    static_assert(TILE_BYTES % 1024 == 0, "tiles are whole 64-lane loads (a query load lies in one region)");
    static_assert(DMA_PER_TILE >= NW, "every wave loads part of each tile");
    static_assert(BM * ROWB % 1024 == 0, "the query tile is whole 64-lane loads");
    static_assert(Q_LDS || DK == D, "query rows loaded into registers have no padding chunk");
    static_assert(LDS_BYTES <= LDS_BUDGET, "LDS budget");
    static_assert(NSTAGE == 4, "the main loop is unrolled over four stages");
};

// One segment: K/V tiles [tile0, tile0 + nt) of the sweep of pair `pair`;
// pslot: where its partial goes, nullptr for a whole sweep.
template <int D, int QB, int KS, int KW, bool PATCH, bool PARTS, bool PING>
__device__ __forceinline__ void attn_segment(const Args& a, unsigned char* lds, int pair, int tile0, int nt,
                                             float* pslot) {
    using C = Cfg<D, QB, KS, KW>;
    constexpr int NT = C::THREADS, BN = C::BN, NST = C::NSTAGE, NKB = C::NKB, NKS = C::NKS;

    // In a partitioned launch the thread index is made opaque to the
    // compiler, so that the lane's addresses are derived anew in each segment
    // rather than kept live across segments (which made the sweep spill).
    int tid = threadIdx.x;
    if constexpr (PARTS) asm volatile("" : "+v"(tid));
    // the wave index is uniform: held in a scalar register, so that the LDS
    // destinations of the tile loads (which go through M0) are scalar too
    const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int c = lane & 31, hf = lane >> 5;
    const int qb = wave % QB, kh = wave / QB;  // query block, key split

    const int qt = pair % a.q_tiles, bh = pair / a.q_tiles;
    uint16_t* const out_base = a.out;
    float* const lse_base = a.lse;
    // this segment's K/V tiles; t counts them from 0, tile tb + t of the
    // sequence (none past the end: with Nk = 0 the one unit has no tile)
    const int all_tiles = (a.Nk + BN - 1) / BN;
    const int tb = tile0;
    const int ntiles = max(0, min(nt, all_tiles - tile0));
    const int hh = bh % a.H, b = bh / a.H;
    const uint32_t rowb = (uint32_t)a.H * D * 2;  // bytes between consecutive rows in memory
    const uint32_t headb = (uint32_t)hh * D * 2;  // byte offset of this head in a row

    // Row 0 of this (batch, head) in each source.  Each tile gets its own
    // buffer resource (scalar work only) whose range ends at the source's
    // last row, so rows past the end read as zero.
    const int64_t headoff = (int64_t)hh * D;
    const uint16_t* kbase = a.k + (int64_t)b * a.Nk * a.H * D + headoff;
    const uint16_t* vbase = a.v + (int64_t)b * a.Nk * a.H * D + headoff;
    const int F = a.len0 + a.len1;  // fresh rows
    const uint16_t* fkbase = PATCH ? a.fk + (int64_t)b * F * a.H * D + headoff : nullptr;
    const uint16_t* fvbase = PATCH ? a.fv + (int64_t)b * F * a.H * D + headoff : nullptr;
    // rows row0 .. rows-1 (none if row0 >= rows)
    auto rows_rsrc = [&](const uint16_t* base, int row0, int rows) -> Rsrc {
        return rsrc(base + (int64_t)row0 * a.H * D, rows > row0 ? (uint32_t)(rows - row0) * rowb - headb : 0u);
    };

    // K and V regions of stage s
    auto kreg = [&](int s) -> unsigned char* { return lds + s * C::REGION; };
    auto vreg = [&](int s) -> unsigned char* { return lds + C::VBASE + s * C::REGION; };
    const uint32_t lds_u32 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) unsigned char*)lds;

    // Constant chunks of every region: 16 zero bytes, then bf16 {1, 0, 0,
    // 0, 0, 0, 0, 0} (the ones entry of the row-sum row of V^T).
    if (tid < 4 * NST) {
        const int rg = tid >> 1;  // regions: K of the stages, then V
        *(u32x4*)(lds + rg * C::REGION + C::CONST_OFF + 16 * (tid & 1)) =
            (tid & 1) ? u32x4{0x3f80u, 0, 0, 0} : u32x4{0, 0, 0, 0};
    }

    // The query tile goes to LDS stage NST-1 (its K region, then its V
    // region: byte o of the tile at qlds(o), a row boundary between them),
    // which no K/V tile uses before iteration 0, in the same load stream as
    // the tiles (issued first, so the wait for tile 0 covers it); rows past
    // Nq read as zero.
    // Routing it through LDS leaves no register with a vector-memory load
    // outstanding, so the compiler never has to wait on one in the loop.
    auto qlds = [&](int o) -> unsigned char* {
        return o < C::TILE_BYTES ? kreg(NST - 1) + o : vreg(NST - 1) + (o - C::TILE_BYTES);
    };
    const int qrow = qt * C::BM + qb * 32 + c;
    const bool qvalid = qrow < a.Nq;
    const Rsrc ro = rsrc(out_base + (int64_t)b * a.Nq * a.H * D, (uint32_t)a.Nq * rowb);
    // the wave's 32 query rows as B operands (lane: query c, dims
    // 16kk+8hf..+7), held in registers for the whole sweep
    bf16x8 qf[C::KSTEPS];
    {
        const Rsrc rq = rows_rsrc(a.q + (int64_t)b * a.Nq * a.H * D + headoff, qt * C::BM, a.Nq);
        if constexpr (C::Q_LDS) {
#pragma unroll
            for (int n = 0; n < C::Q_PER_WAVE; ++n) {
                const int ins = wave + n * C::NW;
                if (C::Q_PIECES % C::NW == 0 || ins < C::Q_PIECES) {
                    // slot p: row p / CH, logical chunk (p % CH) ^ swz(row)
                    const int p = 64 * ins + lane, r = p / C::CH;
                    dma16(rq, qlds(1024 * ins), (uint32_t)r * rowb + 16 * ((p % C::CH) ^ C::swz(r)));
                }
            }
        } else {
            // straight into registers, issued before the tile loads (the
            // prologue's wait for tile 0 covers them)
#pragma unroll
            for (int kk = 0; kk < C::KSTEPS; ++kk)
                qf[kk] = __builtin_bit_cast(bf16x8, bload(rq, (uint32_t)(qb * 32 + c) * rowb + 32 * kk + 16 * hf));
        }
    }
    // Tile loads: load n of this wave fills LDS chunks 64*ins .. 64*ins+63
    // of a tile (ins = wave + n*NW); lane l's chunk p = 64*ins + l holds
    // row p / CH, logical chunk (p % CH) ^ swizzle(row).  dma_off is its
    // byte offset from the tile's first row.
    uint32_t dma_off[C::DMA_PER_WAVE];
#pragma unroll
    for (int n = 0; n < C::DMA_PER_WAVE; ++n) {
        const int p = 64 * (wave + n * C::NW) + lane;
        const int r = p / C::CH, pc = p % C::CH;
        dma_off[n] = (uint32_t)r * rowb + 16 * (pc ^ C::swz(r));
    }

    // Issue the loads of K and V tile t into stage s.  Most tiles hold only
    // buffer (or chunk) rows and take the short path; in a patch, the few
    // tiles that hold fresh rows (ranges of tiles fixed by the host) find
    // their sources on the long one.
    auto load_tile = [&](int t, int s) {
        const int gt = tb + t, lo = gt * BN;
        unsigned char* kdst = kreg(s);
        unsigned char* vdst = vreg(s);
        auto issue = [&](Rsrc rk, Rsrc rv) {
#pragma unroll
            for (int n = 0; n < C::DMA_PER_WAVE; ++n) {
                const int ins = wave + n * C::NW;
                if (C::DMA_PER_TILE % C::NW == 0 || ins < C::DMA_PER_TILE) {
                    dma16(rk, kdst + 1024 * ins, dma_off[n]);
                    dma16(rv, vdst + 1024 * ins, dma_off[n]);
                }
            }
        };
        const bool plain = !PATCH || ((unsigned)(gt - a.sa0) >= (unsigned)a.sn0 &&
                                      (unsigned)(gt - a.sa1) >= (unsigned)a.sn1);
        if (__builtin_expect(plain, 1)) {
            issue(rows_rsrc(kbase, lo, a.Nk), rows_rsrc(vbase, lo, a.Nk));
            return;
        }
        // fresh row of buffer row j: j - off0 in range 0, len0 + j - off1 in
        // range 1
        const int hi = min(lo + BN, a.Nk);
        const bool all0 = a.off0 <= lo && hi <= a.off0 + a.len0;
        const bool all1 = a.off1 <= lo && hi <= a.off1 + a.len1;
        if (all0 || all1) {
            // every row from one fresh range; its resource ends at the
            // range's last fresh row
            const int fbase = all0 ? -a.off0 : a.len0 - a.off1;
            const int fend = all0 ? a.len0 : F;
            issue(rows_rsrc(fkbase, lo + fbase, fend), rows_rsrc(fvbase, lo + fbase, fend));
            return;
        }
        // the tile straddles a range edge (at most four per sweep): each
        // lane loads its row from its own source
        const Rsrc rk = rows_rsrc(kbase, lo, a.Nk), rv = rows_rsrc(vbase, lo, a.Nk);
        const Rsrc fk = rows_rsrc(fkbase, 0, F), fv = rows_rsrc(fvbase, 0, F);
#pragma unroll
        for (int n = 0; n < C::DMA_PER_WAVE; ++n) {
            const int ins = wave + n * C::NW;
            if (C::DMA_PER_TILE % C::NW == 0 || ins < C::DMA_PER_TILE) {
                const int r = (64 * ins + lane) / C::CH;  // row within the tile
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
        }
    };

    // LDS byte offsets (within a stage) of this lane's operand reads.
    //  K (A operand of S^T): row kw0 + 32kb + krow(c), logical chunk
    //  2kk + hf; chunks past d read the zero chunk.
    //  V (A operand of O^T, transposed read from the V tile, which follows
    //  the K tile in the stage): in each 16-lane group, lane 4j+q reads dims
    //  d0+4q..+3 of key kw0 + 16ks + krow(8e + 4hf + j), where d0 = 32db +
    //  16*(group & 1) and e = 0, 1 selects the half k-step; lane i of the
    //  group then holds dim d0 + i of the four keys, in the order of the
    //  weights P (S^T rows).
    //  V tail (A operand of the 16x16x32 tail products, one per pair of
    //  k-steps 2p, 2p+1): every 16-lane group reads dims TB..TB+15, group g
    //  the keys of k-step 2p + (g & 1) and half g >> 1, so that group g
    //  holds contraction rows 8g..8g+7 in the order of the tail weights
    //  (see pv).  Padding dims read the constant chunks (ones for dim d,
    //  zeros after it).
    const int kw0 = kh * KW;  // this wave's first key within a tile
    // LDS byte addresses within stage 0's K region (a stage adds a multiple
    // of REGION); kpad[kb]: the padded last k-step of d = 72, whose lanes of
    // the zero chunk read it in every 32-key block
    uint32_t kaddr[C::KSTEPS];
#pragma unroll
    for (int kk = 0; kk < C::KSTEPS; ++kk) {
        const int r = kw0 + krow<C::PERM>(c), lc = 2 * kk + hf;
        kaddr[kk] = lds_u32 + (lc < C::CH ? r * C::ROWB + 16 * (lc ^ C::swz(r)) : C::CONST_OFF);
    }
    constexpr bool KPAD = C::CH % 2 != 0;  // the last k-step's second half is the zero chunk
    uint32_t kpad[NKB];
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb)
        kpad[kb] = kaddr[C::KSTEPS - 1] + (KPAD && hf ? 0u : (uint32_t)(32 * kb * C::ROWB));
    const int gi = lane & 15, grp = lane >> 4;
    const int vkey0 = kw0 + krow<C::PERM>(4 * hf + (gi >> 2));
    constexpr int NE = C::E_SPLIT ? 2 : 1;
    uint32_t vaddr[C::DBLK][NE];
#pragma unroll
    for (int db = 0; db < C::DBLK; ++db) {
        const int dim = 32 * db + 16 * (grp & 1) + 4 * (gi & 3);
        for (int e = 0; e < NE; ++e) {
            const int r = vkey0 + C::E_ROWS * e;
            vaddr[db][e] = lds_u32 + C::VBASE + r * C::ROWB + 16 * ((dim >> 3) ^ C::swz(r)) + 2 * (dim & 7);
        }
    }
    // tail: vtad[p][e] = read address of k-step pair p, half step e (in
    // stage 0's V region); lanes of padding dims read the constant chunk
    // in every step
    constexpr int NPT = C::TAIL ? NKS / 2 : 0;
    uint32_t vtad[NPT > 0 ? NPT : 1][2] = {};
    if constexpr (C::TAIL) {
        static_assert(!C::E_SPLIT, "tail reads step by E_ROWS rows between half k-steps");
        const int dim = C::TB + 4 * (gi & 3);
        const int r = kw0 + krow<C::PERM>(4 * (grp >> 1) + (gi >> 2)) + 16 * (grp & 1);
        const bool cst = dim >= D;
        const uint32_t base = lds_u32 + C::VBASE +
                              (!cst ? r * C::ROWB + 16 * ((dim >> 3) ^ C::swz(r)) + 2 * (dim & 7)
                                    : (dim == D ? C::CONST_OFF + 16 : C::CONST_OFF));
#pragma unroll
        for (int pp = 0; pp < NPT; ++pp)
#pragma unroll
            for (int e = 0; e < 2; ++e)
                vtad[pp][e] = base + (cst ? 0u : (uint32_t)((32 * pp + C::E_ROWS * e) * C::ROWB));
    }

    f32x16 oacc[C::DBLK];
#pragma unroll
    for (int db = 0; db < C::DBLK; ++db) oacc[db] = f32x16{};
    // tail block: otail[h] = rows TB..TB+15 of O^T for queries 16h..16h+15
    // (16x16 layout: lane l holds query 16h + (l & 15), rows TB + 4(l >> 4)
    // + i)
    f32x4 otail[2] = {f32x4{}, f32x4{}};
    float m_ref = -INFINITY;  // reference max of the raw dot products (this wave's keys)
    float l_run = 0.f;        // this lane's share of the running sum
    float mc = 0.f;           // m_ref * c2, the shift of the exponents
    const float thr = kRescaleLog2 / a.c2;

    // S^T of tile t for this wave's KW keys x 32 queries: s[kb][i] = score of
    // key kw0 + 32kb + krow(8(i/4) + 4hf + (i%4)) of the tile against query c.
    // The stage of tile t is S when S >= 0 (a compile-time constant: its
    // offset is part of every read's immediate), else t % NST.
    auto qk = [&](int t, f32x16 (&s)[NKB], auto stage_c) {
        constexpr int S = decltype(stage_c)::value;
        constexpr uint32_t SI = S >= 0 ? (uint32_t)(S * C::REGION) : 0u;
        const uint32_t so = S >= 0 ? 0u : (uint32_t)((t % NST) * C::REGION);
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb) s[kb] = f32x16{};
#pragma unroll
        for (int kk = 0; kk < C::KSTEPS; ++kk)
#pragma unroll
            for (int kb = 0; kb < NKB; ++kb) {
                uint32_t ad;
                if (!C::SWIZZLED && 2 * kk + 1 < C::CH) {
                    // unswizzled rows: chunk 2kk + hf sits 32kk bytes past
                    // chunk hf, an immediate offset of one address
                    ad = kaddr[0] + so + (SI + 32 * kk + 32 * kb * C::ROWB);
                } else if (KPAD && kk == C::KSTEPS - 1) {
                    ad = kpad[kb] + so + SI;
                } else {
                    ad = kaddr[kk] + so + (SI + 32 * kb * C::ROWB);
                }
                const bf16x8 ka = lds_ld<bf16x8>(ad);
                s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qf[kk], s[kb], 0, 0, 0);
            }
    };
    // keys past the end of a ragged last tile get -inf
    auto mask = [&](int t, f32x16 (&s)[NKB]) {
        if ((tb + t + 1) * BN > a.Nk) {
#pragma unroll
            for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
                for (int i = 0; i < 16; ++i) {
                    const int key = (tb + t) * BN + kw0 + 32 * kb + krow<C::PERM>(8 * (i >> 2) + 4 * hf + (i & 3));
                    if (key >= a.Nk) s[kb][i] = -INFINITY;
                }
        }
    };
    // Row max of a tile (the same value in both lanes of a query).
    auto row_max = [&](const f32x16 (&s)[NKB]) -> float {
        float mx = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
            for (int i = 0; i < 16; ++i) mx = fmaxf(mx, s[kb][i]);
        return halves_max(mx);
    };
    // The reference max is raised (and the running sums rescaled) only if a
    // tile's max exceeds it by more than 2^8 in weight.
    auto update_max = [&](float mx) {
        if (__builtin_amdgcn_ballot_w64(mx > m_ref + thr) != 0) {
            const float m_new = fmaxf(m_ref, mx);
            // m_new = -inf only while a wave has seen no valid key: keep alpha finite
            const float alpha = m_new == -INFINITY ? 1.f : __builtin_amdgcn_exp2f((m_ref - m_new) * a.c2);
            m_ref = m_new;
            l_run *= alpha;
#pragma unroll
            for (int db = 0; db < C::DBLK; ++db) oacc[db] *= alpha;
            if constexpr (C::TAIL) {
                // the tail lanes hold other queries: their own factors
                const float a0 = __shfl(alpha, lane & 15), a1 = __shfl(alpha, 16 + (lane & 15));
                otail[0] *= a0;
                otail[1] *= a1;
            }
        }
        // with no valid key yet every score is -inf and any finite shift gives 0
        mc = m_ref == -INFINITY ? 0.f : m_ref * a.c2;
    };
    // bf16 weights of a tile, pb[ks] = B operand of 16-key PV step ks
    auto weights = [&](const f32x16 (&s)[NKB], bf16x8 (&pb)[NKS]) {
#pragma unroll
        for (int ks = 0; ks < NKS; ++ks) {
            const int kb = ks >> 1, i0 = 8 * (ks & 1);
            // row sums where no padding row of V^T produces them: at d = 64 as
            // float32 adds of the weights, at d = 128 of the bf16 weights, one
            // v_dot2 with ones per pair (fewer VALU instructions; measured
            // 2 % faster at d = 128, 1-3 % slower in the d = 64 patch step)
            constexpr bool SUM_F32 = !C::SUM_BY_MFMA && D <= 96, SUM_DOT = !C::SUM_BY_MFMA && D > 96;
            float p[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                p[e] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[kb][i0 + e], a.c2, -mc));
                if constexpr (SUM_F32) l_run += p[e];
            }
            typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
            typedef float f32x2_t __attribute__((ext_vector_type(2)));
            const bf16x2_t ones = {(__bf16)1.0f, (__bf16)1.0f};
            u32x4 pw;
#pragma unroll
            for (int w = 0; w < 4; ++w) {
                // one v_cvt_pk_bf16_f32 per pair (round to nearest even)
                const bf16x2_t pp = __builtin_convertvector((f32x2_t{p[2 * w], p[2 * w + 1]}), bf16x2_t);
                pw[w] = __builtin_bit_cast(uint32_t, pp);
                // the pair goes to the dot product as the converted value:
                // passed as a bit cast of an element of pw, every dot product
                // read pw's first element (a miscompile of this toolchain)
                if constexpr (SUM_DOT) l_run = __builtin_amdgcn_fdot2_f32_bf16(pp, ones, l_run, false);
            }
            pb[ks] = __builtin_bit_cast(bf16x8, pw);
        }
    };
    // V^T operands of tile t, all NKS k-steps, issued without a wait: the
    // full blocks in vr, the tail (one operand per pair of k-steps) in vt.
    // They are issued in the order pv consumes them: per k-step its full
    // blocks, then after each odd step the tail operand of the pair.
    // reads of k-step j; reads issued after those of step ks's full blocks
    // (tail = false) or after its tail operand (tail = true)
    constexpr auto vt_reads = [](int j) { return 2 * C::DBLK + (C::TAIL && (j & 1) ? 2 : 0); };
    constexpr auto vt_after = [vt_reads](int ks, bool tail) {
        int n = 0;
        for (int j = ks + 1; j < NKS; ++j) n += vt_reads(j);
        return n + (!tail && C::TAIL && (ks & 1) ? 2 : 0);
    };
    auto read_vt = [&](int t, u32x2 (&vr)[NKS][C::DBLK][2], u32x2 (&vt)[NPT > 0 ? NPT : 1][2], auto stage_c) {
        constexpr int S = decltype(stage_c)::value;
        constexpr int SI = S >= 0 ? S * C::REGION : 0;
        const uint32_t so = S >= 0 ? 0u : (uint32_t)((t % NST) * C::REGION);
        static_for<0, NKS>([&](auto ksc) {
            constexpr int ks = decltype(ksc)::value;
            static_for<0, C::DBLK>([&](auto dbc) {
                constexpr int db = decltype(dbc)::value;
                if constexpr (C::E_SPLIT) {
                    vr[ks][db][0] = tr_read<SI + 16 * ks * C::ROWB>(vaddr[db][0] + so);
                    vr[ks][db][1] = tr_read<SI + 16 * ks * C::ROWB>(vaddr[db][NE - 1] + so);
                } else {
                    // unswizzled rows: block db's dims sit 64db bytes past block 0's
                    static_assert(!C::SWIZZLED, "one address for all blocks");
                    vr[ks][db][0] = tr_read<SI + 16 * ks * C::ROWB + 64 * db>(vaddr[0][0] + so);
                    vr[ks][db][1] = tr_read<SI + (16 * ks + C::E_ROWS) * C::ROWB + 64 * db>(vaddr[0][0] + so);
                }
            });
            if constexpr (C::TAIL && (ks & 1)) {
                constexpr int pp = ks >> 1;
                vt[pp][0] = tr_read<SI>(vtad[pp][0] + so);
                vt[pp][1] = tr_read<SI>(vtad[pp][1] + so);
            }
        });
    };
    // O^T += V^T P^T over the NKS k-steps.  Tail: for each pair of k-steps,
    // permlane16_swap of the two steps' weights gives the 16x16x32 B
    // operands of queries 0..15 ({x.r0, y.r0, x.r2, y.r2}: rows of 16 lanes)
    // and 16..31 ({x.r1, y.r1, x.r3, y.r3}); group g then holds the keys of
    // step 2p + (g & 1), half g >> 1, as the tail V^T operand does.
    // The V^T reads of read_vt are still in flight: each k-step waits only
    // for its own operands, so the first products start while the later
    // operands arrive.
    auto pv = [&](u32x2 (&vr)[NKS][C::DBLK][2], u32x2 (&vt)[NPT > 0 ? NPT : 1][2], const bf16x8 (&pb)[NKS]) {
        static_for<0, NKS>([&](auto ksc) {
            constexpr int ks = decltype(ksc)::value;
            if constexpr (C::DBLK == 2)
                lds_wait_upto<vt_after(ks, false)>(vr[ks][0][0], vr[ks][0][1], vr[ks][1][0], vr[ks][1][1]);
            else if constexpr (C::DBLK == 4)
                lds_wait_upto<vt_after(ks, false)>(vr[ks][0][0], vr[ks][0][1], vr[ks][1][0], vr[ks][1][1],
                                                   vr[ks][2][0], vr[ks][2][1], vr[ks][3][0], vr[ks][3][1]);
            else
                static_assert(C::DBLK == 2 || C::DBLK == 4, "full blocks of V^T");
#pragma unroll
            for (int db = 0; db < C::DBLK; ++db) {
                const u32x4 v4 = {vr[ks][db][0][0], vr[ks][db][0][1], vr[ks][db][1][0], vr[ks][db][1][1]};
                oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, v4), pb[ks], oacc[db],
                                                                   0, 0, 0);
            }
            if constexpr (C::TAIL && (ks & 1)) {
                constexpr int pp = ks >> 1;
                lds_wait_upto<vt_after(ks, true)>(vt[pp][0], vt[pp][1]);
                const u32x4 x = __builtin_bit_cast(u32x4, pb[ks - 1]), y = __builtin_bit_cast(u32x4, pb[ks]);
                u32x4 b0, b1;
#pragma unroll
                for (int w = 0; w < 4; ++w) {
                    const auto r = __builtin_amdgcn_permlane16_swap(x[w], y[w], false, false);
                    b0[w] = r[0];
                    b1[w] = r[1];
                }
                const u32x4 v4 = {vt[pp][0][0], vt[pp][0][1], vt[pp][1][0], vt[pp][1][1]};
                const bf16x8 va = __builtin_bit_cast(bf16x8, v4);
                otail[0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, __builtin_bit_cast(bf16x8, b0), otail[0],
                                                                   0, 0, 0);
                otail[1] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, __builtin_bit_cast(bf16x8, b1), otail[1],
                                                                   0, 0, 0);
            }
        });
    };

    // Wait until at most the loads of the N most recently issued tiles are in
    // flight.  A wave issues the same number of loads for every tile (twice
    // as many for a tile that straddles the slice edge, which only makes the
    // wait stricter): 2*DMA_PER_WAVE if it takes one of the leftover 1 KiB
    // pieces of a tile, 2*(DMA_PER_TILE / NW) otherwise.
    const bool extra_piece = wave + (C::DMA_PER_WAVE - 1) * C::NW < C::DMA_PER_TILE;
    auto wait_tiles = [&](auto n_c) {
        constexpr int N = decltype(n_c)::value;
        if (C::DMA_PER_TILE % C::NW != 0 && extra_piece) wait_vmem<N * 2 * C::DMA_PER_WAVE>();
        else wait_vmem<N * C::DMA_MIN_PER_WAVE>();
    };

    // Software pipeline: iteration t computes the weights and PV of tile t
    // and, on the matrix cores meanwhile, the scores of tile t+1; the row
    // max of tile t+1 then runs under the PV products.  Scores of tile t
    // live in sc, those of tile t+1 go to sn.  NEXT: there is a tile t+1;
    // MASK: it may be the ragged last tile.  Tile t sits in stage S when S
    // >= 0, else in stage t % NST.
    auto iteration = [&](int t, f32x16 (&sc)[NKB], f32x16 (&sn)[NKB], auto next_c, auto mask_c, auto stage_c) {
        constexpr bool NEXT = decltype(next_c)::value, MASK = decltype(mask_c)::value;
        constexpr int S = decltype(stage_c)::value;
        using SNext = std::integral_constant<int, S >= 0 ? (S + 1) % NST : -1>;
        if constexpr (NEXT) {
            // Tile t+1 must have landed (tile t+2 may still be in flight with
            // four stages) before anyone reads it: each wave waits for its own
            // loads, then all meet.  A bare s_barrier: the full __syncthreads
            // fence would also drain the younger loads.  Everybody is then
            // done with tile t-1 (its V was read in the previous iteration,
            // its K in the one before), so its stage takes tile t+NST-1.
            if (NST >= 4 && t + 2 < ntiles) wait_tiles(std::integral_constant<int, 1>{});
            else wait_vmem<0>();
            asm volatile("" ::: "memory");  // no LDS access moves across the barrier
            __builtin_amdgcn_s_barrier();
            asm volatile("" ::: "memory");
            if (t + NST - 1 < ntiles) load_tile(t + NST - 1, S >= 0 ? (S + NST - 1) % NST : (t + NST - 1) % NST);
        }
        // the K operand reads of tile t+1 go first: LDS reads complete in
        // issue order, so V^T reads issued before them would hold the QK
        // products back behind the whole V^T batch
        bf16x8 pb[NKS];
        weights(sc, pb);
        if constexpr (NEXT) qk(t + 1, sn, SNext{});
        u32x2 vr[NKS][C::DBLK][2], vt[NPT > 0 ? NPT : 1][2];
        read_vt(t, vr, vt, stage_c);
        float mx = 0.f;
        if constexpr (NEXT) {
            if constexpr (MASK) mask(t + 1, sn);
            mx = row_max(sn);
        }
        pv(vr, vt, pb);
        if constexpr (NEXT) update_max(mx);
    };
    using T_ = std::true_type;
    using F_ = std::false_type;
    using RS = std::integral_constant<int, -1>;  // stage known at run time
    using S0 = std::integral_constant<int, 0>;
    using S1 = std::integral_constant<int, 1>;
    using S2 = std::integral_constant<int, 2>;
    using S3 = std::integral_constant<int, 3>;

    // Prologue: the first NST-1 tiles load whether or not this sweep has
    // that many (a tile past the sequence end reads zeros, one past this
    // split's range lands in a stage nobody reads).
    f32x16 sA[NKB], sB[NKB];
#pragma unroll
    for (int t = 0; t < NST - 1; ++t) load_tile(t, t);
    // tile 0 (and the query tile, loaded before it) must have landed, NST-2
    // younger tiles may be in flight, and the constant chunks must be
    // written before anyone reads them
    wait_tiles(std::integral_constant<int, NST - 2>{});
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    if constexpr (C::Q_LDS) {
#pragma unroll
        for (int kk = 0; kk < C::KSTEPS; ++kk) {
            const int r = qb * 32 + c, lc = 2 * kk + hf;  // chunks past d read the zero chunk
            qf[kk] = *(const bf16x8*)(lc < C::CH ? qlds(16 * (r * C::CH + (lc ^ C::swz(r)))) : kreg(NST - 1) + C::CONST_OFF);
        }
    } else {
        // the compiler waits here for the register loads (all older than
        // the tile loads), so that no path into the loop leaves them
        // outstanding
#pragma unroll
        for (int kk = 0; kk < C::KSTEPS; ++kk) asm volatile("" : "+v"(qf[kk]));
    }
    if constexpr (PING) {
        // Ping-pong of the two halves of the workgroup (waves w and w + NW/2
        // share a SIMD): each iteration is a matrix phase (scores of tile
        // t+1, PV of tile t) and a softmax phase (row max, reference max,
        // weights of tile t+1), each opened by a workgroup barrier.  The
        // second half passes one barrier more at the start and the first
        // half one more at the end, so that between two barriers one half
        // runs its matrix phase while the other runs its softmax phase, and
        // the matrix cores and the vector ALUs of a SIMD work at once.
        // Every wave passes 2 * ntiles + 3 barriers.
        //   Loads: a wave issues its share of tile t+NST-1 at the start of
        // its matrix phase t (the stage of tile t-1, whose last reads, the
        // V^T of tile t-1 in both halves' matrix phase t-1, lie behind the
        // barrier).  Tile t+1 is first read by the first half's matrix
        // phase t; every wave has its share of it landed before the barrier
        // that opens that phase, which is where the first half opens its
        // matrix phase t and the second half its softmax phase t.
        const bool lead = wave < C::NW / 2;
        // nothing moves across the barrier: LDS accesses (memory clobber)
        // nor arithmetic (scheduling barrier)
        auto bar = [&]() {
            asm volatile("" ::: "memory");
            __builtin_amdgcn_sched_barrier(0);
            __builtin_amdgcn_s_barrier();
            __builtin_amdgcn_sched_barrier(0);
            asm volatile("" ::: "memory");
        };
        // the weights are computed in the softmax phase, not in the next
        // matrix phase
        auto pin_pb = [&](bf16x8 (&w)[NKS]) {
#pragma unroll
            for (int ks = 0; ks < NKS; ++ks) asm volatile("" : "+v"(w[ks]));
        };
        // this wave's loads of tile n have landed; tile n+1's may be in
        // flight when this segment has it
        auto landed = [&](int n) {
            if (n + 1 < ntiles) wait_tiles(std::integral_constant<int, 1>{});
            else wait_vmem<0>();
        };
        bf16x8 pb[NKS];
        if (!lead) bar();
        if (ntiles > 0) qk(0, sA, S0{});
        if (!lead) landed(1);
        bar();
        if (ntiles > 0) {
            mask(0, sA);
            update_max(row_max(sA));
            weights(sA, pb);
            pin_pb(pb);
        }
        auto iter_pp = [&](int t, auto next_c, auto mask_c, auto stage_c) {
            constexpr bool NEXT = decltype(next_c)::value, MASK = decltype(mask_c)::value;
            constexpr int S = decltype(stage_c)::value;
            using SNext = std::integral_constant<int, S >= 0 ? (S + 1) % NST : -1>;
            if (lead) landed(t + 1);
            bar();
            if (t + NST - 1 < ntiles) load_tile(t + NST - 1, S >= 0 ? (S + NST - 1) % NST : (t + NST - 1) % NST);
            if constexpr (NEXT) qk(t + 1, sA, SNext{});
            u32x2 vr[NKS][C::DBLK][2], vt[NPT > 0 ? NPT : 1][2];
            read_vt(t, vr, vt, stage_c);
            pv(vr, vt, pb);
            if (!lead) landed(t + 2);
            bar();
            if constexpr (NEXT) {
                if constexpr (MASK) mask(t + 1, sA);
                update_max(row_max(sA));
                weights(sA, pb);
                pin_pb(pb);
            }
        };
        int t = 0;
        for (; t + 5 < ntiles; t += 4) {
            iter_pp(t, T_{}, F_{}, S0{});
            iter_pp(t + 1, T_{}, F_{}, S1{});
            iter_pp(t + 2, T_{}, F_{}, S2{});
            iter_pp(t + 3, T_{}, F_{}, S3{});
        }
        for (; t + 2 < ntiles; ++t) iter_pp(t, T_{}, F_{}, RS{});
        if (t + 2 == ntiles) {
            iter_pp(t, T_{}, T_{}, RS{});
            iter_pp(t + 1, F_{}, F_{}, RS{});
        } else if (t + 1 == ntiles) {
            iter_pp(t, F_{}, F_{}, RS{});
        }
        if (lead) bar();
    } else {
        if (ntiles > 0) {
            qk(0, sA, S0{});
            mask(0, sA);
            update_max(row_max(sA));
        }
        // runs of four iterations (stages 0..3) whose next tile is not the
        // last one, then at most one such pair, then the last one to three
        // tiles
        int t = 0;
        for (; t + 5 < ntiles; t += 4) {
            iteration(t, sA, sB, T_{}, F_{}, S0{});
            iteration(t + 1, sB, sA, T_{}, F_{}, S1{});
            iteration(t + 2, sA, sB, T_{}, F_{}, S2{});
            iteration(t + 3, sB, sA, T_{}, F_{}, S3{});
        }
        if (t + 3 < ntiles) {
            iteration(t, sA, sB, T_{}, F_{}, RS{});
            iteration(t + 1, sB, sA, T_{}, F_{}, RS{});
            t += 2;
        }
        if (t + 3 == ntiles) {
            iteration(t, sA, sB, T_{}, F_{}, RS{});
            iteration(t + 1, sB, sA, T_{}, T_{}, RS{});
            iteration(t + 2, sA, sB, F_{}, F_{}, RS{});
        } else if (t + 2 == ntiles) {
            iteration(t, sA, sB, T_{}, T_{}, RS{});
            iteration(t + 1, sB, sA, F_{}, F_{}, RS{});
        } else if (t + 1 == ntiles) {
            iteration(t, sA, sB, F_{}, F_{}, RS{});
        }
    }
    // Every wave is done with the stages, and no tile load is in flight
    // (with fewer than NST-1 tiles the prologue's spare loads are still
    // outstanding here; the key-split exchange below reuses their LDS).
    wait_vmem<0>();
    __syncthreads();

    // Patch mode: this workgroup's share of the fresh rows goes into the
    // buffer (the workgroups of a (batch, head) split the rows).  Nothing in
    // this kernel reads the fresh ranges of the buffer: tiles take those rows
    // from the fresh tensors.  The copy runs after the sweep, so its memory
    // operations hold up none of the sweep's waits, and the first batch's
    // loads are in flight during the key-split merge and the output.
    constexpr int CU = 4;  // 16-byte chunks per lane and batch
    // the share of this segment's units among the head's q_tiles * T
    const int64_t hu = (int64_t)a.q_tiles * a.T, u0 = (int64_t)qt * a.T + tile0;
    const int cr0 = (int)((int64_t)F * u0 / hu);
    const int cn = ((int)((int64_t)F * (u0 + nt) / hu) - cr0) * C::CH;  // chunks of the share
    uint32_t cd[CU];
    u32x4 ck[CU], cv[CU];
    // loads of batch e0 .. e0 + CU*NT - 1; chunks past the share use the
    // out-of-range offset (reads give zero, writes are dropped)
    auto copy_load = [&](int e0) {
        const Rsrc fk = rows_rsrc(fkbase, 0, F), fv = rows_rsrc(fvbase, 0, F);
#pragma unroll
        for (int u = 0; u < CU; ++u) {
            const int e = e0 + tid + u * NT;
            const int fr = cr0 + e / C::CH, cc = 16 * (e % C::CH);
            const int j = fr < a.len0 ? a.off0 + fr : a.off1 + fr - a.len0;  // buffer row
            const uint32_t cs = e < cn ? (uint32_t)fr * rowb + cc : kOOB;
            cd[u] = e < cn ? (uint32_t)j * rowb + cc : kOOB;
            ck[u] = bload(fk, cs);
            cv[u] = bload(fv, cs);
        }
    };
    // stores of the loaded batch, then the remaining batches
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

    // Merge the KS partial sweeps of each query block.  Slots are lane-major
    // so the exchange is free of bank conflicts.
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
            if constexpr (C::TAIL)
#pragma unroll
                for (int i = 0; i < 8; ++i) slot[(2 + 16 * C::DBLK + i) * 64 + lane] = otail[i >> 2][i & 3];
        }
        // LDS only: a bare barrier, which leaves the copy loads in flight
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
        if (kh == 0) {
            float M = m_ref;
#pragma unroll
            for (int k2 = 1; k2 < KS; ++k2) M = fmaxf(M, xs[((k2 - 1) * QB + qb) * C::XSLOT + lane]);
            const float mM = M == -INFINITY ? 0.f : M;
            const float a0 = m_ref == -INFINITY ? 0.f : __builtin_amdgcn_exp2f((m_ref - mM) * a.c2);
            l_run *= a0;
#pragma unroll
            for (int db = 0; db < C::DBLK; ++db) oacc[db] *= a0;
            // tail lanes hold queries 16h + (lane & 15): factors of those queries
            const int tq = lane & 15;
            if constexpr (C::TAIL) {
                otail[0] *= __shfl(a0, tq);
                otail[1] *= __shfl(a0, 16 + tq);
            }
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
                if constexpr (C::TAIL) {
                    const float t0 = __shfl(ak, tq), t1 = __shfl(ak, 16 + tq);
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        otail[0][i] = __builtin_fmaf(t0, slot[(2 + 16 * C::DBLK + i) * 64 + lane], otail[0][i]);
                        otail[1][i] = __builtin_fmaf(t1, slot[(2 + 16 * C::DBLK + 4 + i) * 64 + lane], otail[1][i]);
                    }
                }
            }
            m_ref = M;
        }
    }
    if (kh != 0) {
        if constexpr (PATCH) copy_rest();
        return;
    }

    float l_tot;
    if constexpr (C::SUM_BY_MFMA) {
        // row D of O^T: tail row lr, held (16x16 layout) by lane 16(lr/4) + q%16
        // of otail[q/16], register lr%4
        constexpr int lr = D - C::TB;
        const float s0 = __shfl(otail[0][lr % 4], 16 * (lr / 4) + (c & 15));
        const float s1 = __shfl(otail[1][lr % 4], 16 * (lr / 4) + (c & 15));
        l_tot = c < 16 ? s0 : s1;
    } else {
        l_tot = halves_sum(l_run);
    }
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
    constexpr float kLn2 = 0.69314718055994531f;
    const float lse_new = l_tot > 0.f ? (m_ref * a.c2 + __log2f(l_tot)) * kLn2 : -INFINITY;
    if (pslot != nullptr) {
        // partial sweep: normalised O and the LSE in float32, for the
        // fix-up; chunk k4 (dims 4k4..4k4+3) of tile row r at float4 k4*BM + r
        f32x4* po = (f32x4*)pslot;
        const int r = qb * 32 + c;
#pragma unroll
        for (int db = 0; db < C::DBLK; ++db)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const f32x4 y = {oacc[db][4 * g] * inv, oacc[db][4 * g + 1] * inv, oacc[db][4 * g + 2] * inv,
                                 oacc[db][4 * g + 3] * inv};
                po[(8 * db + 2 * g + hf) * C::BM + r] = y;
            }
        if constexpr (C::TAIL) {
            const int k4 = C::TB / 4 + (lane >> 4);
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                const float iv = __shfl(inv, 16 * h + (lane & 15));
                if (4 * k4 < D) po[k4 * C::BM + qb * 32 + 16 * h + (lane & 15)] = otail[h] * iv;
            }
        }
        if (hf == 0) pslot[C::BM * D + r] = lse_new;
        if constexpr (PATCH) copy_rest();
        return;
    }
    const int64_t lidx = ((int64_t)b * a.H + hh) * a.Nq + qrow;
    // Merge into a running (out, lse) (the ring's accumulation over chunks,
    // Section 4.1.1): weights e^{lse_prev - L} and e^{lse_new - L} with
    // L = ln(e^{lse_prev} + e^{lse_new}); a running lse of -inf marks an empty
    // state whose output is ignored.
    float w_prev = 0.f, w_new = inv, lse_out = lse_new;
    if (a.accum) {
        const float lse_prev = qvalid ? lse_base[lidx] : -INFINITY;
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
    for (int db = 0; db < C::DBLK; ++db)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            // dims 32db + 8g + 4hf .. +3
            const int dim = 32 * db + 8 * g + 4 * hf;
            if (dim < D) {
                const f32x16& o16 = oacc[db];
                const uint32_t o = qvalid ? (uint32_t)qrow * rowb + headb + 2 * dim : kOOB;
                float y[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) y[e] = o16[4 * g + e] * w_new;
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
        }
    if constexpr (C::TAIL) {
        // tail dims TB + 4(lane >> 4) .. +3 of queries 16h + (lane & 15),
        // with those queries' weights
        const int dim = C::TB + 4 * (lane >> 4);
        const float wn[2] = {__shfl(w_new, lane & 15), __shfl(w_new, 16 + (lane & 15))};
        const float wp[2] = {__shfl(w_prev, lane & 15), __shfl(w_prev, 16 + (lane & 15))};
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int qr = qt * C::BM + qb * 32 + 16 * h + (lane & 15);
            if (dim < D) {
                const uint32_t o = qr < a.Nq ? (uint32_t)qr * rowb + headb + 2 * dim : kOOB;
                float y[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) y[e] = otail[h][e] * wn[h];
                if (wp[h] != 0.f) {
                    const u32x2 pv = __builtin_amdgcn_raw_buffer_load_b64(ro, o, 0, 0);
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const uint32_t hw = pv[e >> 1];
                        const float x = __uint_as_float((e & 1) ? (hw & 0xffff0000u) : (hw << 16));
                        y[e] = __builtin_fmaf(wp[h], x, y[e]);
                    }
                }
                const u32x2 w = {pack_bf16x2(y[0], y[1]), pack_bf16x2(y[2], y[3])};
                __builtin_amdgcn_raw_buffer_store_b64(w, ro, o, 0, 0);
            }
        }
    }
    if (lse_base && hf == 0 && qvalid) lse_base[lidx] = lse_out;
    if constexpr (PATCH) copy_rest();
}

// One workgroup per query tile (PARTS = false: workgroup L sweeps pair L
// whole), or a partitioned launch (PARTS = true, see Args).  Workgroup ids
// are remapped per group (whole sweeps, cut ranges) so that neighbouring
// pairs share an XCD; G1 is a multiple of 8, so both groups start on XCD 0.
// Workgroups of 4 waves (one per SIMD) are built to run two per CU: each
// wave is then held to 256 registers, so that every SIMD interleaves two
// waves of independent workgroups, which no barrier keeps in step.
template <int D, int QB, int KS, int KW, bool PATCH, bool PARTS, bool PING>
__global__ __launch_bounds__(64 * QB * KS, QB * KS == 4 ? 2 : 1) void attn_bf16_kernel(Args a) {
    using C = Cfg<D, QB, KS, KW>;
    __shared__ __attribute__((aligned(1024))) unsigned char lds[C::LDS_BYTES];
    if constexpr (!PARTS) {
        attn_segment<D, QB, KS, KW, PATCH, false, PING>(a, lds, xcd_remap(blockIdx.x, gridDim.x), 0, a.T, nullptr);
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
        if (u != ub) __syncthreads();  // the previous segment is done with LDS
        attn_segment<D, QB, KS, KW, PATCH, true, PING>(a, lds, pair, t0, nt, slot);
        u += nt;
    }
}

// Fix-up of a launch whose partition cut some sweeps: the partials of every
// range that meets a cut sweep are merged (the LSE merge of Section 4.1.1
// over the key parts) into out and lse, by workgroups (x, rb) for tile rows
// 16rb..16rb+15.  When each of the cut query tiles is cut into s_al even
// parts (s_al > 0), workgroup x handles the x-th of them, whose parts are
// ranges x*s_al .. x*s_al + s_al - 1.  Otherwise workgroup x handles the
// boundary between ranges x and x + 1 when it falls inside a sweep and is
// the first boundary inside it, and finds the ranges that meet that sweep.
// A sweep with a single non-empty part was swept whole by that part, which
// wrote out and lse itself (no slot): such a sweep is left alone.
// With accum, the merged chunk result is merged in turn into the running
// (out, lse), as the sweep kernel's epilogue does for whole sweeps.
// Thread t: row 16rb + t % 16, dim chunks t / 16, t / 16 + 16, ...
struct FixArgs {
    uint16_t* out;
    float* lse;
    const float* part;
    int B, H, Nq, q_tiles, T, G2, s_al;
    int accum;
    int64_t base, rem;  // the cut ranges split units [base, base + rem)
};

constexpr int kMaxParts = kMaxSweepParts;
constexpr int kFixRows = 16;  // tile rows per fix-up workgroup

template <int D, int BM>
__global__ __launch_bounds__(256) void fixup_kernel(FixArgs a) {
    // thread 0 finds the sweep and its parts (64-bit index arithmetic) and
    // hands them to the others through LDS
    __shared__ int64_t sh_pair;
    __shared__ int64_t sh_slot[kMaxParts];
    __shared__ int sh_n;
    if (threadIdx.x == 0 && a.s_al > 0) {
        // part i of cut sweep x is range x*s + i: units T*i/s .. T*(i+1)/s of
        // the sweep (empty when that is)
        const int x = blockIdx.x, sa = a.s_al;
        int n = 0;
        for (int i = 0; i < sa && n < kMaxParts; ++i)
            if (a.T * (i + 1) / sa > a.T * i / sa) sh_slot[n++] = (int64_t)x * sa + i;
        sh_pair = a.base / a.T + x;
        sh_n = n;
    } else if (threadIdx.x == 0) {
        const int g = blockIdx.x + 1;
        const int64_t G = a.G2, T = a.T;
        auto ub = [&](int64_t w) { return a.base + a.rem * w / G; };
        const int64_t bg = ub(g), P = bg / T, pu0 = P * T, pu1 = pu0 + T;
        int n = 0;
        // only a boundary inside a sweep, and the first one inside it
        if (bg != pu0 && ub(g - 1) <= pu0) {
            // the parts: ranges w >= g - 1 that are non-empty and meet
            // [pu0, pu1); slot w if the part is w's first segment, G + w
            // otherwise (the host bounds their number by kMaxParts)
            int64_t w = g - 1, b0 = ub(w);
            while (w < G && n < kMaxParts) {
                const int64_t b1 = ub(w + 1);
                if (b0 >= pu1) break;
                if (b1 > b0) sh_slot[n++] = b0 >= pu0 ? w : G + w;
                ++w;
                b0 = b1;
            }
        }
        sh_pair = P;
        sh_n = n;
    }
    __syncthreads();
    const int n = sh_n;
    // no cut sweep here, or one part that swept it whole (and wrote it)
    if (n <= 1) return;
    const int64_t P = sh_pair;
    const int qt = (int)(P % a.q_tiles), bh = (int)(P / a.q_tiles), hh = bh % a.H, b = bh / a.H;
    const int r = kFixRows * blockIdx.y + (int)threadIdx.x % kFixRows, dg = (int)threadIdx.x / kFixRows;
    const int qrow = qt * BM + r;
    const int64_t lidx = ((int64_t)b * a.H + hh) * a.Nq + qrow;
    // the running LSE of the row is read by every thread of the row before
    // the row's first thread overwrites it
    float lse_prev = -INFINITY;
    if (a.accum) {
        if (qrow < a.Nq) lse_prev = a.lse[lidx];
        __syncthreads();
    }
    if (qrow >= a.Nq) return;
    constexpr int SLOT = BM * (D + 1);
    // every load of the thread issued up front (parts beyond n predicated
    // off): the merge is latency-bound otherwise
    const float* base[kMaxParts];
    float lw[kMaxParts];
#pragma unroll
    for (int i = 0; i < kMaxParts; ++i) {
        base[i] = a.part + (i < n ? sh_slot[i] : 0) * SLOT;
        lw[i] = i < n ? base[i][BM * D + r] : -INFINITY;
    }
    typedef float f32x4_t __attribute__((ext_vector_type(4)));
    typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
    constexpr int C4 = D / 4, NG = 256 / kFixRows, PER = (C4 + NG - 1) / NG;
    f32x4_t x[kMaxParts][PER];
#pragma unroll
    for (int i = 0; i < kMaxParts; ++i)
#pragma unroll
        for (int kk = 0; kk < PER; ++kk)
            if (i < n && dg + NG * kk < C4) x[i][kk] = ((const f32x4_t*)base[i])[(dg + NG * kk) * BM + r];
    float M = -INFINITY;
#pragma unroll
    for (int i = 0; i < kMaxParts; ++i) M = fmaxf(M, lw[i]);
    float sum = 0.f;
#pragma unroll
    for (int i = 0; i < kMaxParts; ++i) sum += lw[i] == -INFINITY ? 0.f : __expf(lw[i] - M);
    const float L = M == -INFINITY ? -INFINITY : M + __logf(sum);
    // O = sum_i exp(lse_i - L) O_i over this thread's dim chunks
    f32x4_t acc[PER];
#pragma unroll
    for (int kk = 0; kk < PER; ++kk) acc[kk] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < kMaxParts; ++i) {
        const float w = lw[i] == -INFINITY ? 0.f : __expf(lw[i] - L);
#pragma unroll
        for (int kk = 0; kk < PER; ++kk)
            if (i < n && dg + NG * kk < C4) acc[kk] += w * x[i][kk];
    }
    uint16_t* orow = a.out + (((int64_t)b * a.Nq + qrow) * a.H + hh) * D;
    // merge into the running state: weights e^{lse_prev - L2}, e^{L - L2}
    // with L2 = ln(e^{lse_prev} + e^{L}); an empty running state (-inf)
    // is ignored, an empty chunk (L = -inf) leaves the state as it is
    float w_prev = 0.f, w_new = 1.f, L_out = L;
    if (a.accum && lse_prev != -INFINITY) {
        if (L == -INFINITY) {
            w_prev = 1.f;
            w_new = 0.f;
            L_out = lse_prev;
        } else {
            const float M2 = fmaxf(lse_prev, L);
            const float e1 = __expf(lse_prev - M2), e2 = __expf(L - M2);
            const float rs = 1.f / (e1 + e2);
            w_prev = e1 * rs;
            w_new = e2 * rs;
            L_out = M2 + __logf(e1 + e2);
        }
    }
#pragma unroll
    for (int kk = 0; kk < PER; ++kk)
        if (dg + NG * kk < C4) {
            u32x2_t* dst = (u32x2_t*)orow + dg + NG * kk;
            f32x4_t y = acc[kk] * w_new;
            if (w_prev != 0.f) {
                const u32x2_t pv = *dst;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const uint32_t h = pv[e >> 1];
                    const float x0 = __uint_as_float((e & 1) ? (h & 0xffff0000u) : (h << 16));
                    y[e] = __builtin_fmaf(w_prev, x0, y[e]);
                }
            }
            *dst = u32x2_t{pack_bf16x2(y[0], y[1]), pack_bf16x2(y[2], y[3])};
        }
    if (a.lse && dg == 0) a.lse[lidx] = L_out;
}

// The fix-up launch after a partitioned sweep of 128-row query tiles, each
// sweep T K/V tiles long: merges the partials of the cut sweeps.
template <int D>
hipError_t launch_fixup(const AttnParams& p, int q_tiles, int T, hipStream_t s) {
    constexpr int BM = kPartSlotRows;
    if (p.parts < 2) return hipSuccess;
    const int64_t pairs = (int64_t)q_tiles * p.H * p.B;
    FixArgs f;
    f.out = (uint16_t*)p.out;
    f.lse = p.lse;
    f.part = p.part;
    f.B = p.B;
    f.H = p.H;
    f.Nq = p.Nq;
    f.q_tiles = q_tiles;
    f.T = T;
    f.G2 = (int)p.parts;
    f.base = p.whole * T;
    f.rem = pairs * T - f.base;
    const int64_t cut = pairs - p.whole;  // query tiles in the cut ranges
    f.s_al = p.parts % cut == 0 ? (int)(p.parts / cut) : 0;
    f.accum = p.accum;
    // one part per cut query tile, or sweeps of one tile: every part swept
    // its query tile whole and wrote it, nothing to merge
    if (f.s_al == 1 || T == 1) return hipSuccess;
    const int64_t gx = f.s_al > 0 ? cut : p.parts - 1;
    hipLaunchKernelGGL((fixup_kernel<D, BM>), dim3((unsigned)gx, BM / kFixRows), dim3(256), 0, s, f);
    return hipGetLastError();
}

template <int D, int QB, int KS, int KW, bool PATCH, bool PING = false>
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
    a.off0 = p.off0;
    a.len0 = p.len0;
    a.off1 = p.off1;
    a.len1 = p.len1;
    // tiles holding rows of each fresh range
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
    const bool parts = p.parts > 0;
    if (!parts) {
        hipLaunchKernelGGL((attn_bf16_kernel<D, QB, KS, KW, PATCH, false, PING>), dim3((unsigned)pairs), dim3(C::THREADS),
                           0, s, a);
        return hipGetLastError();
    }
    if constexpr (C::BM != kPartSlotRows) {
        return hipErrorInvalidValue;  // only the 128-row shape runs partitioned launches (slot layout)
    } else {
        if (p.whole < 0 || p.whole > pairs || p.whole % 8 != 0) return hipErrorInvalidValue;
        hipLaunchKernelGGL((attn_bf16_kernel<D, QB, KS, KW, PATCH, true, PING>), dim3((unsigned)(p.whole + p.parts)),
                           dim3(C::THREADS), 0, s, a);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        return launch_fixup<D>(p, a.q_tiles, a.T, s);
    }
}

// Shapes of 8-wave workgroup.  "Wide": 128 query rows as 4 query blocks x 2
// key splits (a 128-key tile at d <= 72, 64 keys at d = 128 for the register
// and LDS budget).  "Narrow" (d <= 72): 64 query rows x 4 key splits of a
// 128-key tile, for query counts whose 128-row tiles would leave many of the
// 256 CUs idle.
constexpr int kCUs = 256;

double fill(int64_t blocks) {
    const int64_t rounds = (blocks + kCUs - 1) / kCUs;
    return rounds ? (double)blocks / (double)(rounds * kCUs) : 1.0;
}

// XDIT_ATTN_TILE forces one shape (tuning and tests): "wide", "narrow"
// (8 waves; both fall back to the default at d = 128) or "quad" (4 waves,
// 128 rows, 64-key tiles; d <= 72, unpartitioned launches); anything else,
// or unset, picks by the fill estimate.
int forced_shape() {
    const char* e = getenv("XDIT_ATTN_TILE");
    if (e == nullptr) return 0;
    if (strcmp(e, "wide") == 0) return 1;
    if (strcmp(e, "narrow") == 0) return 2;
    if (strcmp(e, "quad") == 0) return 3;
    return 0;
}

// XDIT_ATTN_KERNEL selects the decomposition: "w64" (64 query rows per
// wave, attn_w64.hip, head dim 128), "o2" (workgroups of 4 waves, two per
// CU), "w32" (the 8-wave workgroups of this file, and at d <= 72 the 4-wave
// 128-row shape where the grid has more query tiles than CUs) or "pp" (the
// 8-wave shapes with the two halves in ping-pong).  Unset: o2 at d = 128
// (the Flux chunk step measured 221 vs 228-236 us), w32 at d <= 72 (o2's
// 64-row, 64-key shape measured 10-18 % slower there).
static int attn_kernel_choice(int D) {
    const char* e = getenv("XDIT_ATTN_KERNEL");
    if (e != nullptr && strcmp(e, "w64") == 0) return 64;
    if (e != nullptr && strcmp(e, "o2") == 0) return 2;
    if (e != nullptr && strcmp(e, "w32") == 0) return 32;
    if (e != nullptr && strcmp(e, "pp") == 0) return 3;
    return D > 96 ? 2 : 32;
}

template <int D, bool PATCH>
hipError_t dispatch(const AttnParams& p, hipStream_t s) {
    if (attn_kernel_choice(D) == 2) {
        // 128 rows x 32-key tiles at d = 128; 64 rows (2 blocks x 2 key
        // splits of a 64-key tile) at d <= 72, whose partitioned launches
        // keep the 8-wave shape (128-row slots)
        if constexpr (D > 96) return launch<D, 4, 1, 32, PATCH>(p, s);
        else if (p.parts <= 0) return launch<D, 2, 2, 32, PATCH>(p, s);
    }
    if (attn_kernel_choice(D) == 3) {
        if constexpr (D > 96) return launch<D, 4, 2, 32, PATCH, true>(p, s);
        else return launch<D, 4, 2, 64, PATCH, true>(p, s);
    }
    if constexpr (D > 96) {
        return launch<D, 4, 2, 32, PATCH>(p, s);
    } else {
        const int forced = forced_shape();
        const int64_t bh = (int64_t)p.B * p.H;
        const int64_t wide = (p.Nq + 127) / 128 * bh, narrow = (p.Nq + 63) / 64 * bh;
        // More 128-row query tiles than CUs: workgroups of 4 waves (128
        // rows, one key split, 64-key tiles), two per CU, whose waves
        // interleave on each SIMD as at d = 128 (cog chunk step 630 -> 543
        // us, patch step 317 -> 308 us).  With no more tiles than CUs most
        // CUs would get one such workgroup, one wave per SIMD (sd3 patch
        // step 44 -> 52 us), and the 8-wave shapes stay.
        if (p.parts <= 0 && (forced == 3 || (forced == 0 && wide > kCUs))) return launch<D, 4, 1, 64, PATCH>(p, s);
        // split keys fill the GPU by themselves: 128-row query tiles
        if (forced == 1 || p.parts > 0) return launch<D, 4, 2, 64, PATCH>(p, s);
        if (forced == 2) return launch<D, 2, 4, 32, PATCH>(p, s);
        const double qfill_w = (double)p.Nq / ((p.Nq + 127) / 128 * 128.0);
        const double qfill_n = (double)p.Nq / ((p.Nq + 63) / 64 * 64.0);
        if (fill(narrow) * qfill_n > 1.1 * fill(wide) * qfill_w) return launch<D, 2, 4, 32, PATCH>(p, s);
        return launch<D, 4, 2, 64, PATCH>(p, s);
    }
}

}  // namespace

hipError_t launch_attn_fixup(const AttnParams& p, int q_tiles, int T, hipStream_t s) {
    switch (p.D) {
        case 64: return launch_fixup<64>(p, q_tiles, T, s);
        case 72: return launch_fixup<72>(p, q_tiles, T, s);
        case 128: return launch_fixup<128>(p, q_tiles, T, s);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_attn_bf16(const AttnParams& p, hipStream_t s) {
    const bool patch = p.fresh_k != nullptr;
    if (p.D == 128 && attn_kernel_choice(p.D) == 64) return launch_attn_w64(p, s);
    switch (p.D) {
        case 64: return patch ? dispatch<64, true>(p, s) : dispatch<64, false>(p, s);
        case 72: return patch ? dispatch<72, true>(p, s) : dispatch<72, false>(p, s);
        case 128: return patch ? dispatch<128, true>(p, s) : dispatch<128, false>(p, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace xdit
