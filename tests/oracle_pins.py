"""Pins for the fp64 oracle: checks against facts fixed by the paper and by
mathematics, never against the oracle's own formulas.

Each pin takes an oracle handle and raises AssertionError when it fails, so
the same pins can be run against deliberately broken builds of the oracle
(see test_oracle_pins.py) to show that they catch plausible mistakes.

The paper prints no numeric worked example for attention, the patch step or
the merge, so the pins are: brute force on tiny inputs (direct softmax with no
max shift, math.fsum sums), closed forms, a library routine (scipy's
logsumexp/softmax) on special cases, and the invariants the paper states:
SP over sharded sequence gives the serial result (Section 4.1.1), the fresh
area grows patch by patch within a step (Section 4.1.2), attention is full
rather than causal (Section 4.1.2).
"""
from __future__ import annotations

import itertools
import math

import numpy as np
import scipy.special

from paper_2411_01738_amd.inputs import random_io

TOL = 1e-12


def _close(a, b, tol=TOL, what=""):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    assert a.shape == b.shape, f"{what}: shape {a.shape} vs {b.shape}"
    if a.size == 0:
        return
    both_inf = np.isinf(a) & np.isinf(b) & (np.sign(a) == np.sign(b))
    err = np.where(both_inf, 0.0, np.abs(a - b))
    assert np.all(np.isfinite(err)), f"{what}: non-finite mismatch"
    assert err.max() <= tol, f"{what}: max err {err.max():.3e} > {tol:.1e}"


def brute_attention(q, k, v):
    """Direct definition in pure Python: weights exp(s_j) with no max shift,
    sums with math.fsum.  Tiny inputs only."""
    B, Nq, H, d = q.shape
    Nk = k.shape[1]
    scale = 1.0 / math.sqrt(d)
    out = np.zeros((B, Nq, H, d))
    lse = np.zeros((B, H, Nq))
    for b in range(B):
        for h in range(H):
            for i in range(Nq):
                s = [scale * math.fsum(float(q[b, i, h, c]) * float(k[b, j, h, c])
                                       for c in range(d)) for j in range(Nk)]
                w = [math.exp(x) for x in s]
                z = math.fsum(w)
                lse[b, h, i] = math.log(z)
                for c in range(d):
                    out[b, i, h, c] = math.fsum(w[j] * float(v[b, j, h, c])
                                                for j in range(Nk)) / z
    return out, lse


def _rand(shape, seed, scale=1.0):
    return random_io(shape, "f32", seed, scale)


# --------------------------------------------------------------------------
# attention
# --------------------------------------------------------------------------
def pin_brute_force(orc):
    for (B, Nq, Nk, H, d), seed in [((1, 5, 7, 2, 8), 11), ((2, 3, 4, 3, 4), 12),
                                    ((1, 1, 16, 1, 6), 13), ((1, 16, 1, 2, 8), 14)]:
        q = _rand((B, Nq, H, d), seed)
        k = _rand((B, Nk, H, d), seed + 100)
        v = _rand((B, Nk, H, d), seed + 200)
        o, l = orc.attention(q, k, v)
        ob, lb = brute_attention(q, k, v)
        _close(o, ob, 1e-12, "brute out")
        _close(l, lb, 1e-12, "brute lse")


def pin_scipy_softmax(orc):
    """A moderate case against scipy's logsumexp and softmax."""
    B, Nq, Nk, H, d = 1, 12, 64, 2, 16
    q, k, v = _rand((B, Nq, H, d), 21), _rand((B, Nk, H, d), 22), _rand((B, Nk, H, d), 23)
    o, l = orc.attention(q, k, v)
    q64, k64, v64 = (x.astype(np.float64) for x in (q, k, v))
    for h in range(H):
        s = q64[0, :, h, :] @ k64[0, :, h, :].T / math.sqrt(d)
        _close(l[0, h], scipy.special.logsumexp(s, axis=1), 1e-12, "scipy lse")
        _close(o[0, :, h, :], scipy.special.softmax(s, axis=1) @ v64[0, :, h, :], 1e-12,
               "scipy out")


def pin_closed_forms(orc):
    B, Nq, Nk, H, d = 2, 6, 9, 2, 8
    v = _rand((B, Nk, H, d), 31)
    # C1: zero queries -> uniform weights: o = mean of V, lse = ln Nk
    q0 = np.zeros((B, Nq, H, d), np.float32)
    k = _rand((B, Nk, H, d), 32)
    o, l = orc.attention(q0, k, v)
    _close(o, np.broadcast_to(v.astype(np.float64).mean(axis=1, keepdims=True), o.shape),
           1e-13, "C1 out")
    _close(l, np.full(l.shape, math.log(Nk)), 1e-13, "C1 lse")
    # C2: all keys equal -> o = mean V, lse = s q.k + ln Nk
    q = _rand((B, Nq, H, d), 33)
    krow = _rand((B, 1, H, d), 34)
    kk = np.ascontiguousarray(np.broadcast_to(krow, (B, Nk, H, d)))
    o, l = orc.attention(q, kk, v)
    _close(o, np.broadcast_to(v.astype(np.float64).mean(axis=1, keepdims=True), o.shape),
           1e-12, "C2 out")
    dots = np.einsum("bihc,bhc->bhi", q.astype(np.float64), krow[:, 0].astype(np.float64))
    _close(l, dots / math.sqrt(d) + math.log(Nk), 1e-12, "C2 lse")
    # C3: a single key -> o = v0, lse = s q.k0
    o, l = orc.attention(q, k[:, :1].copy(), v[:, :1].copy())
    _close(o, np.broadcast_to(v[:, :1].astype(np.float64), o.shape), 0.0, "C3 out")
    dots = np.einsum("bihc,bhc->bhi", q.astype(np.float64), k[:, 0].astype(np.float64))
    _close(l, dots / math.sqrt(d), 1e-12, "C3 lse")
    # C4: constant value rows -> o = that constant (softmax rows sum to one)
    vc = np.ascontiguousarray(np.broadcast_to(_rand((B, 1, H, d), 35), (B, Nk, H, d)))
    o, _ = orc.attention(q, k, vc)
    _close(o, np.broadcast_to(vc[:, :1].astype(np.float64), o.shape), 1e-13, "C4 out")
    # two keys: weights are the logistic function of the score difference
    k2, v2 = k[:, :2].copy(), v[:, :2].copy()
    o, l = orc.attention(q, k2, v2)
    s = np.einsum("bihc,bjhc->bhij", q.astype(np.float64), k2.astype(np.float64)) / math.sqrt(d)
    w0 = scipy.special.expit(s[..., 0] - s[..., 1])          # [B,H,Nq]
    exp_o = (w0[..., None] * v2[:, 0][:, :, None, :].astype(np.float64)
             + (1 - w0)[..., None] * v2[:, 1][:, :, None, :].astype(np.float64))
    _close(o, exp_o.transpose(0, 2, 1, 3), 1e-13, "two-key out")
    _close(l, np.logaddexp(s[..., 0], s[..., 1]), 1e-13, "two-key lse")


def pin_empty_and_rows(orc):
    B, Nq, H, d = 1, 4, 2, 8
    q = _rand((B, Nq, H, d), 41)
    e = np.zeros((B, 0, H, d), np.float32)
    o, l = orc.attention(q, e, e)
    assert np.all(o == 0) and np.all(np.isneginf(l)), "empty K/V"
    k, v = _rand((B, 10, H, d), 42), _rand((B, 10, H, d), 43)
    o, l = orc.attention(q, k, v)
    rows = [3, 0, 2]
    os_, ls_ = orc.attention(q, k, v, rows=rows)
    _close(os_, o[:, rows], 0.0, "row subset out")
    _close(ls_, l[:, :, rows], 0.0, "row subset lse")


def pin_permutation_and_independence(orc):
    """C5: permuting K/V rows jointly leaves (o, lse) unchanged; permuting Q
    rows permutes the results; (b, h) slices do not interact; no causal mask
    (a query attends to later keys as well)."""
    B, Nq, Nk, H, d = 2, 7, 11, 3, 8
    q, k, v = _rand((B, Nq, H, d), 51), _rand((B, Nk, H, d), 52), _rand((B, Nk, H, d), 53)
    o, l = orc.attention(q, k, v)
    perm = np.random.Generator(np.random.PCG64(5)).permutation(Nk)
    o2, l2 = orc.attention(q, k[:, perm].copy(), v[:, perm].copy())
    _close(o2, o, 1e-13, "kv perm out")
    _close(l2, l, 1e-13, "kv perm lse")
    qp = np.random.Generator(np.random.PCG64(6)).permutation(Nq)
    o3, l3 = orc.attention(q[:, qp].copy(), k, v)
    _close(o3, o[:, qp], 0.0, "q perm out")
    _close(l3, l[:, :, qp], 0.0, "q perm lse")
    k4, v4 = k.copy(), v.copy()
    k4[1, :, 2] = 7.0
    v4[0, :, 1] = -3.0
    o4, l4 = orc.attention(q, k4, v4)
    keep = np.ones((B, H), bool)
    keep[1, 2] = keep[0, 1] = False
    for b, h in itertools.product(range(B), range(H)):
        if keep[b, h]:
            _close(o4[b, :, h], o[b, :, h], 0.0, "independent out")
            _close(l4[b, h], l[b, h], 0.0, "independent lse")
    # full attention: the first query sees the last key
    k5 = k.copy()
    k5[:, -1] = q[:, 0]
    o5, _ = orc.attention(q, k5, v)
    assert np.abs(o5[:, 0] - o[:, 0]).max() > 1e-6, "first query ignores the last key"


# --------------------------------------------------------------------------
# chunk + merge (Section 4.1.1: the sharded computation equals the serial one)
# --------------------------------------------------------------------------
def _chunked(orc, q, k, v, bounds):
    outs, lses = [], []
    for s, e in bounds:
        o, l = orc.attention(q, k[:, s:e].copy(), v[:, s:e].copy())
        outs.append(o.astype(np.float32))  # partials cross the merge boundary as float
        lses.append(l.astype(np.float32))
    return outs, lses


def pin_merge_equals_full(orc):
    B, Nq, Nk, H, d = 2, 9, 40, 2, 8
    q, k, v = _rand((B, Nq, H, d), 61), _rand((B, Nk, H, d), 62), _rand((B, Nk, H, d), 63)
    o_full, l_full = orc.attention(q, k, v)
    splits = {
        1: [(0, 40)],
        2: [(0, 20), (20, 40)],
        4: [(0, 10), (10, 20), (20, 30), (30, 40)],
        8: [(5 * r, 5 * r + 5) for r in range(8)],
        "uneven": [(0, 3), (3, 17), (17, 18), (18, 40)],
        "empty": [(0, 12), (12, 12), (12, 40)],
    }
    for name, bounds in splits.items():
        # float32 rounding of the partials is the only error source
        outs, lses = _chunked(orc, q, k, v, bounds)
        o, l = orc.merge(outs, lses)
        _close(o, o_full, 2e-6, f"merge {name} out")
        _close(l, l_full, 2e-6, f"merge {name} lse")
    # exact fp64 check of the identity through the oracle's own partials:
    # merge of the two halves' (o, lse) computed on dyadic-friendly inputs
    qz = np.zeros((1, 2, 1, 4), np.float32)
    kz = np.zeros((1, 4, 1, 4), np.float32)
    vz = np.arange(16, dtype=np.float32).reshape(1, 4, 1, 4)
    outs, lses = _chunked(orc, qz, kz, vz, [(0, 1), (1, 4)])
    o, l = orc.merge(outs, lses)
    _close(o[0, :, 0], np.broadcast_to(np.array([6.0, 7.0, 8.0, 9.0]), (2, 4)), 1e-6,
           "merge mean")
    _close(l, np.full((1, 1, 2), math.log(4.0)), 1e-6, "merge lse ln4")


def pin_merge_algebra(orc):
    """C6: n = 1 is the identity; the merge is symmetric in its partials and a
    tree of merges equals the flat merge; all-empty gives zeros and -inf."""
    B, Nq, H, d = 1, 5, 2, 8
    outs = [_rand((B, Nq, H, d), 70 + r) for r in range(4)]
    lses = [_rand((B, H, Nq), 80 + r, 2.0) for r in range(4)]
    o1, l1 = orc.merge(outs[:1], lses[:1])
    _close(o1, outs[0], 0.0, "merge n=1 out")
    _close(l1, lses[0], 0.0, "merge n=1 lse")
    o, l = orc.merge(outs, lses)
    for perm in [(3, 1, 0, 2), (1, 0, 3, 2)]:
        op, lp = orc.merge([outs[i] for i in perm], [lses[i] for i in perm])
        _close(op, o, 1e-14, "merge symmetric out")
        _close(lp, l, 1e-14, "merge symmetric lse")
    oa, la = orc.merge(outs[:2], lses[:2])
    ob, lb = orc.merge(outs[2:], lses[2:])
    ot, lt = orc.merge([oa.astype(np.float32), ob.astype(np.float32)],
                       [la.astype(np.float32), lb.astype(np.float32)])
    _close(ot, o, 1e-6, "tree merge out")
    _close(lt, l, 1e-6, "tree merge lse")
    # explicit two-partial weights: sigmoid of the LSE difference
    o2, l2 = orc.merge(outs[:2], lses[:2])
    w0 = scipy.special.expit(lses[0].astype(np.float64) - lses[1].astype(np.float64))
    exp = (w0.transpose(0, 2, 1)[..., None] * outs[0]
           + (1 - w0).transpose(0, 2, 1)[..., None] * outs[1])
    _close(o2, exp, 1e-13, "two-partial weights")
    _close(l2, np.logaddexp(lses[0].astype(np.float64), lses[1].astype(np.float64)), 1e-13,
           "two-partial lse")
    ninf = [np.full((B, H, Nq), -np.inf, np.float32)] * 2
    oe, le = orc.merge(outs[:2], ninf)
    assert np.all(oe == 0) and np.all(np.isneginf(le)), "all-empty merge"
    le2 = [lses[0], ninf[0]]
    oe2, le2o = orc.merge(outs[:2], le2)
    _close(oe2, outs[0], 0.0, "empty partial ignored")
    _close(le2o, lses[0], 0.0, "empty partial lse")


# --------------------------------------------------------------------------
# patch step (Section 4.1.2 PipeFusion; Section 4.1.4 buffer contents)
# --------------------------------------------------------------------------
def pin_patch_update_exact(orc):
    B, N, H, d = 2, 20, 2, 4
    kv = np.stack([_rand((B, N, H, d), 91), _rand((B, N, H, d), 92)])
    before = kv.copy()
    fk, fv = _rand((B, 6, H, d), 93), _rand((B, 6, H, d), 94)
    orc.patch_update(kv, 5, fk, fv)
    assert np.array_equal(kv[0, :, 5:11], fk) and np.array_equal(kv[1, :, 5:11], fv), \
        "slice not replaced by the fresh rows"
    assert np.array_equal(kv[:, :, :5], before[:, :, :5]), "rows before the slice changed"
    assert np.array_equal(kv[:, :, 11:], before[:, :, 11:]), "rows after the slice changed"
    e = np.zeros((B, 0, H, d), np.float32)
    orc.patch_update(kv, N, e, e)  # empty patch at the end is allowed
    try:
        orc.patch_update(kv, N - 2, fk, fv)
    except ValueError:
        pass
    else:
        raise AssertionError("out-of-range slice accepted")


def pin_patch_semantics(orc):
    """All-fresh buffer: a patch step equals plain attention.  Sequential patch
    steps over a stale buffer: after patch p, slices <= p are fresh and > p
    stale; after the last one the buffer is all fresh and the last patch's
    output equals fresh full attention of its rows."""
    B, N, H, d, M = 1, 24, 2, 8, 4
    L = N // M
    q = _rand((B, N, H, d), 101)
    kf, vf = _rand((B, N, H, d), 102), _rand((B, N, H, d), 103)
    ks = kf + np.float32(0.05) * _rand((B, N, H, d), 104)
    vs = vf + np.float32(0.05) * _rand((B, N, H, d), 105)
    o_full, l_full = orc.attention(q, kf, vf)
    # I3: all-fresh buffer
    for p in range(M):
        kv = np.stack([kf, vf]).copy()
        o, l = orc.patch(q[:, p * L:(p + 1) * L].copy(), kv, p * L,
                         kf[:, p * L:(p + 1) * L].copy(), vf[:, p * L:(p + 1) * L].copy())
        _close(o, o_full[:, p * L:(p + 1) * L], 0.0, "all-fresh patch out")
        _close(l, l_full[:, :, p * L:(p + 1) * L], 0.0, "all-fresh patch lse")
    # sequential steps on one stale buffer
    kv = np.stack([ks, vs]).copy()
    for p in range(M):
        sl = slice(p * L, (p + 1) * L)
        o, l = orc.patch(q[:, sl].copy(), kv, p * L, kf[:, sl].copy(), vf[:, sl].copy())
        fresh_upto = (p + 1) * L
        assert np.array_equal(kv[0, :, :fresh_upto], kf[:, :fresh_upto]), "fresh area K"
        assert np.array_equal(kv[1, :, :fresh_upto], vf[:, :fresh_upto]), "fresh area V"
        assert np.array_equal(kv[0, :, fresh_upto:], ks[:, fresh_upto:]), "stale area K"
        assert np.array_equal(kv[1, :, fresh_upto:], vs[:, fresh_upto:]), "stale area V"
        # the same step written as attention over an explicitly assembled buffer
        kx = np.concatenate([kf[:, :fresh_upto], ks[:, fresh_upto:]], axis=1)
        vx = np.concatenate([vf[:, :fresh_upto], vs[:, fresh_upto:]], axis=1)
        oe, le = orc.attention(q[:, sl].copy(), kx, vx)
        _close(o, oe, 0.0, "sequential patch out")
        _close(l, le, 0.0, "sequential patch lse")
        if p < M - 1:
            assert np.abs(o - o_full[:, sl]).max() > 1e-6, "stale rows had no effect"
    _close(o, o_full[:, (M - 1) * L:], 0.0, "last patch equals fresh attention")


# --------------------------------------------------------------------------
# patch step over several fresh ranges with its own queries (Section 4.1.2:
# in-context text travels with patch 0; Section 4.1.4: hybrid parallelism
# stores SP-gathered K/V and attends with the local query shard)
# --------------------------------------------------------------------------
def pin_patch_ranges_brute_force(orc):
    """Two fresh ranges on a tiny buffer against the direct definition: the
    buffer rows are rebuilt by hand, row by row, and attention is the brute
    force softmax (no max shift, math.fsum)."""
    B, N, H, d = 1, 12, 2, 4
    kv = np.stack([_rand((B, N, H, d), 111), _rand((B, N, H, d), 112)])
    before = kv.copy()
    ranges = [(1, 3), (9, 3)]
    fk, fv = _rand((B, 6, H, d), 113), _rand((B, 6, H, d), 114)
    q = _rand((B, 5, H, d), 115)
    o, l = orc.patch_ranges(q, kv, ranges, fk, fv)
    k_ref, v_ref = before[0].copy(), before[1].copy()
    src = 0
    for off, ln in ranges:
        for i in range(ln):
            k_ref[:, off + i] = fk[:, src]
            v_ref[:, off + i] = fv[:, src]
            src += 1
    assert np.array_equal(kv[0], k_ref) and np.array_equal(kv[1], v_ref), "buffer after the update"
    ob, lb = brute_attention(q, k_ref, v_ref)
    _close(o, ob, TOL, "two-range patch out")
    _close(l, lb, TOL, "two-range patch lse")


def pin_patch_ranges_in_context(orc):
    """Patch 0 carrying the text (image rows [0, n_img), text rows after them):
    one step refreshes patch 0 and the text rows; the image patches after it
    stay stale; text and patch-0 queries both see the fresh rows.  With M = 1
    (one patch = the whole image) the step is plain attention over the fresh
    sequence."""
    B, H, d, n_img, n_txt, M = 1, 2, 8, 12, 4, 3
    N, L = n_img + n_txt, n_img // M
    q = _rand((B, N, H, d), 121)
    kf, vf = _rand((B, N, H, d), 122), _rand((B, N, H, d), 123)
    ks = kf + np.float32(0.05) * _rand((B, N, H, d), 124)
    vs = vf + np.float32(0.05) * _rand((B, N, H, d), 125)
    rows = np.r_[0:L, n_img:N]
    kv = np.stack([ks, vs]).copy()
    o, l = orc.patch_ranges(q[:, rows].copy(), kv, [(0, L), (n_img, n_txt)],
                            kf[:, rows].copy(), vf[:, rows].copy())
    fresh = np.zeros(N, bool)
    fresh[rows] = True
    assert np.array_equal(kv[0][:, fresh], kf[:, fresh]) and np.array_equal(kv[0][:, ~fresh], ks[:, ~fresh])
    assert np.array_equal(kv[1][:, fresh], vf[:, fresh]) and np.array_equal(kv[1][:, ~fresh], vs[:, ~fresh])
    ob, lb = brute_attention(q[:, rows], np.where(fresh[None, :, None, None], kf, ks),
                             np.where(fresh[None, :, None, None], vf, vs))
    _close(o, ob, TOL, "in-context patch 0 out")
    _close(l, lb, TOL, "in-context patch 0 lse")
    kv = np.stack([ks, vs]).copy()
    o1, l1 = orc.patch_ranges(q, kv, [(0, n_img), (n_img, n_txt)], kf, vf)
    of, lf = brute_attention(q, kf, vf)
    _close(o1, of, TOL, "single patch with text = fresh attention")
    _close(l1, lf, TOL, "single patch with text lse")


def pin_patch_ranges_sp_shards(orc):
    """Hybrid SP x PipeFusion at one GPU's share: every SP rank stores the
    same gathered fresh K/V and attends with its own shard of the patch's
    queries; the ranks' buffers end identical and their outputs, put side by
    side, are the unsharded step's (here against brute force)."""
    B, N, H, d, sp = 1, 16, 2, 4, 4
    kv0 = np.stack([_rand((B, N, H, d), 131), _rand((B, N, H, d), 132)])
    off, ln = 4, 8
    fk, fv = _rand((B, ln, H, d), 133), _rand((B, ln, H, d), 134)
    q = _rand((B, ln, H, d), 135)
    outs, lses, bufs = [], [], []
    for r in range(sp):
        kv = kv0.copy()
        sh = slice(r * ln // sp, (r + 1) * ln // sp)
        o, l = orc.patch_ranges(q[:, sh].copy(), kv, [(off, ln)], fk, fv)
        outs.append(o)
        lses.append(l)
        bufs.append(kv)
    for kv in bufs[1:]:
        assert np.array_equal(kv, bufs[0]), "SP ranks' buffers differ"
    k_ref, v_ref = kv0[0].copy(), kv0[1].copy()
    k_ref[:, off:off + ln], v_ref[:, off:off + ln] = fk, fv
    ob, lb = brute_attention(q, k_ref, v_ref)
    _close(np.concatenate(outs, axis=1), ob, TOL, "sharded queries out")
    _close(np.concatenate(lses, axis=2), lb, TOL, "sharded queries lse")


def _stage_inputs(B, L, N, H, d, C, seed):
    x = random_io((B, L, C), "bf16", seed)
    w = [random_io((C, H * d), "bf16", seed + s, 1.0 / math.sqrt(C)) for s in (1, 2, 3)]
    wo = random_io((H * d, C), "bf16", seed + 4, 1.0 / math.sqrt(H * d))
    kv = np.ascontiguousarray(random_io((2, B, N, H, d), "bf16", seed + 5))
    return x, w, wo, kv


def pin_stage_brute_force(orc):
    """Stage micro-step on tiny inputs by its definition in pure Python: the
    projections as math.fsum dot products, the patch step with the direct
    softmax (no max shift), the output projection; also the buffer's fresh
    rows (the projections rounded to float) and the returned q/k/v."""
    B, L, N, H, d, C, off = 2, 3, 7, 2, 3, 5, 2
    x, (wq, wk, wv), wo, kv = _stage_inputs(B, L, N, H, d, C, 70)
    kv0 = kv.copy()
    res = orc.stage_step(x, wq, wk, wv, wo, kv, off)

    def proj(w):
        out = np.zeros((B, L, H, d))
        for b, i, h, c in itertools.product(range(B), range(L), range(H), range(d)):
            out[b, i, h, c] = math.fsum(float(x[b, i, e]) * float(w[e, h * d + c]) for e in range(C))
        return out
    q, k, v = proj(wq), proj(wk), proj(wv)
    kb, vb = kv0[0].astype(np.float64), kv0[1].astype(np.float64)
    kb[:, off:off + L], vb[:, off:off + L] = k, v
    o, _ = brute_attention(q, kb, vb)
    y = np.zeros((B, L, C))
    for b, i, e in itertools.product(range(B), range(L), range(C)):
        y[b, i, e] = math.fsum(o[b, i, n // d, n % d] * float(wo[n, e]) for n in range(H * d))
    _close(res["q"], q, TOL, "stage q")
    _close(res["k"], k, TOL, "stage k")
    _close(res["v"], v, TOL, "stage v")
    _close(res["o"], o, TOL, "stage attention output")
    _close(res["y"], y, TOL, "stage y")
    exp_kv = kv0.copy()
    exp_kv[0][:, off:off + L], exp_kv[1][:, off:off + L] = k.astype(np.float32), v.astype(np.float32)
    assert np.array_equal(kv, exp_kv), "stage buffer update"


def pin_stage_identity_is_patch_step(orc):
    """With C = H*d and every projection the identity, the stage micro-step
    is the patch step with q = k = v = x (the pinned patch oracle), and the
    output projection returns its output unchanged."""
    B, L, N, H, d, off = 2, 4, 9, 2, 3, 3
    C = H * d
    x = random_io((B, L, C), "bf16", 80)
    kv = np.ascontiguousarray(random_io((2, B, N, H, d), "bf16", 81))
    kv_p = kv.copy()
    eye = np.eye(C, dtype=np.float32)
    res = orc.stage_step(x, eye, eye, eye, eye, kv, off)
    xq = x.reshape(B, L, H, d)
    o, _ = orc.patch(xq, kv_p, off, xq, xq)
    _close(res["o"], o, TOL, "identity stage vs patch step")
    _close(res["y"], o.reshape(B, L, C), TOL, "identity output projection")
    assert np.array_equal(kv, kv_p), "identity stage buffer vs patch step buffer"


def pin_stage_head_permutation(orc):
    """Multi-head attention does not depend on the order of its heads:
    permuting the heads of Wq, Wk, Wv (columns), of Wo (rows) and of the
    buffer leaves y unchanged, and permutes the attention output's heads."""
    B, L, N, H, d, C, off = 1, 3, 8, 3, 2, 4, 4
    x, (wq, wk, wv), wo, kv = _stage_inputs(B, L, N, H, d, C, 90)
    perm = [2, 0, 1]
    cols = np.concatenate([np.arange(h * d, (h + 1) * d) for h in perm])
    res = orc.stage_step(x, wq, wk, wv, wo, kv.copy(), off)
    kvp = np.ascontiguousarray(kv[:, :, :, perm, :])
    resp = orc.stage_step(x, wq[:, cols], wk[:, cols], wv[:, cols], wo[cols, :], kvp, off)
    _close(resp["y"], res["y"], 1e-12, "head-permuted stage y")
    _close(resp["o"], res["o"][:, :, perm, :], 1e-12, "head-permuted stage o")


PINS = [pin_brute_force, pin_scipy_softmax, pin_closed_forms, pin_empty_and_rows,
        pin_permutation_and_independence, pin_merge_equals_full, pin_merge_algebra,
        pin_patch_update_exact, pin_patch_semantics, pin_patch_ranges_brute_force,
        pin_patch_ranges_in_context, pin_patch_ranges_sp_shards, pin_stage_brute_force,
        pin_stage_identity_is_patch_step, pin_stage_head_permutation]
