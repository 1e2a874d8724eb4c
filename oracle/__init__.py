"""fp64 CPU oracle for the xDiT attention hot path (arXiv 2411.01738).

TEST INFRASTRUCTURE ONLY.  Only the tests, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this package.  It shares no code
with the HIP library and never imports it.

The arithmetic lives in ``xdit_oracle.c`` (plain double-precision loops, one
query row at a time); this module compiles it with gcc, loads it with ctypes
and marshals numpy arrays.  Definitions (see the C file for the formulas):

* ``attention``   full multi-head self-attention with scale 1/sqrt(d)
                  (Section 2; Section 4.1.2 notes DiT attention is not causal)
* ``merge``       log-sum-exp recombination of chunk partials (Section 4.1.1,
                  SP-Ring as parallel FlashAttention; sharded result equals the
                  serial one)
* ``patch``       PipeFusion patch step over a fresh/stale K/V buffer
                  (Section 4.1.2; Section 4.1.4 for the buffer contents)
* ``stage_step``  one stage micro-step at one attention layer: QKV
                  projections, the patch step, the output projection
                  (Section 4.1.2; Section 3 on the projections)

Layouts: activations [B, N, H, d]; K/V buffer [2, B, N, H, d]; LSE [B, H, Nq].
Inputs are float32 arrays holding the exact values given to the GPU (bf16
values are exact in float32); results are float64.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SOURCE = os.path.join(HERE, "xdit_oracle.c")
LIBRARY = os.path.join(HERE, "liboracle.so")

_f32p = np.ctypeslib.ndpointer(dtype=np.float32, flags="C_CONTIGUOUS")
_f64p = np.ctypeslib.ndpointer(dtype=np.float64, flags="C_CONTIGUOUS")
_i64 = ctypes.c_int64


def build(source: str = SOURCE, output: str = LIBRARY) -> str:
    """Compile the C oracle with gcc (-O2, OpenMP, no fast-math)."""
    cmd = ["gcc", "-O2", "-fopenmp", "-fno-fast-math", "-shared", "-fPIC", "-o", output,
           source, "-lm"]
    subprocess.run(cmd, check=True)
    return output


class Oracle:
    """ctypes handle on one build of the C oracle."""

    def __init__(self, path: str = LIBRARY):
        if not os.path.exists(path):
            build(output=path)
        self.path = path
        lib = ctypes.CDLL(path)
        lib.xo_attention.restype = ctypes.c_int
        lib.xo_attention.argtypes = [_f32p, _f32p, _f32p, _i64, _i64, _i64, _i64, _i64,
                                     ctypes.c_void_p, _i64, _f64p, ctypes.c_void_p]
        lib.xo_merge.restype = ctypes.c_int
        lib.xo_merge.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int32, _i64, _i64,
                                 _i64, _i64, _f64p, ctypes.c_void_p]
        lib.xo_patch_update.restype = ctypes.c_int
        lib.xo_patch_update.argtypes = [_f32p, _i64, _i64, _f32p, _f32p, _i64, _i64, _i64, _i64]
        lib.xo_patch.restype = ctypes.c_int
        lib.xo_patch.argtypes = [_f32p, _f32p, _i64, _i64, _f32p, _f32p, _i64, _i64, _i64, _i64,
                                 ctypes.c_void_p, _i64, _f64p, ctypes.c_void_p]
        lib.xo_patch_ranges.restype = ctypes.c_int
        lib.xo_patch_ranges.argtypes = [_f32p, _i64, _f32p, ctypes.c_int32, ctypes.c_void_p,
                                        ctypes.c_void_p, _f32p, _f32p, _i64, _i64, _i64, _i64,
                                        ctypes.c_void_p, _i64, _f64p, ctypes.c_void_p]
        lib.xo_stage.restype = ctypes.c_int
        lib.xo_stage.argtypes = [_f32p, _f32p, _f32p, _f32p, _f32p, _f32p, _i64, _i64, _i64, _i64,
                                 _i64, _i64, _i64, ctypes.c_void_p, _i64, ctypes.c_void_p,
                                 ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                 ctypes.c_void_p]
        lib.xo_num_threads.restype = ctypes.c_int
        lib.xo_set_num_threads.argtypes = [ctypes.c_int]
        self.lib = lib

    # -- helpers -----------------------------------------------------------
    @staticmethod
    def _f32(x) -> np.ndarray:
        x = np.asarray(x)
        if x.dtype != np.float32:
            raise TypeError("oracle inputs are float32 arrays holding the uploaded values")
        return np.ascontiguousarray(x)

    def num_threads(self) -> int:
        return int(self.lib.xo_num_threads())

    def set_num_threads(self, n: int) -> None:
        self.lib.xo_set_num_threads(int(n))

    # -- definitions -------------------------------------------------------
    def attention(self, q, k, v, rows=None):
        """softmax(Q K^T / sqrt(d)) V for q [B,Nq,H,d], k/v [B,Nk,H,d].

        rows: optional sequence of query indices to evaluate.
        Returns (out [B, nrows, H, d] f64, lse [B, H, nrows] f64, natural log).
        """
        q, k, v = self._f32(q), self._f32(k), self._f32(v)
        B, Nq, H, d = q.shape
        if k.shape != v.shape or k.shape[0] != B or k.shape[2:] != (H, d):
            raise ValueError("shape mismatch")
        Nk = k.shape[1]
        if rows is None:
            rows_arr, rows_ptr, nrows = None, None, Nq
        else:
            rows_arr = np.ascontiguousarray(np.asarray(rows, dtype=np.int64))
            rows_ptr, nrows = rows_arr.ctypes.data, rows_arr.size
        out = np.zeros((B, nrows, H, d), np.float64)
        lse = np.zeros((B, H, nrows), np.float64)
        rc = self.lib.xo_attention(q, k, v, B, Nq, Nk, H, d, rows_ptr, nrows, out,
                                   lse.ctypes.data)
        if rc:
            raise ValueError("xo_attention rejected its arguments")
        return out, lse

    def merge(self, outs, lses):
        """Merge n partials (o_r [B,Nq,H,d], lse_r [B,H,Nq]) -> (o, lse) in f64."""
        outs = [self._f32(o) for o in outs]
        lses = [self._f32(l) for l in lses]
        n = len(outs)
        if n < 1 or len(lses) != n:
            raise ValueError("need n >= 1 matching partials")
        B, Nq, H, d = outs[0].shape
        for o, l in zip(outs, lses):
            if o.shape != (B, Nq, H, d) or l.shape != (B, H, Nq):
                raise ValueError("partial shape mismatch")
        optrs = (ctypes.c_void_p * n)(*[o.ctypes.data for o in outs])
        lptrs = (ctypes.c_void_p * n)(*[l.ctypes.data for l in lses])
        out = np.zeros((B, Nq, H, d), np.float64)
        lse = np.zeros((B, H, Nq), np.float64)
        rc = self.lib.xo_merge(optrs, lptrs, n, B, Nq, H, d, out, lse.ctypes.data)
        if rc:
            raise ValueError("xo_merge rejected its arguments")
        return out, lse

    def patch_update(self, kv_buf, off, fresh_k, fresh_v):
        """Overwrite rows [off, off+len) of kv_buf [2,B,N,H,d] (float32, in place)."""
        if kv_buf.dtype != np.float32 or not kv_buf.flags.c_contiguous:
            raise TypeError("kv_buf must be a C-contiguous float32 array")
        fresh_k, fresh_v = self._f32(fresh_k), self._f32(fresh_v)
        _, B, N, H, d = kv_buf.shape
        length = fresh_k.shape[1]
        if fresh_k.shape != (B, length, H, d) or fresh_v.shape != fresh_k.shape:
            raise ValueError("fresh K/V shape mismatch")
        rc = self.lib.xo_patch_update(kv_buf, int(off), int(length), fresh_k, fresh_v, B, N, H,
                                      d)
        if rc:
            raise ValueError("xo_patch_update rejected its arguments")

    def patch(self, q, kv_buf, off, fresh_k, fresh_v, rows=None):
        """PipeFusion patch step: overwrite rows [off, off+len) of kv_buf
        [2,B,N,H,d] (float32, in place) with the fresh K/V, then the patch's
        queries q [B,len,H,d] attend over the whole updated buffer.
        Returns (out, lse) as attention() does."""
        if kv_buf.dtype != np.float32 or not kv_buf.flags.c_contiguous:
            raise TypeError("kv_buf must be a C-contiguous float32 array")
        q, fresh_k, fresh_v = self._f32(q), self._f32(fresh_k), self._f32(fresh_v)
        _, B, N, H, d = kv_buf.shape
        length = fresh_k.shape[1]
        if (fresh_k.shape != (B, length, H, d) or fresh_v.shape != fresh_k.shape
                or q.shape != fresh_k.shape):
            raise ValueError("q / fresh K/V shape mismatch")
        if rows is None:
            rows_arr, rows_ptr, nrows = None, None, length
        else:
            rows_arr = np.ascontiguousarray(np.asarray(rows, dtype=np.int64))
            rows_ptr, nrows = rows_arr.ctypes.data, rows_arr.size
        out = np.zeros((B, nrows, H, d), np.float64)
        lse = np.zeros((B, H, nrows), np.float64)
        rc = self.lib.xo_patch(q, kv_buf, int(off), int(length), fresh_k, fresh_v, B, N, H, d,
                               rows_ptr, nrows, out, lse.ctypes.data)
        if rc:
            raise ValueError("xo_patch rejected its arguments")
        return out, lse

    def patch_ranges(self, q, kv_buf, ranges, fresh_k, fresh_v, rows=None):
        """Patch step with fresh rows over several disjoint row ranges
        [(off, len), ...] of kv_buf [2,B,N,H,d] (float32, in place; fresh_k/v
        [B, sum(len), H, d] hold the ranges' rows in range order) and its own
        queries q [B,Nq,H,d].  Returns (out, lse) as attention() does."""
        if kv_buf.dtype != np.float32 or not kv_buf.flags.c_contiguous:
            raise TypeError("kv_buf must be a C-contiguous float32 array")
        q, fresh_k, fresh_v = self._f32(q), self._f32(fresh_k), self._f32(fresh_v)
        _, B, N, H, d = kv_buf.shape
        offs = np.ascontiguousarray(np.array([r[0] for r in ranges], dtype=np.int64))
        lens = np.ascontiguousarray(np.array([r[1] for r in ranges], dtype=np.int64))
        F = int(lens.sum())
        if fresh_k.shape != (B, F, H, d) or fresh_v.shape != fresh_k.shape:
            raise ValueError("fresh K/V shape mismatch")
        if q.shape[0] != B or q.shape[2:] != (H, d):
            raise ValueError("q shape mismatch")
        Nq = q.shape[1]
        if rows is None:
            rows_arr, rows_ptr, nrows = None, None, Nq
        else:
            rows_arr = np.ascontiguousarray(np.asarray(rows, dtype=np.int64))
            rows_ptr, nrows = rows_arr.ctypes.data, rows_arr.size
        out = np.zeros((B, nrows, H, d), np.float64)
        lse = np.zeros((B, H, nrows), np.float64)
        rc = self.lib.xo_patch_ranges(q, Nq, kv_buf, len(ranges), offs.ctypes.data,
                                      lens.ctypes.data, fresh_k, fresh_v, B, N, H, d, rows_ptr,
                                      nrows, out, lse.ctypes.data)
        if rc:
            raise ValueError("xo_patch_ranges rejected its arguments")
        return out, lse

    def stage_step(self, x, wq, wk, wv, wo, kv_buf, off, rows=None):
        """One PipeFusion stage micro-step at one attention layer: q/k/v =
        x W{q,k,v} for the patch rows x [B,L,C] (W [C,H*d]), the patch step
        over kv_buf [2,B,N,H,d] (float32, in place: rows [off, off+L) take k/v
        rounded to float), y = o Wo (Wo [H*d,C]).  Returns a dict of float64
        arrays: y [B,nrows,C], o [B,nrows,H,d], q/k/v [B,L,H,d]."""
        if kv_buf.dtype != np.float32 or not kv_buf.flags.c_contiguous:
            raise TypeError("kv_buf must be a C-contiguous float32 array")
        x, wq, wk, wv, wo = (self._f32(a) for a in (x, wq, wk, wv, wo))
        _, B, N, H, d = kv_buf.shape
        L, C = x.shape[1], x.shape[2]
        HD = H * d
        if (x.shape[0] != B or wq.shape != (C, HD) or wk.shape != (C, HD) or wv.shape != (C, HD)
                or wo.shape != (HD, C)):
            raise ValueError("stage shapes mismatch")
        if rows is None:
            rows_ptr, nrows = None, L
        else:
            rows_arr = np.ascontiguousarray(np.asarray(rows, dtype=np.int64))
            rows_ptr, nrows = rows_arr.ctypes.data, rows_arr.size
        res = {"y": np.zeros((B, nrows, C)), "o": np.zeros((B, nrows, H, d)),
               "q": np.zeros((B, L, H, d)), "k": np.zeros((B, L, H, d)), "v": np.zeros((B, L, H, d))}
        rc = self.lib.xo_stage(x, wq, wk, wv, wo, kv_buf, int(off), L, B, N, H, d, C, rows_ptr,
                               nrows, res["y"].ctypes.data, res["o"].ctypes.data,
                               res["q"].ctypes.data, res["k"].ctypes.data, res["v"].ctypes.data)
        if rc:
            raise ValueError("xo_stage rejected its arguments")
        return res


_default = None


def get() -> Oracle:
    """The oracle built from this directory's source (built on first use)."""
    global _default
    if _default is None:
        _default = Oracle(LIBRARY)
    return _default
