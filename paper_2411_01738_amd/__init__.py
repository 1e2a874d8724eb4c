"""MI355X (gfx950) DiT attention hot path of xDiT (arXiv 2411.01738).

Thin binding over the C ABI of libxdit.so (include/xdit.h): each function
takes torch tensors that already live on the GPU, checks that they are dense,
reads their sizes, passes raw device pointers and torch's current stream, and
raises XditError when the library rejects the call.  All arithmetic runs in
the library's HIP kernels; there is no host or PyTorch fallback.

Layouts: activations [B, N, H, d]; K/V buffer [2, B, N, H, d]; LSE [B, H, Nq]
float32.  dtypes: bfloat16 or float32 (LSE always float32).
"""
from __future__ import annotations

import ctypes

from ._lib import (XDIT_BF16, XDIT_F32, XDIT_MAX_PARTIALS, XDIT_MAX_RANGES, XDIT_MAX_SPLITS,
                   XditError, check, lib)

__all__ = ["xdit_patch_attn", "xdit_patch_attn_ranges", "xdit_chunk_attn",
           "xdit_chunk_attn_accum", "xdit_chunk_attn_accum_split", "xdit_chunk_attn_split",
           "xdit_patch_attn_split", "xdit_chunk_attn_split_noalloc",
           "split_workspace_bytes", "xdit_lse_merge",
           "xdit_kv_update", "xdit_stage_step", "set_stream", "XditError", "XDIT_MAX_PARTIALS", "XDIT_MAX_RANGES",
           "version"]


def _torch():
    import torch
    return torch


def _dtype_code(t) -> int:
    torch = _torch()
    if t.dtype == torch.bfloat16:
        return XDIT_BF16
    if t.dtype == torch.float32:
        return XDIT_F32
    raise XditError(-2, f"unsupported dtype {t.dtype}")


def _dense(t, name: str, ndim: int):
    if t is None:
        return None
    if not t.is_cuda:
        raise XditError(-1, f"{name} must be a GPU tensor")
    if t.dim() != ndim:
        raise XditError(-3, f"{name} must have {ndim} dims, got {tuple(t.shape)}")
    if not t.is_contiguous():
        raise XditError(-5, f"{name} must be contiguous")
    return t


def _ptr(t) -> int | None:
    return None if t is None else t.data_ptr()


def _use_current_stream() -> None:
    lib().xdit_set_stream(_torch().cuda.current_stream().cuda_stream)


def set_stream(stream) -> None:
    """Route later calls of this thread to `stream` (a torch.cuda.Stream or a raw
    hipStream_t handle).  The functions below always use torch's current stream."""
    handle = getattr(stream, "cuda_stream", stream)
    check(lib().xdit_set_stream(handle))


def version() -> str:
    return lib().xdit_version().decode()


def xdit_patch_attn(q, kv_buf, patch_off: int, patch_len: int, fresh_k, fresh_v, out) -> None:
    """PipeFusion patch step: write fresh_k/fresh_v into rows
    [patch_off, patch_off+patch_len) of kv_buf [2,B,N,H,d] (in place), then
    out = attention(q, updated K, updated V) for the patch's queries
    q [B,patch_len,H,d]."""
    _dense(kv_buf, "kv_buf", 5)
    for t, n in ((q, "q"), (fresh_k, "fresh_k"), (fresh_v, "fresh_v"), (out, "out")):
        _dense(t, n, 4)
    _, B, N, H, d = kv_buf.shape
    for t, n in ((q, "q"), (fresh_k, "fresh_k"), (fresh_v, "fresh_v"), (out, "out")):
        if tuple(t.shape) != (B, patch_len, H, d):
            raise XditError(-3, f"{n} has shape {tuple(t.shape)}, expected {(B, patch_len, H, d)}")
        if t.dtype != kv_buf.dtype:
            raise XditError(-2, f"{n} dtype {t.dtype} differs from kv_buf's {kv_buf.dtype}")
    _use_current_stream()
    check(lib().xdit_patch_attn(_ptr(q), _ptr(kv_buf), int(patch_off), int(patch_len),
                                _ptr(fresh_k), _ptr(fresh_v), _ptr(out), B, N, H, d,
                                _dtype_code(kv_buf)))


def xdit_patch_attn_ranges(q, kv_buf, ranges, fresh_k, fresh_v, out, lse=None) -> None:
    """General patch step: write fresh_k/fresh_v [B, F, H, d] into the row
    ranges [(off, len), ...] of kv_buf [2,B,N,H,d] (range 0's rows first; F =
    sum of the lengths), then out = attention(q, updated K, updated V) for the
    queries q [B,Nq,H,d] and, if given, lse [B,H,Nq] (natural log)."""
    _dense(kv_buf, "kv_buf", 5)
    for t, n in ((q, "q"), (fresh_k, "fresh_k"), (fresh_v, "fresh_v"), (out, "out")):
        _dense(t, n, 4)
    _dense(lse, "lse", 3)
    _, B, N, H, d = kv_buf.shape
    nr = len(ranges)
    F = sum(int(r[1]) for r in ranges)
    Nq = q.shape[1]
    for t, n, rows in ((q, "q", Nq), (out, "out", Nq), (fresh_k, "fresh_k", F),
                       (fresh_v, "fresh_v", F)):
        if tuple(t.shape) != (B, rows, H, d):
            raise XditError(-3, f"{n} has shape {tuple(t.shape)}, expected {(B, rows, H, d)}")
        if t.dtype != kv_buf.dtype:
            raise XditError(-2, f"{n} dtype {t.dtype} differs from kv_buf's {kv_buf.dtype}")
    if lse is not None:
        torch = _torch()
        if lse.dtype != torch.float32 or tuple(lse.shape) != (B, H, Nq):
            raise XditError(-3, f"lse must be float32 [B,H,Nq] = {(B, H, Nq)}")
    offs = (ctypes.c_int64 * max(nr, 1))(*[int(r[0]) for r in ranges])
    lens = (ctypes.c_int64 * max(nr, 1))(*[int(r[1]) for r in ranges])
    _use_current_stream()
    check(lib().xdit_patch_attn_ranges(_ptr(q), Nq, _ptr(kv_buf), nr, offs, lens, _ptr(fresh_k),
                                       _ptr(fresh_v), _ptr(out), _ptr(lse), B, N, H, d,
                                       _dtype_code(kv_buf)))


def _chunk_args(q, k, v, out, lse):
    for t, n in ((q, "q"), (k, "k"), (v, "v"), (out, "out")):
        _dense(t, n, 4)
    _dense(lse, "lse", 3)
    B, Nq, H, d = q.shape
    Nk = k.shape[1]
    if tuple(k.shape) != (B, Nk, H, d) or tuple(v.shape) != (B, Nk, H, d):
        raise XditError(-3, f"k/v shapes {tuple(k.shape)}/{tuple(v.shape)} do not match q")
    if tuple(out.shape) != (B, Nq, H, d):
        raise XditError(-3, "out shape differs from q")
    for t, n in ((k, "k"), (v, "v"), (out, "out")):
        if t.dtype != q.dtype:
            raise XditError(-2, f"{n} dtype differs from q's")
    if lse is not None:
        torch = _torch()
        if lse.dtype != torch.float32 or tuple(lse.shape) != (B, H, Nq):
            raise XditError(-3, f"lse must be float32 [B,H,Nq] = {(B, H, Nq)}")
    return (_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(lse), B, Nq, Nk, H, d, _dtype_code(q))


def xdit_chunk_attn(q, k, v, out, lse=None) -> None:
    """Chunk attention: out = attention(q, k, v) and, if given,
    lse [B,H,Nq] = log-sum-exp of the scaled scores (natural log)."""
    args = _chunk_args(q, k, v, out, lse)
    _use_current_stream()
    check(lib().xdit_chunk_attn(*args))


def split_workspace_bytes(q, kv_len: int, splits: int = 0) -> int:
    """Bytes of workspace the *_split calls need for queries shaped like q
    [B,Nq,H,d] over kv_len keys (0 when no split happens)."""
    B, Nq, H, d = q.shape
    n = lib().xdit_split_workspace_bytes(B, Nq, int(kv_len), H, d, _dtype_code(q), int(splits))
    if n < 0:
        raise XditError(-3, "xdit_split_workspace_bytes rejected the sizes")
    return int(n)


def _workspace(ws):
    if ws is None:
        return None, 0
    if not ws.is_cuda or not ws.is_contiguous():
        raise XditError(-5, "workspace must be a dense GPU tensor")
    return ws.data_ptr(), ws.numel() * ws.element_size()


def xdit_chunk_attn_split(q, k, v, out, lse=None, splits: int = 0, workspace=None) -> None:
    """xdit_chunk_attn with each query tile's keys split `splits` ways (0: the
    library chooses); workspace: a GPU tensor of split_workspace_bytes bytes."""
    args = _chunk_args(q, k, v, out, lse)
    wp, wb = _workspace(workspace)
    _use_current_stream()
    check(lib().xdit_chunk_attn_split(*args[:5], int(splits), wp, wb, *args[5:]))


def xdit_chunk_attn_split_noalloc(q, k, v, out, lse=None, splits: int = 0) -> None:
    """xdit_chunk_attn_split with the partials kept in the library's fixed
    per-GPU scratch array (no workspace, nothing allocated)."""
    args = _chunk_args(q, k, v, out, lse)
    _use_current_stream()
    check(lib().xdit_chunk_attn_split_noalloc(*args[:5], int(splits), *args[5:]))


def xdit_patch_attn_split(q, kv_buf, ranges, fresh_k, fresh_v, out, lse=None, splits: int = 0,
                          workspace=None) -> None:
    """xdit_patch_attn_ranges with the keys split `splits` ways (0: the
    library chooses); workspace as for xdit_chunk_attn_split."""
    _dense(kv_buf, "kv_buf", 5)
    for t, n in ((q, "q"), (fresh_k, "fresh_k"), (fresh_v, "fresh_v"), (out, "out")):
        _dense(t, n, 4)
    _dense(lse, "lse", 3)
    _, B, N, H, d = kv_buf.shape
    nr = len(ranges)
    offs = (ctypes.c_int64 * max(nr, 1))(*[int(r[0]) for r in ranges])
    lens = (ctypes.c_int64 * max(nr, 1))(*[int(r[1]) for r in ranges])
    wp, wb = _workspace(workspace)
    _use_current_stream()
    check(lib().xdit_patch_attn_split(_ptr(q), q.shape[1], _ptr(kv_buf), nr, offs, lens,
                                      _ptr(fresh_k), _ptr(fresh_v), _ptr(out), _ptr(lse),
                                      int(splits), wp, wb, B, N, H, d, _dtype_code(kv_buf)))


def xdit_chunk_attn_accum(q, k, v, out, lse) -> None:
    """Ring step: merge attention(q, k, v) into the running (out, lse) in
    place.  lse = -inf marks an empty running state (out then ignored)."""
    if lse is None:
        raise XditError(-1, "the running lse is required")
    args = _chunk_args(q, k, v, out, lse)
    _use_current_stream()
    check(lib().xdit_chunk_attn_accum(*args))


def xdit_chunk_attn_accum_split(q, k, v, out, lse, splits: int = 0, workspace=None) -> None:
    """xdit_chunk_attn_accum with each query tile's keys split `splits` ways
    (0: the library chooses); workspace as for xdit_chunk_attn_split."""
    if lse is None:
        raise XditError(-1, "the running lse is required")
    args = _chunk_args(q, k, v, out, lse)
    wp, wb = _workspace(workspace)
    _use_current_stream()
    check(lib().xdit_chunk_attn_accum_split(*args[:5], int(splits), wp, wb, *args[5:]))


def xdit_lse_merge(outs, lses, n: int, out, lse_out=None) -> None:
    """Merge n chunk partials (outs[r] [B,Nq,H,d], lses[r] [B,H,Nq] float32)
    into out, and the merged log-sum-exp into lse_out if given."""
    n = int(n)
    if n < 1 or n > len(outs) or n > len(lses):
        raise XditError(-4, f"n = {n} does not match {len(outs)} outs / {len(lses)} lses")
    _dense(out, "out", 4)
    _dense(lse_out, "lse_out", 3)
    B, Nq, H, d = out.shape
    torch = _torch()
    for r in range(n):
        _dense(outs[r], f"outs[{r}]", 4)
        _dense(lses[r], f"lses[{r}]", 3)
        if tuple(outs[r].shape) != (B, Nq, H, d) or outs[r].dtype != out.dtype:
            raise XditError(-3, f"outs[{r}] does not match out")
        if tuple(lses[r].shape) != (B, H, Nq) or lses[r].dtype != torch.float32:
            raise XditError(-3, f"lses[{r}] must be float32 {(B, H, Nq)}")
    optrs = (ctypes.c_void_p * n)(*[outs[r].data_ptr() for r in range(n)])
    lptrs = (ctypes.c_void_p * n)(*[lses[r].data_ptr() for r in range(n)])
    _use_current_stream()
    check(lib().xdit_lse_merge(optrs, lptrs, n, _ptr(out), _ptr(lse_out), B, Nq, H, d,
                               _dtype_code(out)))


def xdit_kv_update(kv_buf, patch_off: int, patch_len: int, fresh_k, fresh_v) -> None:
    """Copy fresh K/V [B,patch_len,H,d] into rows [patch_off, patch_off+patch_len)
    of kv_buf [2,B,N,H,d], bit for bit."""
    _dense(kv_buf, "kv_buf", 5)
    _dense(fresh_k, "fresh_k", 4)
    _dense(fresh_v, "fresh_v", 4)
    _, B, N, H, d = kv_buf.shape
    for t, nm in ((fresh_k, "fresh_k"), (fresh_v, "fresh_v")):
        if tuple(t.shape) != (B, patch_len, H, d) or t.dtype != kv_buf.dtype:
            raise XditError(-3, f"{nm} must be {(B, patch_len, H, d)} of kv_buf's dtype")
    _use_current_stream()
    check(lib().xdit_kv_update(_ptr(kv_buf), int(patch_off), int(patch_len), _ptr(fresh_k),
                               _ptr(fresh_v), B, N, H, d, _dtype_code(kv_buf)))


def xdit_stage_step(x, wq, wk, wv, wo, kv_buf, patch_off: int, q, k, v, o, y) -> None:
    """One PipeFusion stage micro-step at one attention layer: q/k/v = x
    W{q,k,v} (x [B,L,C], W [C,H*d]), the patch step over kv_buf [2,B,N,H,d]
    at rows [patch_off, patch_off+L) with fresh K/V (k, v) and output o, then
    y = o wo (wo [H*d,C]).  q, k, v, o [B,L,H,d] and y [B,L,C] are written."""
    _dense(kv_buf, "kv_buf", 5)
    _, B, N, H, d = kv_buf.shape
    _dense(x, "x", 3)
    L, C = x.shape[1], x.shape[2]
    if x.shape[0] != B:
        raise XditError(-3, f"x must be [B, L, C] with B = {B}")
    for t, nm, shp in ((wq, "wq", (C, H * d)), (wk, "wk", (C, H * d)), (wv, "wv", (C, H * d)),
                       (wo, "wo", (H * d, C)), (y, "y", (B, L, C))):
        _dense(t, nm, len(shp))
        if tuple(t.shape) != shp or t.dtype != x.dtype:
            raise XditError(-3, f"{nm} must be {shp} of x's dtype")
    for t, nm in ((q, "q"), (k, "k"), (v, "v"), (o, "o")):
        _dense(t, nm, 4)
        if tuple(t.shape) != (B, L, H, d) or t.dtype != x.dtype:
            raise XditError(-3, f"{nm} must be {(B, L, H, d)} of x's dtype")
    if kv_buf.dtype != x.dtype:
        raise XditError(-3, "kv_buf must have x's dtype")
    _use_current_stream()
    check(lib().xdit_stage_step(_ptr(x), _ptr(wq), _ptr(wk), _ptr(wv), _ptr(wo), _ptr(kv_buf),
                                int(patch_off), L, _ptr(q), _ptr(k), _ptr(v), _ptr(o), _ptr(y), B,
                                N, H, d, C, _dtype_code(x)))
