"""Device-resident state of one workload and the calls of one hot-path step.

A step is one pass over every part of the path for one layer:
  * the PipeFusion patch steps p = 0..M-1 in order over the layer's K/V
    buffer (each call updates patch p's rows, plus the text rows for patch 0
    with in-context conditioning, and attends over the buffer with the
    patch's queries, or this GPU's shard of them under hybrid parallelism;
    Sections 4.1.2 and 4.1.4), and
    With a hidden size, each patch step is a stage micro-step instead: the
    patch rows' QKV projections, the patch step, the output projection
    (Section 4.1.2).
  * the sequence-parallel share: chunk attention of the local query shard
    against each K/V chunk, then the log-sum-exp merge of the partials
    (Section 4.1.1).
Inputs are uploaded once; every per-call operand is its own dense tensor, as
it would arrive from a projection or a peer, so the timed region holds only
library calls.  Repeating a step is idempotent: after the first pass the
buffer is all fresh and each patch step rewrites the same rows.
"""
from __future__ import annotations

import numpy as np

from . import (split_workspace_bytes, xdit_chunk_attn, xdit_chunk_attn_accum,
               xdit_chunk_attn_accum_split, xdit_chunk_attn_split, xdit_lse_merge, xdit_patch_attn,
               xdit_patch_attn_ranges, xdit_patch_attn_split, xdit_stage_step)
from .inputs import Tensors, Workload


class HotPath:
    def __init__(self, w: Workload, t: Tensors, device: str = "cuda", split: bool = True):
        """split: let the library split each query tile's keys over several
        workgroups where one workgroup per query tile would leave CUs idle."""
        import torch

        self.w = w
        dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
        self.dt = dt

        def up(x):
            return torch.from_numpy(np.ascontiguousarray(x, np.float32)).to(device).to(dt)

        B, H, d = w.B, w.H, w.d
        # K/V buffer at the start of a diffusion step: stale image rows,
        # fresh text rows
        self.kv_stale = up(np.stack([t.k_stale, t.v_stale]))
        self.kv_buf = self.kv_stale.clone()
        # per patch step: fresh ranges and query rows (see Workload.patch_calls)
        self.calls = w.patch_calls()
        self.patch_q, self.patch_k, self.patch_v, self.patch_out = [], [], [], []
        for ranges, qrows in self.calls:
            frows = np.concatenate([np.arange(o, o + n) for o, n in ranges])
            self.patch_q.append(up(t.q[:, qrows]))
            self.patch_k.append(up(t.k_fresh[:, frows]))
            self.patch_v.append(up(t.v_fresh[:, frows]))
            self.patch_out.append(torch.empty((B, len(qrows), H, d), device=device, dtype=dt))
        # stage micro-steps: hidden states of the patch rows, the projections,
        # and the intermediates the library writes
        self.stage = None
        if w.hidden:
            C = w.hidden
            # wq, wk, wv in one [3, C, H*d] tensor and q, k, v of a step in one
            # [3, B, L, H, d] tensor: the library then runs the three
            # projections as one batched GEMM
            wqkv = up(np.stack([t.extra[n] for n in ("wq", "wk", "wv")]))
            self.stage = {"w": [wqkv[0], wqkv[1], wqkv[2], up(t.extra["wo"])],
                          "x": [], "y": [], "qkvo": []}
            for ranges, qrows in self.calls:
                (off, ln), = ranges
                self.stage["x"].append(up(t.extra["x"][:, off:off + ln]))
                self.stage["y"].append(torch.empty((B, ln, C), device=device, dtype=dt))
                qkv = torch.empty((3, B, ln, H, d), device=device, dtype=dt)
                self.stage["qkvo"].append([qkv[0], qkv[1], qkv[2],
                                           torch.empty((B, ln, H, d), device=device, dtype=dt)])
        self.sp_q = self.sp_out = self.sp_lse = None
        self.chunk_k, self.chunk_v, self.chunk_out, self.chunk_lse = [], [], [], []
        if w.sp_chunks:
            q0, q1 = w.sp_q
            nq = q1 - q0
            self.sp_q = up(t.q[:, q0:q1])
            for s, e in w.sp_chunks:
                self.chunk_k.append(up(t.k_fresh[:, s:e]))
                self.chunk_v.append(up(t.v_fresh[:, s:e]))
                if not w.sp_ring:
                    self.chunk_out.append(torch.empty((B, nq, H, d), device=device, dtype=dt))
                    self.chunk_lse.append(torch.empty((B, H, nq), device=device,
                                                      dtype=torch.float32))
            self.sp_out = torch.empty((B, nq, H, d), device=device, dtype=dt)
            self.sp_lse = torch.empty((B, H, nq), device=device, dtype=torch.float32)
        # key-split workspace: the largest any call of the step needs
        need = 0
        self.patch_split = [False] * len(self.calls)
        self.chunk_split = False
        if split and self.stage is None:
            for p in range(len(self.calls)):
                n = split_workspace_bytes(self.patch_q[p], w.N)
                self.patch_split[p] = n > 0
                need = max(need, n)
            if self.sp_q is not None:
                for s_, e_ in w.sp_chunks:
                    n = split_workspace_bytes(self.sp_q, e_ - s_)
                    self.chunk_split = self.chunk_split or n > 0
                    need = max(need, n)
        self.workspace = torch.empty(need, device=device, dtype=torch.uint8) if need else None

    # -- calls ---------------------------------------------------------------
    def reset_buffer(self) -> None:
        self.kv_buf.copy_(self.kv_stale)

    def patch_step(self, p: int) -> None:
        ranges, qrows = self.calls[p]
        if self.stage is not None:
            st = self.stage
            xdit_stage_step(st["x"][p], *st["w"], self.kv_buf, ranges[0][0], *st["qkvo"][p],
                            st["y"][p])
        elif self.patch_split[p]:
            xdit_patch_attn_split(self.patch_q[p], self.kv_buf, ranges, self.patch_k[p],
                                  self.patch_v[p], self.patch_out[p], None, 0, self.workspace)
        elif len(ranges) == 1 and len(qrows) == ranges[0][1]:
            off, ln = ranges[0]
            xdit_patch_attn(self.patch_q[p], self.kv_buf, off, ln, self.patch_k[p],
                            self.patch_v[p], self.patch_out[p])
        else:
            xdit_patch_attn_ranges(self.patch_q[p], self.kv_buf, ranges, self.patch_k[p],
                                   self.patch_v[p], self.patch_out[p])

    def chunk_step(self, r: int) -> None:
        if self.w.sp_ring:
            # ring form: the first chunk starts the running (out, lse), the
            # others are merged into it
            if self.chunk_split:
                f = xdit_chunk_attn_split if r == 0 else xdit_chunk_attn_accum_split
                f(self.sp_q, self.chunk_k[r], self.chunk_v[r], self.sp_out, self.sp_lse, 0,
                  self.workspace)
            else:
                f = xdit_chunk_attn if r == 0 else xdit_chunk_attn_accum
                f(self.sp_q, self.chunk_k[r], self.chunk_v[r], self.sp_out, self.sp_lse)
        elif self.chunk_split:
            xdit_chunk_attn_split(self.sp_q, self.chunk_k[r], self.chunk_v[r], self.chunk_out[r],
                                  self.chunk_lse[r], 0, self.workspace)
        else:
            xdit_chunk_attn(self.sp_q, self.chunk_k[r], self.chunk_v[r], self.chunk_out[r],
                            self.chunk_lse[r])

    def merge(self) -> None:
        n = len(self.chunk_out)
        if n == 0:
            return
        xdit_lse_merge(self.chunk_out, self.chunk_lse, n, self.sp_out, self.sp_lse)

    def step(self) -> None:
        for p in range(len(self.patch_q)):
            self.patch_step(p)
        if self.sp_q is not None:
            for r in range(len(self.chunk_k)):
                self.chunk_step(r)
            if not self.w.sp_ring:
                self.merge()

    # -- accounting ----------------------------------------------------------
    def patch_flops(self, p: int) -> float:
        f = self.w.attn_flops(len(self.calls[p][1]), self.w.N)
        if self.stage is not None:
            f += self.gemm_flops(p)
        return f

    def gemm_flops(self, p: int) -> float:
        """The stage micro-step's four projections, 2*B*L*C*(H*d) each."""
        w = self.w
        return 4 * 2.0 * w.B * len(self.calls[p][1]) * w.hidden * w.H * w.d if w.hidden else 0.0

    def chunk_flops(self, r: int) -> float:
        s, e = self.w.sp_chunks[r]
        return self.w.attn_flops(self.w.sp_q[1] - self.w.sp_q[0], e - s)

    def step_flops(self) -> float:
        f = sum(self.patch_flops(p) for p in range(len(self.patch_q)))
        if self.sp_q is not None:
            f += sum(self.chunk_flops(r) for r in range(len(self.chunk_k)))
        return f

    def merge_bytes(self) -> float:
        """n partials (O and LSE) read, merged O and LSE written."""
        w = self.w
        nq = w.sp_q[1] - w.sp_q[0]
        n = len(w.sp_chunks)
        o = w.B * nq * w.H * w.d * w.esize
        lse = 4 * w.B * w.H * nq
        return n * (o + lse) + o + lse

    def update_bytes(self, p: int) -> float:
        """K and V fresh rows: read from the fresh tensors and written to the buffer."""
        w = self.w
        ln = sum(n for _, n in self.calls[p][0])
        return 2 * 2 * w.B * ln * w.H * w.d * w.esize
