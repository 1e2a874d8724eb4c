"""Seeded synthetic inputs for the DiT attention workloads.

This module is shared by the tests, the benchmark and the oracle checks.  It
holds only input generation (random draws, bf16 rounding, sizes) and none of
the attention arithmetic.

The workloads follow the model shapes of the paper's experiments (Section 5:
Pixart, SD3, Flux.1 and CogVideoX).  The real models' activations and weights
are not available, so every tensor is iid N(0, 1) from a fixed seed and the
stale K/V of the previous diffusion step is the fresh K/V plus N(0, 0.05^2)
noise (input temporal redundancy, Section 2), drawn in float32 and then
rounded to the I/O dtype.  Text (condition) tokens sit after the image tokens
in the joint sequence (Section 3: MM-DiT concatenates them on the sequence
axis) and are never stale.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    dtype: str            # "bf16" or "f32": the I/O dtype of Q/K/V/O
    B: int                # batch (2 = the classifier-free-guidance pair)
    H: int                # heads
    d: int                # head dim
    n_img: int            # image / video tokens (the patched part of the sequence)
    n_txt: int            # text tokens appended after the image tokens
    M: int                # PipeFusion patch count over the image tokens
    seed: int
    # sequence-parallel leg: query rows and K/V chunk boundaries (row ranges)
    sp_q: tuple = ()      # (start, stop) of the query rows of the local shard
    sp_chunks: tuple = ()  # ((start, stop), ...) K/V row ranges, one per chunk
    # PipeFusion variants (Sections 4.1.2 and 4.1.4)
    in_context: bool = False  # the text rows travel with patch 0
    balanced: bool = False    # with in_context: patch 0 takes fewer image rows, so
                              # that every patch step refreshes about as many rows
    sp_degree: int = 1        # hybrid SP x PipeFusion: this GPU's queries are the
                              # first 1/sp_degree of each patch step's query rows
    sp_ring: bool = False     # SP chunks merged into a running (out, lse) one by one
                              # instead of stored as partials and merged at the end
    hidden: int = 0           # > 0: each patch step is a stage micro-step with QKV
                              # and output projections of this hidden size
    note: str = ""

    @property
    def N(self) -> int:
        return self.n_img + self.n_txt

    def patches(self):
        """(offset, length) of the M patches: contiguous splits of the image
        rows, near-equal (the first n_img mod M one row longer), or, for
        a balanced in-context partition, patch 0 cut to about
        (n_img + n_txt) / M - n_txt rows and the rest split near-equally
        over the other patches, so that patch 0 with the text rows is no
        longer than the others."""
        if self.M == 0:
            return []
        lens = []
        if self.in_context and self.balanced and self.M > 1:
            first = max(0, min(self.n_img, (self.n_img + self.n_txt) // self.M - self.n_txt))
            base, extra = divmod(self.n_img - first, self.M - 1)
            lens = [first] + [base + (1 if p < extra else 0) for p in range(self.M - 1)]
        else:
            base, extra = divmod(self.n_img, self.M)
            lens = [base + (1 if p < extra else 0) for p in range(self.M)]
        out, off = [], 0
        for ln in lens:
            out.append((off, ln))
            off += ln
        return out

    def patch_calls(self):
        """Per patch step: (fresh ranges [(off, len), ...], query rows).  The
        fresh rows are the patch's image rows, plus the text rows for patch 0
        when in_context; the query rows are those rows, cut to this GPU's
        first shard of sp_degree when sp_degree > 1."""
        calls = []
        for p, (off, ln) in enumerate(self.patches()):
            ranges = [(off, ln)]
            if self.in_context and p == 0 and self.n_txt > 0:
                ranges.append((self.n_img, self.n_txt))
            rows = np.concatenate([np.arange(o, o + n) for o, n in ranges]).astype(np.int64)
            if self.sp_degree > 1:
                rows = rows[:(len(rows) + self.sp_degree - 1) // self.sp_degree]
            calls.append((ranges, rows))
        return calls

    def attn_flops(self, nq: int, nk: int) -> float:
        """Algorithmic attention FLOPs, 4*B*H*Nq*Nk*d (QK^T and PV)."""
        return 4.0 * self.B * self.H * nq * nk * self.d

    @property
    def esize(self) -> int:
        return 2 if self.dtype == "bf16" else 4


def _even_chunks(n: int, parts: int):
    base, extra = divmod(n, parts)
    out, s = [], 0
    for r in range(parts):
        ln = base + (1 if r < extra else 0)
        out.append((s, s + ln))
        s += ln
    return tuple(out)


WORKLOADS = {
    "tiny": Workload("tiny", "f32", 1, 2, 64, 256, 0, 4, 0,
                     sp_q=(0, 256), sp_chunks=_even_chunks(256, 4),
                     note="tiny DiT attention, fp32, 4 patches of 64, 4-chunk merge"),
    "pixart": Workload("pixart", "bf16", 2, 16, 72, 4096, 0, 4, 1,
                       sp_q=(0, 1024), sp_chunks=_even_chunks(4096, 4),
                       note="Pixart 1024px: 128x128 latent, 2x2 patchify, CFG pair"),
    "sd3": Workload("sd3", "bf16", 2, 24, 64, 4096, 333, 8, 2,
                    note="SD3 joint attention: 4096 image + 333 text tokens"),
    "sd3_ic": Workload("sd3_ic", "bf16", 2, 24, 64, 4096, 333, 8, 2, in_context=True,
                       note="SD3 with in-context conditioning: the 333 text tokens travel"
                            " with patch 0"),
    "sd3_ic_bal": Workload("sd3_ic_bal", "bf16", 2, 24, 64, 4096, 333, 8, 2, in_context=True,
                           balanced=True,
                           note="SD3 with in-context conditioning and a load-balanced image"
                                " partition: patch 0 takes 220 image rows + the 333 text rows"),
    "pixart_stage": Workload("pixart_stage", "bf16", 2, 16, 72, 4096, 0, 4, 1, hidden=1152,
                             note="Pixart 1024px stage micro-steps: per patch, QKV projections"
                                  " (hidden 1152), the patch step, the output projection"),
    "pixart_hybrid": Workload("pixart_hybrid", "bf16", 2, 16, 72, 4096, 0, 4, 1, sp_degree=2,
                              note="Pixart 1024px, PipeFusion x 2-way sequence parallelism:"
                                   " gathered fresh K/V, this GPU's half of each patch's"
                                   " queries"),
    "flux": Workload("flux", "bf16", 1, 24, 128, 16384, 512, 0, 3,
                     sp_q=(0, 4224), sp_chunks=_even_chunks(16896, 4),
                     note="Flux 2048px sequence-parallel share: 4 shards of 4096 image"
                          " + 128 text tokens; Q is shard 0"),
    "flux_ring": Workload("flux_ring", "bf16", 1, 24, 128, 16384, 512, 0, 3,
                          sp_q=(0, 4224), sp_chunks=_even_chunks(16896, 4), sp_ring=True,
                          note="Flux 2048px sequence-parallel share, ring form: each chunk"
                               " is merged into the running output as it arrives"),
    "cog": Workload("cog", "bf16", 1, 48, 64, 17550, 226, 16, 4,
                    sp_q=(0, 17776), sp_chunks=_even_chunks(17776, 8),
                    note="CogVideoX video: 13x30x45 latent grid + 226 text tokens"),
}


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round float32 to the nearest bfloat16 (ties to even); returns float32
    holding the rounded values.  Finite inputs only."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    bias = ((u >> 16) & np.uint32(1)) + np.uint32(0x7FFF)
    r = ((u + bias) & np.uint32(0xFFFF0000)).astype(np.uint32)
    return r.view(np.float32)


def to_io(x: np.ndarray, dtype: str) -> np.ndarray:
    return bf16_round(x) if dtype == "bf16" else np.ascontiguousarray(x, dtype=np.float32)


@dataclass
class Tensors:
    """float32 arrays holding the exact I/O-dtype values."""
    q: np.ndarray          # [B, N, H, d]
    k_fresh: np.ndarray    # [B, N, H, d]
    v_fresh: np.ndarray    # [B, N, H, d]
    k_stale: np.ndarray    # [B, N, H, d] (text rows equal the fresh ones)
    v_stale: np.ndarray
    extra: dict = field(default_factory=dict)


def generate(w: Workload, seed: int | None = None) -> Tensors:
    """Draw, in this order from numpy PCG64(seed): Q, K, V [B, N, H, d], then
    the K and V staleness noise [B, n_img, H, d]; all standard normal float32.
    stale = fresh + 0.05 * noise on image rows (float32), then every tensor is
    rounded to the I/O dtype.  With hidden = C > 0, the same generator then
    draws the image rows' hidden states x [B, n_img, C] (standard normal) and
    the projections wq, wk, wv [C, H*d] (scale 1/sqrt(C)) and wo [H*d, C]
    (scale 1/sqrt(H*d)), kept in extra."""
    rng = np.random.Generator(np.random.PCG64(w.seed if seed is None else seed))
    shape = (w.B, w.N, w.H, w.d)
    q = rng.standard_normal(shape, dtype=np.float32)
    k = rng.standard_normal(shape, dtype=np.float32)
    v = rng.standard_normal(shape, dtype=np.float32)
    nshape = (w.B, w.n_img, w.H, w.d)
    k_stale = k.copy()
    k_stale[:, :w.n_img] += np.float32(0.05) * rng.standard_normal(nshape, dtype=np.float32)
    v_stale = v.copy()
    v_stale[:, :w.n_img] += np.float32(0.05) * rng.standard_normal(nshape, dtype=np.float32)
    t = Tensors(to_io(q, w.dtype), to_io(k, w.dtype), to_io(v, w.dtype),
                to_io(k_stale, w.dtype), to_io(v_stale, w.dtype))
    if w.hidden:
        C, HD = w.hidden, w.H * w.d
        t.extra["x"] = to_io(rng.standard_normal((w.B, w.n_img, C), dtype=np.float32), w.dtype)
        for name in ("wq", "wk", "wv"):
            t.extra[name] = to_io(rng.standard_normal((C, HD), dtype=np.float32)
                                  * np.float32(1.0 / np.sqrt(C)), w.dtype)
        t.extra["wo"] = to_io(rng.standard_normal((HD, C), dtype=np.float32)
                              * np.float32(1.0 / np.sqrt(HD)), w.dtype)
    return t


def random_io(shape, dtype: str, seed: int, scale: float = 1.0) -> np.ndarray:
    """iid N(0, scale^2) float32 of `shape`, rounded to the I/O dtype."""
    rng = np.random.Generator(np.random.PCG64(seed))
    x = rng.standard_normal(shape, dtype=np.float32) * np.float32(scale)
    return to_io(x, dtype)


def sample_rows(n: int, step: int = 7, extra=()) -> np.ndarray:
    """Deterministic row sample: every `step`-th row, the first and last row,
    and the given extra rows (e.g. patch or chunk boundaries)."""
    rows = set(range(0, n, step)) | {0, n - 1} | {r for r in extra if 0 <= r < n}
    return np.array(sorted(rows), dtype=np.int64)
