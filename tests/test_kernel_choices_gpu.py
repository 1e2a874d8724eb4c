"""Parity of each bf16 attention decomposition, forced with
XDIT_ATTN_KERNEL whatever the default for the head dim: "o2" (workgroups of
4 waves, two per CU), "w32" (8-wave workgroups), "pp" (8-wave workgroups
whose two halves alternate matrix and softmax phases) and "w64" (64 query
rows per wave with the output accumulators in AGPRs, head dim 128), on the
chunk step, the patch step, the ring step and partitioned launches, against
the fp64 oracle.  The library's default choice runs every other GPU test."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
import paper_2411_01738_amd as xd
from paper_2411_01738_amd.inputs import random_io
from tests.gpu_util import check_lse, check_out, to_gpu, to_np, torch_mod

pytestmark = pytest.mark.gpu


@pytest.fixture(params=["o2", "w32", "pp", "w64"])
def choice(request, monkeypatch):
    monkeypatch.setenv("XDIT_ATTN_KERNEL", request.param)
    return request.param


def _dims(choice):
    return [128] if choice == "w64" else [64, 72, 128]


CHUNKS = [(2, 200, 333, 3), (1, 1, 1, 1), (1, 130, 645, 2), (2, 129, 190, 2), (1, 64, 0, 2)]


def test_chunk(choice):
    torch = torch_mod()
    orc = oracle.get()
    for d in _dims(choice):
        for B, Nq, Nk, H in CHUNKS:
            seed = 1000 + Nq + Nk + d
            q = random_io((B, Nq, H, d), "bf16", seed)
            k = random_io((B, Nk, H, d), "bf16", seed + 1)
            v = random_io((B, Nk, H, d), "bf16", seed + 2)
            out = torch.full((B, Nq, H, d), float("nan"), device="cuda", dtype=torch.bfloat16)
            lse = torch.full((B, H, Nq), float("nan"), device="cuda", dtype=torch.float32)
            xd.xdit_chunk_attn(to_gpu(q, "bf16"), to_gpu(k, "bf16"), to_gpu(v, "bf16"), out, lse)
            torch.cuda.synchronize()
            ro, rl = orc.attention(q, k, v)
            check_out(to_np(out), ro, "bf16", f"{choice} chunk d={d} {B, Nq, Nk, H}")
            check_lse(lse.cpu().numpy(), rl, "bf16", f"{choice} chunk lse d={d} {B, Nq, Nk, H}")


def test_patch_steps(choice):
    """Sequential patch steps with ranges that straddle tiles, buffer bit-exact."""
    torch = torch_mod()
    orc = oracle.get()
    for d in _dims(choice):
        B, N, H = 2, 300, 2
        seed = 2000 + d
        q = random_io((B, N, H, d), "bf16", seed)
        kf = random_io((B, N, H, d), "bf16", seed + 1)
        vf = random_io((B, N, H, d), "bf16", seed + 2)
        kv_ref = np.ascontiguousarray(np.stack([random_io((B, N, H, d), "bf16", seed + 3),
                                                random_io((B, N, H, d), "bf16", seed + 4)]))
        kv = to_gpu(kv_ref, "bf16")
        for off, ln in [(37, 150), (0, 37), (187, 113)]:
            sl = slice(off, off + ln)
            ref_o, _ = orc.patch(q[:, sl].copy(), kv_ref, off, kf[:, sl].copy(), vf[:, sl].copy())
            out = torch.full((B, ln, H, d), float("nan"), device="cuda", dtype=torch.bfloat16)
            xd.xdit_patch_attn(to_gpu(q[:, sl], "bf16"), kv, off, ln, to_gpu(kf[:, sl], "bf16"),
                               to_gpu(vf[:, sl], "bf16"), out)
            torch.cuda.synchronize()
            check_out(to_np(out), ref_o, "bf16", f"{choice} patch d={d} ({off},{ln})")
            assert np.array_equal(to_np(kv), kv_ref), f"{choice} d={d}: buffer not bit-exact"


def test_ring_and_splits(choice):
    """The ring step unsplit and split, and a forced split of the chunk step,
    over a K/V length of many tiles with a ragged end."""
    torch = torch_mod()
    orc = oracle.get()
    for d in _dims(choice):
        B, Nq, H, Nk = 2, 200, 2, 1300
        seed = 3000 + d
        q = random_io((B, Nq, H, d), "bf16", seed)
        k = random_io((B, Nk, H, d), "bf16", seed + 1)
        v = random_io((B, Nk, H, d), "bf16", seed + 2)
        qg = to_gpu(q, "bf16")
        ro, rl = orc.attention(q, k, v)
        chunks = [(0, 500), (500, 1300)]
        for split in (False, True):
            ws = torch.empty(max(1, max(xd.split_workspace_bytes(qg, e - s_, 3) for s_, e in chunks)),
                             device="cuda", dtype=torch.uint8)
            out = torch.full((B, Nq, H, d), float("nan"), device="cuda", dtype=torch.bfloat16)
            lse = torch.full((B, H, Nq), float("-inf"), device="cuda", dtype=torch.float32)
            for s_, e in chunks:
                kc, vc = to_gpu(k[:, s_:e], "bf16"), to_gpu(v[:, s_:e], "bf16")
                if split:
                    xd.xdit_chunk_attn_accum_split(qg, kc, vc, out, lse, 3, ws)
                else:
                    xd.xdit_chunk_attn_accum(qg, kc, vc, out, lse)
            torch.cuda.synchronize()
            check_out(to_np(out), ro, "bf16", f"{choice} ring d={d} split={split}")
            check_lse(lse.cpu().numpy(), rl, "bf16", f"{choice} ring lse d={d} split={split}")
        ws = torch.empty(xd.split_workspace_bytes(qg, Nk, 4), device="cuda", dtype=torch.uint8)
        out = torch.full((B, Nq, H, d), float("nan"), device="cuda", dtype=torch.bfloat16)
        lse = torch.empty((B, H, Nq), device="cuda", dtype=torch.float32)
        xd.xdit_chunk_attn_split(qg, to_gpu(k, "bf16"), to_gpu(v, "bf16"), out, lse, 4, ws)
        torch.cuda.synchronize()
        check_out(to_np(out), ro, "bf16", f"{choice} split 4 d={d}")
        check_lse(lse.cpu().numpy(), rl, "bf16", f"{choice} split 4 lse d={d}")
