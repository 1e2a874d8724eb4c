"""The allocation-free split entry point against the workspace one: same
partition, same kernels, so the results must agree bit for bit; two calls in
a row on the shared scratch array, the second smaller, and a partition too
large for the array rejected before any launch."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
import paper_2411_01738_amd as xd
from paper_2411_01738_amd import _lib
from paper_2411_01738_amd.inputs import random_io
from tests.gpu_util import check_lse, check_out, to_gpu, to_np, torch_mod

pytestmark = pytest.mark.gpu


def _run_pair(torch, B, Nq, Nk, H, d, splits, seed):
    q = random_io((B, Nq, H, d), "bf16", seed)
    k = random_io((B, Nk, H, d), "bf16", seed + 1)
    v = random_io((B, Nk, H, d), "bf16", seed + 2)
    qg, kg, vg = to_gpu(q, "bf16"), to_gpu(k, "bf16"), to_gpu(v, "bf16")
    need = xd.split_workspace_bytes(qg, Nk, splits)
    assert 0 < need <= _lib.lib().xdit_noalloc_scratch_bytes(), need
    # reference: the workspace entry point, with a NaN-filled workspace
    ws = torch.full((need // 4,), float("nan"), device="cuda", dtype=torch.float32)
    o_ref = torch.full((B, Nq, H, d), float("nan"), device="cuda", dtype=torch.bfloat16)
    l_ref = torch.full((B, H, Nq), float("nan"), device="cuda", dtype=torch.float32)
    xd.xdit_chunk_attn_split(qg, kg, vg, o_ref, l_ref, splits, ws)
    o = torch.full((B, Nq, H, d), float("nan"), device="cuda", dtype=torch.bfloat16)
    l = torch.full((B, H, Nq), float("nan"), device="cuda", dtype=torch.float32)
    xd.xdit_chunk_attn_split_noalloc(qg, kg, vg, o, l, splits)
    torch.cuda.synchronize()
    return q, k, v, o, l, o_ref, l_ref


def test_noalloc_split_matches_workspace_form():
    torch = torch_mod()
    orc = oracle.get()
    # first call: the library's partition for 272 query tiles (16 left over
    # after one round of 256, each cut in 16): 256 slots of the array
    q, k, v, o, l, o_ref, l_ref = _run_pair(torch, 1, 2048, 4096, 17, 64, 0, 520)
    assert torch.equal(o, o_ref) and torch.equal(l, l_ref), "first call differs from the workspace form"
    rows = np.arange(0, 2048, 37)
    ref_o, ref_l = orc.attention(q, k, v, rows=rows)
    check_out(to_np(o)[:, rows], ref_o, "bf16", "noalloc first call out (sampled rows)")
    check_lse(l.cpu().numpy()[:, :, rows], ref_l, "bf16", "noalloc first call lse (sampled rows)")
    # second call, smaller: every sweep cut in 4, 24 slots; the array still
    # holds the first call's partials, which must not leak into this result
    q, k, v, o, l, o_ref, l_ref = _run_pair(torch, 1, 200, 1000, 3, 128, 4, 530)
    assert torch.equal(o, o_ref) and torch.equal(l, l_ref), "second call differs from the workspace form"
    ref_o, ref_l = orc.attention(q, k, v)
    check_out(to_np(o), ref_o, "bf16", "noalloc second call out")
    check_lse(l.cpu().numpy(), ref_l, "bf16", "noalloc second call lse")


def test_noalloc_split_rejects_partitions_above_the_limit():
    torch = torch_mod()
    B, Nq, Nk, H, d = 1, 4096, 8192, 32, 128
    q = torch.zeros((B, Nq, H, d), device="cuda", dtype=torch.bfloat16)
    k = torch.zeros((B, Nk, H, d), device="cuda", dtype=torch.bfloat16)
    out = torch.full((B, Nq, H, d), 7.0, device="cuda", dtype=torch.bfloat16)
    # 32 x 32 query tiles, every sweep cut in 16: 16384 slots, about 1 GiB
    assert xd.split_workspace_bytes(q, Nk, 16) > _lib.lib().xdit_noalloc_scratch_bytes()
    with pytest.raises(xd.XditError) as e:
        xd.xdit_chunk_attn_split_noalloc(q, k, k, out, None, 16)
    assert e.value.code == -4
    torch.cuda.synchronize()
    assert torch.all(out == 7.0).item(), "a rejected call wrote its output"
