"""The fused-kernel comparison (Sec. 6.3, Fig. ablation-fused) computes the
same thing three ways; the outputs must agree.

A suffix-cached request (evicted head + 128 new tokens) run as one fused MSA
launch and as one launch per segment (each launch holding that segment of
every request) gives bit-identical rows: a row's arithmetic does not depend
on which other rows share its tile (steps past a row's position add exact
zeros).  The fused result also matches the oracle.
"""
import numpy as np
import pytest
import torch

import workloads

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # collected on a CPU-only host with -m gpu
    pytest.skip("no GPU visible", allow_module_level=True)

from gpu_helpers import (LSE_ABS, MAX_ABS, MEAN_ABS, DeviceInstance, bf16_to_f32, check_o,  # noqa: E402
                         errors, run)
import paper_2606_02964_amd as msa  # noqa: E402


@pytest.mark.parametrize("ctx,batch,cached", [(1024, 2, 384), (1024, 3, 0), (2048, 2, 1280),
                                              (1024, 2, 896)])
def test_fused_equals_per_segment_launches(oracle_lib, ctx, batch, cached):
    segs = workloads.fused_ablation_layout(ctx, cached, "suffix")
    inst = workloads.make_layout(900 + ctx + batch + cached, [ctx] * batch, [segs] * batch,
                                 32, 8, 128, keep_logical=False)
    dinst = DeviceInstance(inst)
    o_fused, lse_fused, _ = run(dinst)
    # packed rows of segment k of every request
    nseg = len(segs)
    offs = np.cumsum([0] + [n for (_, n) in segs])
    for k, (st, n) in enumerate(segs):
        idx = np.concatenate([b * offs[-1] + np.arange(offs[k], offs[k] + n) for b in range(batch)])
        idx_t = torch.from_numpy(idx).cuda()
        q_k = dinst.q[idx_t].contiguous()
        shape = dinst.shape()
        plan = msa.msa_plan(shape, inst.seq_kv_len, np.arange(batch + 1, dtype=np.int32),
                            [st] * batch, [n] * batch)
        o_k = torch.full_like(q_k, float("nan"))
        lse_k = torch.full((idx.size, 32), float("nan"), dtype=torch.float32, device="cuda")
        info = plan.info()
        ws = (torch.empty(info["workspace_bytes"], dtype=torch.uint8, device="cuda")
              if info["workspace_bytes"] else None)
        msa.msa_forward(plan, q_k, dinst.k, dinst.v, dinst.bt, o_k, lse_k, ws)
        torch.cuda.synchronize()
        assert torch.equal(o_k.view(torch.int16), o_fused[idx_t].view(torch.int16)), f"segment {k}"
        assert torch.equal(lse_k, lse_fused[idx_t]), f"segment {k} lse"
    assert nseg == (1 if cached == ctx - 128 else 2)
    # and the fused launch against the oracle on a sample of rows
    rng = np.random.default_rng(ctx + cached)
    rows = rng.integers(0, inst.total_q, 96)
    heads = rng.integers(0, 32, 96)
    ro, rl = oracle_lib.forward(inst, rows=rows, heads=heads)
    go = bf16_to_f32(o_fused)[rows, heads]
    check_o(go, ro)
    gl = lse_fused.cpu().numpy()[rows, heads].astype(np.float64)
    assert float(np.abs(gl - rl).max()) <= LSE_ABS
