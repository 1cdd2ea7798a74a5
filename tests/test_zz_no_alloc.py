"""msa_forward_noalloc, the entry point for callers that cannot allocate,
against msa_forward on the same inputs (GPU only).

Its workspace is the library's per-device scratch array, so the outputs
must be bit-identical to msa_forward's with a workspace of its own, and
within the oracle bar.  Two calls in a row share the array, the second on a
smaller input; plans whose workspace exceeds the array are refused before
anything is launched.
"""
import numpy as np
import pytest
import torch

import workloads

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # collected on a CPU-only host with -m gpu
    pytest.skip("no GPU visible", allow_module_level=True)

from gpu_helpers import DeviceInstance, bf16_to_f32, check_o, run  # noqa: E402
import paper_2606_02964_amd as msa  # noqa: E402


def _outputs(inst):
    o = torch.full((inst.total_q, inst.num_q_heads, inst.head_dim), float("nan"), dtype=torch.bfloat16,
                   device="cuda")
    lse = torch.full((inst.total_q, inst.num_q_heads), float("nan"), dtype=torch.float32, device="cuda")
    return o, lse


@pytest.mark.parametrize("tile", [0, msa.MSA_PLAN_TILE_ROWS_32])
def test_noalloc_matches_forward_on_two_calls_in_a_row(oracle_lib, tile):
    big = workloads.make_random(401, num_seqs=3, num_q_heads=16, num_kv_heads=4, head_dim=128,
                                min_len=600, max_len=2000, max_segs=5, keep_logical=False)
    small = workloads.make_random(402, num_seqs=2, num_q_heads=8, num_kv_heads=2, head_dim=64,
                                  min_len=100, max_len=700, max_segs=3, keep_logical=False)
    cases = []
    for inst, split in ((big, 512), (small, 64)):
        d = DeviceInstance(inst)
        plan = d.plan(kv_split_tokens=split, flags=tile)
        info = plan.info()
        assert info["num_merge"] > 0 and 0 < info["workspace_bytes"] <= msa.MSA_NOALLOC_WORKSPACE_BYTES
        o_ref, l_ref, _ = run(d, plan=plan)
        cases.append((inst, d, plan, info, o_ref, l_ref))
    assert cases[1][3]["workspace_bytes"] < cases[0][3]["workspace_bytes"]
    outs = []
    for inst, d, plan, _, _, _ in cases:   # the two no-allocation calls back to back
        o, lse = _outputs(inst)
        msa.msa_forward_noalloc(plan, d.q, d.k, d.v, d.bt, o, lse)
        outs.append((o, lse))
    torch.cuda.synchronize()
    for (inst, _, _, _, o_ref, l_ref), (o, lse) in zip(cases, outs):
        assert torch.equal(o.view(torch.int16), o_ref.view(torch.int16))
        assert torch.equal(lse.view(torch.int32), l_ref.view(torch.int32))
        ro, rl = oracle_lib.forward(inst)
        check_o(bf16_to_f32(o), ro, lse.cpu().numpy(), rl)


def test_noalloc_without_workspace(oracle_lib):
    """A plan with no key splits needs no workspace: same outputs."""
    inst = workloads.make_config(1)
    d = DeviceInstance(inst)
    plan = d.plan(flags=msa.MSA_PLAN_NO_AUTO_SPLIT)
    assert plan.info()["workspace_bytes"] == 0
    o_ref, l_ref, _ = run(d, plan=plan)
    o, lse = _outputs(inst)
    msa.msa_forward_noalloc(plan, d.q, d.k, d.v, d.bt, o, lse)
    torch.cuda.synchronize()
    assert torch.equal(o.view(torch.int16), o_ref.view(torch.int16))
    assert torch.equal(lse.view(torch.int32), l_ref.view(torch.int32))


def test_noalloc_refuses_a_workspace_beyond_its_array():
    """2048 partial slots of 256 rows (270 MB) exceed the 64 MiB array: the
    call is refused and writes nothing.  The tensors are real and sized for
    the plan, so nothing here could read out of bounds either way."""
    L = 32768
    inst = workloads.make_layout(403, [L], [[(L - 512, 512)]], 32, 8, 128, keep_logical=False)
    d = DeviceInstance(inst)
    plan = d.plan(kv_split_tokens=1024, flags=msa.MSA_PLAN_TILE_ROWS_256)
    assert plan.info()["workspace_bytes"] > msa.MSA_NOALLOC_WORKSPACE_BYTES
    o, lse = _outputs(inst)
    with pytest.raises(msa.MsaError) as e:
        msa.msa_forward_noalloc(plan, d.q, d.k, d.v, d.bt, o, lse)
    assert e.value.status == msa.MSA_ERR_UNSUPPORTED
    assert "scratch" in msa.msa_last_error()
    torch.cuda.synchronize()
    assert torch.isnan(o.float()).all().item() and torch.isnan(lse).all().item()
