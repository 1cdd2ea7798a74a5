"""Moving seeded instances to the GPU and running the HIP path through the
C ABI (via the thin binding).  GPU-only; imported by ``-m gpu`` tests, the
smoke check and the benchmark."""
from __future__ import annotations

import numpy as np
import torch

import paper_2606_02964_amd as msa


def dev_bf16(bits: np.ndarray, device="cuda") -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(device).view(torch.bfloat16)


def bf16_to_f32(t: torch.Tensor) -> np.ndarray:
    return t.float().cpu().numpy()


class DeviceInstance:
    """Device copies of an instance's tensors (contiguous ABI layouts)."""

    def __init__(self, inst, device="cuda"):
        self.inst = inst
        self.q = dev_bf16(inst.q, device)
        self.k = dev_bf16(inst.k_cache, device)
        self.v = dev_bf16(inst.v_cache, device)
        self.bt = torch.from_numpy(np.ascontiguousarray(inst.block_table)).to(device)

    def shape(self, o_strides=None, q_strides=None):
        i = self.inst
        return msa.make_shape(i.num_seqs, i.num_q_heads, i.num_kv_heads, i.head_dim,
                              i.max_blocks_per_seq, int(self.k.shape[0]), i.scale,
                              o_strides=o_strides, q_strides=q_strides)

    def plan(self, **kw):
        i = self.inst
        return msa.msa_plan(self.shape(kw.pop("o_strides", None), kw.pop("q_strides", None)),
                            i.seq_kv_len, i.seg_indptr, i.seg_start, i.seg_len, **kw)


def run(dinst: DeviceInstance, plan=None, with_lse=True, sync=True, **plan_kw):
    """(o [total_q, Hq, d] bf16 tensor, lse or None, plan)."""
    i = dinst.inst
    if plan is None:
        plan = dinst.plan(**plan_kw)
    info = plan.info()
    o = torch.full((i.total_q, i.num_q_heads, i.head_dim), float("nan"), dtype=torch.bfloat16,
                   device=dinst.q.device)
    lse = (torch.full((i.total_q, i.num_q_heads), float("nan"), dtype=torch.float32,
                      device=dinst.q.device) if with_lse else None)
    ws = None
    if info["workspace_bytes"]:
        ws = torch.empty(info["workspace_bytes"], dtype=torch.uint8, device=dinst.q.device)
    msa.msa_forward(plan, dinst.q, dinst.k, dinst.v, dinst.bt, o, lse, ws)
    if sync:
        torch.cuda.synchronize()
    return o, lse, plan


def errors(gpu_o: np.ndarray, ref_o: np.ndarray):
    d = np.abs(gpu_o.astype(np.float64) - ref_o)
    return float(d.max()), float(d.mean())


# tolerance of the GPU path against the oracle (bf16 inputs, bf16 output):
# the stated bar for O
MAX_ABS = 1e-2
MEAN_ABS = 1e-3
# lse (natural log): the row sum adds softmax weights rounded to bf16, each
# within a relative 2^-9 of its exact value, so ln(l) moves by at most 2^-9;
# fp32 scores add well under 1e-4 at these magnitudes
LSE_ABS = 2.0 ** -9 + 1e-4
