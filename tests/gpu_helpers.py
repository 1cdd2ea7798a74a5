"""Moving seeded instances to the GPU and running the HIP path through the
C ABI (via the thin binding).  GPU-only; imported by the ``-m gpu`` tests."""
from __future__ import annotations

import json
import os

import numpy as np
import torch

import paper_2606_02964_amd as msa
from tolerance import LSE_ABS, MAX_ABS, MEAN_ABS, errors, raw_max_abs  # noqa: F401  (re-exported)


def log_parity(**fields) -> None:
    """Append one JSON line of parity figures (with the running test's id)
    to the file named by MSA_PARITY_LOG, if set."""
    path = os.environ.get("MSA_PARITY_LOG")
    if not path:
        return
    fields["test"] = os.environ.get("PYTEST_CURRENT_TEST", "").split(" ")[0]
    with open(path, "a") as f:
        f.write(json.dumps(fields) + "\n")


def check_o(go: np.ndarray, ro: np.ndarray, lse=None, rl=None, lse_tol: float = LSE_ABS) -> None:
    """The O bar (max-abs per ``tolerance.py``, mean-abs) and, if given, the
    lse bar; the plain max-abs over every element is logged beside them."""
    go = np.asarray(go, dtype=np.float32)
    mx, mean = errors(go, ro)
    raw = raw_max_abs(go, ro)
    lerr = None
    if lse is not None:
        lerr = float(np.abs(np.asarray(lse, dtype=np.float64) - rl).max()) if np.size(rl) else 0.0
    log_parity(elements=int(go.size), bar_max=mx, plain_max=raw, mean=mean, lse_max=lerr)
    assert np.isfinite(go).all(), "some outputs are not finite"
    assert mx <= MAX_ABS and mean <= MEAN_ABS, (mx, mean, raw)
    if lerr is not None:
        assert lerr <= lse_tol, lerr


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

