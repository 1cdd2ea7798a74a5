"""Parity of the HIP paged K/V append (through the C ABI) with the CPU oracle.

The append is byte work, so the bar is bit-exact: after ``msa_kv_append``
both whole caches (every block, every head, every slot, also blocks no row
touches) equal the oracle's, on random layouts, on the named workloads at
full size, with strided sources, with block-table entries that have no slot,
and as the first half of a layer (append, then attention over the new cache).
"""
import copy

import numpy as np
import pytest
import torch

import workloads

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # collected on a CPU-only host with -m gpu
    pytest.skip("no GPU visible", allow_module_level=True)

from gpu_helpers import (LSE_ABS, MAX_ABS, MEAN_ABS, DeviceInstance, bf16_to_f32, check_o,  # noqa: E402
                         dev_bf16, errors, run)
import paper_2606_02964_amd as msa  # noqa: E402


def bits(t: torch.Tensor) -> np.ndarray:
    return t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def append_on_gpu(inst, kn, vn, bt=None, fused=False):
    """Device caches after msa_kv_append (host bf16 bits)."""
    d = DeviceInstance(inst)
    if bt is not None:
        d.bt = torch.from_numpy(np.ascontiguousarray(bt)).cuda()
    plan = d.plan()
    if fused:
        # fresh K/V as views into one [T, (Hq + 2 Hkv) * d] projection output
        T, Hkv, hd = kn.shape
        Hq = inst.num_q_heads
        qkv = torch.zeros((T, (Hq + 2 * Hkv) * hd), dtype=torch.bfloat16, device="cuda")
        qkv[:, Hq * hd:(Hq + Hkv) * hd] = dev_bf16(kn).reshape(T, Hkv * hd)
        qkv[:, (Hq + Hkv) * hd:] = dev_bf16(vn).reshape(T, Hkv * hd)
        k_new = qkv[:, Hq * hd:(Hq + Hkv) * hd].view(T, Hkv, hd)
        v_new = qkv[:, (Hq + Hkv) * hd:].view(T, Hkv, hd)
        assert k_new.stride() == ((Hq + 2 * Hkv) * hd, hd, 1)
    else:
        k_new, v_new = dev_bf16(kn), dev_bf16(vn)
    msa.msa_kv_append(plan, k_new, v_new, d.bt, d.k, d.v)
    torch.cuda.synchronize()
    return bits(d.k), bits(d.v), d


def check_bitexact(inst, kn, vn, oracle_lib, **kw):
    gk, gv, d = append_on_gpu(inst, kn, vn, **kw)
    ek, ev = oracle_lib.kv_append(inst, kn, vn)
    assert np.array_equal(gk, ek), "K cache differs from the oracle's"
    assert np.array_equal(gv, ev), "V cache differs from the oracle's"
    return d


RANDOM = [
    # seed, B, Hq, Hkv, d, max_len, max_segs
    (201, 3, 4, 4, 64, 700, 5),
    (202, 4, 32, 8, 128, 1500, 8),
    (203, 2, 24, 12, 128, 400, 3),   # 12 KV heads: two head passes
    (204, 5, 8, 1, 64, 333, 9),
    (205, 6, 2, 2, 128, 70, 3),      # short sequences, ragged last blocks
    (206, 3, 16, 16, 64, 900, 12),   # many short segments at odd offsets
]


@pytest.mark.parametrize("case", RANDOM)
def test_append_random_layouts_bitexact(oracle_lib, case):
    seed, B, Hq, Hkv, d, max_len, max_segs = case
    inst = workloads.make_random(seed, num_seqs=B, num_q_heads=Hq, num_kv_heads=Hkv,
                                 head_dim=d, max_len=max_len, max_segs=max_segs,
                                 keep_logical=False)
    kn, vn = workloads.make_fresh_kv(inst, seed + 7)
    check_bitexact(inst, kn, vn, oracle_lib)


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_append_named_workloads_bitexact(oracle_lib, cfg):
    inst = workloads.make_config(cfg)
    kn, vn = workloads.make_fresh_kv(inst, 1000 + cfg)
    check_bitexact(inst, kn, vn, oracle_lib)


def test_append_decode_rows_bitexact(oracle_lib):
    """One row per sequence at arbitrary offsets: no 8-row runs at all."""
    inst = workloads.make_config(5, decode_only=True)
    kn, vn = workloads.make_fresh_kv(inst, 77)
    check_bitexact(inst, kn, vn, oracle_lib)


def test_append_from_fused_projection_views(oracle_lib):
    inst = workloads.make_random(211, num_seqs=3, num_q_heads=8, num_kv_heads=2, head_dim=128,
                                 max_len=600, max_segs=4, keep_logical=False)
    kn, vn = workloads.make_fresh_kv(inst, 5)
    check_bitexact(inst, kn, vn, oracle_lib, fused=True)


def test_append_untouched_blocks_and_rows_without_slot(oracle_lib):
    """Blocks nobody references keep their bytes; rows whose block-table entry
    is -1 or num_blocks write nothing (the kernel's bounds check)."""
    base = workloads.make_layout(212, [300, 170, 64], [[(5, 40), (100, 3)], [(16, 16), (160, 10)],
                                                       [(0, 64)]], 8, 2, 64, extra_blocks=6)
    inst = copy.copy(base)
    inst.k_cache = base.k_cache.copy()
    inst.v_cache = base.v_cache.copy()
    extra = np.arange(base.num_blocks - 6, base.num_blocks)
    inst.k_cache[extra] = 0x7FC0  # NaN bit patterns in unreferenced blocks
    inst.v_cache[extra] = 0x7FC0
    bt = inst.block_table.copy()
    bt[0, 100 // 16] = -1
    bt[1, 160 // 16] = inst.num_blocks
    cut = copy.copy(inst)
    cut.block_table = bt
    kn, vn = workloads.make_fresh_kv(inst, 9)
    gk, gv, _ = append_on_gpu(inst, kn, vn, bt=bt)
    ek, ev = oracle_lib.kv_append(cut, kn, vn)
    assert np.array_equal(gk, ek) and np.array_equal(gv, ev)
    assert np.array_equal(gk[extra], inst.k_cache[extra])
    assert np.array_equal(gv[extra], inst.v_cache[extra])


def test_append_empty_plan_is_noop():
    inst = workloads.make_layout(213, [64, 32], [[], []], 4, 2, 64)
    d = DeviceInstance(inst)
    plan = d.plan()
    k0, v0 = bits(d.k), bits(d.v)
    empty = torch.empty((0, 2, 64), dtype=torch.bfloat16, device="cuda")
    msa.msa_kv_append(plan, empty, empty, d.bt, d.k, d.v)
    torch.cuda.synchronize()
    assert np.array_equal(bits(d.k), k0) and np.array_equal(bits(d.v), v0)


@pytest.mark.parametrize("cfg_or_case", [1, (214, 3, 8, 2, 128, 900, 5)])
def test_append_then_attention(oracle_lib, cfg_or_case):
    """One layer's cache write then MSA, against the oracle on the oracle's
    appended caches."""
    if isinstance(cfg_or_case, int):
        inst = workloads.make_config(cfg_or_case)
    else:
        seed, B, Hq, Hkv, d, max_len, max_segs = cfg_or_case
        inst = workloads.make_random(seed, num_seqs=B, num_q_heads=Hq, num_kv_heads=Hkv,
                                     head_dim=d, max_len=max_len, max_segs=max_segs,
                                     keep_logical=False)
    kn, vn = workloads.make_fresh_kv(inst, 31)
    gk, gv, dinst = append_on_gpu(inst, kn, vn)
    o, lse, _ = run(dinst)
    after = copy.copy(inst)
    after.k_cache, after.v_cache = oracle_lib.kv_append(inst, kn, vn)
    assert np.array_equal(gk, after.k_cache) and np.array_equal(gv, after.v_cache)
    ro, rl = oracle_lib.forward(after)
    check_o(bf16_to_f32(o), ro)
    assert float(np.abs(lse.cpu().numpy().astype(np.float64) - rl).max()) <= LSE_ABS
