"""Pins of the oracle's paged K/V append (CPU only).

The append stores every packed row's fresh key and value at the row's
absolute position in the paged cache (Sec. 4.1: all segments' tokens run
through one forward pass; Sec. 5.3: the cache is PagedAttention's).  The
oracle does that element by element; the pins reach the same caches by other
routes:

* bulk layout: the generator's whole-block reshape/transpose of the logical
  K/V with the fresh rows substituted at their positions;
* attention round trip: dense causal SDPA on the substituted logical K/V
  equals the attention oracle on the appended caches (the two caches'
  layouts must agree with the attention's addressing);
* slots without a valid block-table entry are skipped and nothing else moves.

Plausible mistakes planted in a copy of the oracle source fail these pins.
"""
import copy
import os
import subprocess

import numpy as np
import pytest

import oracle
import workloads
from msa_pins import dense_reference, positions_of

CASES = [
    # seed, B, Hq, Hkv, d, max_len, max_segs
    (31, 3, 4, 2, 64, 200, 5),
    (32, 2, 8, 2, 128, 260, 3),
    (33, 4, 6, 3, 24, 90, 4),
    (34, 1, 8, 8, 64, 400, 7),
]


def _case(case):
    seed, B, Hq, Hkv, d, max_len, max_segs = case
    inst = workloads.make_random(seed, num_seqs=B, num_q_heads=Hq, num_kv_heads=Hkv,
                                 head_dim=d, max_len=max_len, max_segs=max_segs,
                                 keep_logical=True)
    kn, vn = workloads.make_fresh_kv(inst, seed + 1000)
    return inst, kn, vn


def _substituted_logical(inst, kn, vn):
    seq, pos = positions_of(inst)
    k_log = [x.copy() for x in inst.k_logical]
    v_log = [x.copy() for x in inst.v_logical]
    for r, (b, p) in enumerate(zip(seq, pos)):
        k_log[b][p] = kn[r]
        v_log[b][p] = vn[r]
    return k_log, v_log


def _bulk_expected(inst, kn, vn):
    k_log, v_log = _substituted_logical(inst, kn, vn)
    return workloads.layout_cache(inst.block_table, inst.num_blocks, k_log, v_log,
                                  inst.block_size)


@pytest.mark.parametrize("case", CASES)
def test_append_matches_bulk_layout(case):
    inst, kn, vn = _case(case)
    k, v = oracle.kv_append(inst, kn, vn)
    ek, ev = _bulk_expected(inst, kn, vn)
    assert np.array_equal(k, ek)
    assert np.array_equal(v, ev)
    # the instance's own caches are untouched
    k0, v0 = workloads.layout_cache(inst.block_table, inst.num_blocks, inst.k_logical,
                                    inst.v_logical, inst.block_size)
    assert np.array_equal(inst.k_cache, k0) and np.array_equal(inst.v_cache, v0)


@pytest.mark.parametrize("case", CASES[:2])
def test_append_then_attention_matches_dense(case):
    inst, kn, vn = _case(case)
    k, v = oracle.kv_append(inst, kn, vn)
    after = copy.copy(inst)
    after.k_cache, after.v_cache = k, v
    after.k_logical, after.v_logical = _substituted_logical(inst, kn, vn)
    o, lse = oracle.forward(after)
    ro, rlse = dense_reference(after)
    np.testing.assert_allclose(o, ro, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, rlse, rtol=0, atol=1e-12)


def test_append_skips_rows_without_a_block():
    inst, kn, vn = _case(CASES[0])
    seq, pos = positions_of(inst)
    bt = inst.block_table.copy()
    # drop the block of the first row of sequence 0 and of the last row
    dropped = {(int(seq[0]), int(pos[0]) // 16), (int(seq[-1]), int(pos[-1]) // 16)}
    for (b, jb) in dropped:
        bt[b, jb] = -1
    cut = copy.copy(inst)
    cut.block_table = bt
    k, v = oracle.kv_append(cut, kn, vn)
    # expected: substitute only rows whose block survived
    k_log = [x.copy() for x in inst.k_logical]
    v_log = [x.copy() for x in inst.v_logical]
    for r, (b, p) in enumerate(zip(seq, pos)):
        if (int(b), int(p) // 16) not in dropped:
            k_log[b][p] = kn[r]
            v_log[b][p] = vn[r]
    ek, ev = workloads.layout_cache(inst.block_table, inst.num_blocks, k_log, v_log)
    assert np.array_equal(k, ek) and np.array_equal(v, ev)


def test_append_no_rows_is_identity():
    inst = workloads.make_layout(7, [100, 40], [[], []], 4, 2, 64)
    kn = np.zeros((0, 2, 64), np.uint16)
    k, v = oracle.kv_append(inst, kn, kn)
    assert np.array_equal(k, inst.k_cache) and np.array_equal(v, inst.v_cache)


def test_append_rejects_bad_segments():
    inst, kn, vn = _case(CASES[0])
    bad = copy.copy(inst)
    bad.seg_start = inst.seg_start.copy()
    bad.seg_start[0] = inst.seq_kv_len[0]  # past the context
    with pytest.raises(ValueError):
        oracle.kv_append(bad, kn, vn)


SRC = os.path.join(os.path.dirname(oracle.__file__), "msa_oracle.c")

MUTANTS = {
    "v_written_token_major": ("c * v_stride_dim + off] =", "off * v_stride_dim + c] ="),
    "offset_off_by_one": ("const int32_t off = p % block_size;",
                          "const int32_t off = (p + 1) % block_size;"),
    "block_of_next_sequence": ("block_table[(int64_t)b * max_blocks_per_seq + p / block_size]",
                               "block_table[(int64_t)((b + 1) % num_seqs) * max_blocks_per_seq"
                               " + p / block_size]"),
    "kv_heads_swapped": ("k_new[r * kn_stride_tok + g * kn_stride_head + c]",
                         "k_new[r * kn_stride_tok + (num_kv_heads - 1 - g) * kn_stride_head + c]"),
    "row_counter_per_sequence": ("  int64_t r = 0;\n  for (int32_t b = 0; b < num_seqs; ++b)\n"
                                 "    for (int32_t s = seg_indptr[b];",
                                 "  int64_t r = 0;\n  for (int32_t b = 0; b < num_seqs; ++b, r = 0)\n"
                                 "    for (int32_t s = seg_indptr[b];"),
}


def _build(tmp_path, name, src):
    c = tmp_path / f"{name}.c"
    so = tmp_path / f"{name}.so"
    c.write_text(src)
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
                           "-pthread", str(c), "-o", str(so), "-lm"])
    return oracle.load_library(str(so))


def _pins_pass(lib) -> bool:
    for case in CASES:
        inst, kn, vn = _case(case)
        k, v = oracle.kv_append(inst, kn, vn, lib=lib)
        ek, ev = _bulk_expected(inst, kn, vn)
        if not (np.array_equal(k, ek) and np.array_equal(v, ev)):
            return False
    return True


def test_unmutated_append_copy_passes(tmp_path):
    assert _pins_pass(_build(tmp_path, "same", open(SRC).read()))


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_append_mutant_is_caught(tmp_path, name):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation anchor for {name} not found exactly once"
    assert not _pins_pass(_build(tmp_path, name, src.replace(old, new)))
