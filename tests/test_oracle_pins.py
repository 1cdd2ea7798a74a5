"""Pins of the CPU oracle against things other than itself (CPU only).

* brute force: dense causal attention (library SDPA, float64) on the logical
  K/V, never touching the paged cache (Sec. 2.1 Eq. 1, Sec. 4.1 Eq. 2);
* special cases the paper names: a single segment [0, L) is plain causal
  prefill (FlashAttention's case), a single last token is decode over the
  whole context (PagedAttention's case) (Sec. 5.3);
* closed forms: a position-0 row returns v_0 exactly; a zero query averages
  v_0..v_p with lse = ln(p+1); identical keys give uniform weights;
* invariances: physical block permutation, splitting a segment into two
  adjacent ones, causality of Eq. 2 (keys after a segment do not affect it),
  independence of sequences, GQA == MHA with repeated K/V heads.
"""
import copy

import numpy as np
import pytest

import workloads
from msa_pins import dense_reference, positions_of, repermute, split_segments, to_f64

RANDOM_CASES = [
    # seed, B, Hq, Hkv, d, max_len, max_segs
    (1, 2, 4, 4, 64, 300, 4),
    (2, 3, 4, 2, 64, 200, 5),
    (3, 2, 8, 2, 128, 260, 3),
    (4, 1, 8, 1, 128, 400, 6),
    (5, 3, 6, 3, 24, 90, 4),
    (6, 4, 2, 1, 64, 33, 3),
]


def _rand(case, **kw):
    seed, B, Hq, Hkv, d, max_len, max_segs = case
    return workloads.make_random(seed, num_seqs=B, num_q_heads=Hq, num_kv_heads=Hkv,
                                 head_dim=d, max_len=max_len, max_segs=max_segs, **kw)


@pytest.mark.parametrize("case", RANDOM_CASES)
def test_oracle_matches_dense_causal_sdpa(oracle_lib, case):
    inst = _rand(case)
    o, lse = oracle_lib.forward(inst)
    ro, rlse = dense_reference(inst)
    assert inst.total_q > 0
    np.testing.assert_allclose(o, ro, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, rlse, rtol=0, atol=1e-12)


@pytest.mark.parametrize("qscale", [4.0, 16.0])
def test_oracle_matches_dense_on_peaky_logits(oracle_lib, qscale):
    """Q scaled by a power of two (exact in bf16): scores spread over many
    log2 units, weights sit on a few keys, and the max subtraction and the
    float64 sums still give the dense result."""
    inst = _rand(RANDOM_CASES[2], keep_logical=True)
    inst.q = workloads.f32_to_bf16_bits(workloads.bf16_bits_to_f32(inst.q) * np.float32(qscale))
    o, lse = oracle_lib.forward(inst)
    ro, rlse = dense_reference(inst)
    np.testing.assert_allclose(o, ro, rtol=0, atol=1e-11)
    np.testing.assert_allclose(lse, rlse, rtol=0, atol=1e-10)


def test_oracle_config1_matches_dense(oracle_lib):
    inst = workloads.make_config(1, keep_logical=True)
    o, lse = oracle_lib.forward(inst)
    ro, rlse = dense_reference(inst)
    np.testing.assert_allclose(o, ro, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, rlse, rtol=0, atol=1e-12)


def test_prefill_special_case(oracle_lib):
    """One segment [0, L): every row of the sequence is a query -> plain causal
    prefill attention over the whole sequence."""
    import torch
    L, Hq, Hkv, d = 77, 4, 2, 64
    inst = workloads.make_layout(21, [L], [[(0, L)]], Hq, Hkv, d)
    o, _ = oracle_lib.forward(inst)
    q = to_f64(inst.q).permute(1, 0, 2)[None]
    k = to_f64(inst.k_logical[0]).repeat_interleave(Hq // Hkv, dim=1).permute(1, 0, 2)[None]
    v = to_f64(inst.v_logical[0]).repeat_interleave(Hq // Hkv, dim=1).permute(1, 0, 2)[None]
    ref = torch.nn.functional.scaled_dot_product_attention(q, k, v, is_causal=True,
                                                           scale=inst.scale)[0].permute(1, 0, 2)
    np.testing.assert_allclose(o, ref.numpy(), rtol=0, atol=1e-12)


def test_decode_special_case(oracle_lib):
    """One segment [L-1, L): one query attending to all L keys, no mask."""
    import torch
    L, Hq, Hkv, d = 203, 8, 2, 128
    inst = workloads.make_layout(22, [L], [[(L - 1, 1)]], Hq, Hkv, d)
    o, _ = oracle_lib.forward(inst)
    q = to_f64(inst.q).permute(1, 0, 2)[None]                       # [1, Hq, 1, d]
    k = to_f64(inst.k_logical[0]).repeat_interleave(Hq // Hkv, dim=1).permute(1, 0, 2)[None]
    v = to_f64(inst.v_logical[0]).repeat_interleave(Hq // Hkv, dim=1).permute(1, 0, 2)[None]
    ref = torch.nn.functional.scaled_dot_product_attention(q, k, v, is_causal=False,
                                                           scale=inst.scale)[0].permute(1, 0, 2)
    np.testing.assert_allclose(o, ref.numpy(), rtol=0, atol=1e-12)


def test_position_zero_row_is_v0(oracle_lib):
    """Only key 0 is visible: weight 1, o = v_0 exactly, lse = scale * q.k_0."""
    Hq, Hkv, d = 4, 2, 64
    inst = workloads.make_layout(23, [40, 40], [[(0, 3), (20, 2)], [(0, 1)]], Hq, Hkv, d)
    o, lse = oracle_lib.forward(inst)
    q = to_f64(inst.q).numpy()
    for r in (0, 5):  # row 0 of sequence 0 and of sequence 1, both at position 0
        b = 0 if r == 0 else 1
        for h in range(Hq):
            g = h // (Hq // Hkv)
            v0 = to_f64(inst.v_logical[b][0, g]).numpy()
            k0 = to_f64(inst.k_logical[b][0, g]).numpy()
            assert np.array_equal(o[r, h], v0)
            assert abs(lse[r, h] - inst.scale * float(np.dot(q[r, h], k0))) < 1e-12


def test_zero_query_averages_visible_values(oracle_lib):
    """q = 0: all visible scores equal -> o = mean(v_0..v_p), lse = ln(p+1)."""
    Hq, Hkv, d = 4, 1, 64
    inst = workloads.make_layout(24, [130], [[(5, 3), (64, 17), (129, 1)]], Hq, Hkv, d)
    inst.q = np.zeros_like(inst.q)
    o, lse = oracle_lib.forward(inst)
    _, pos = positions_of(inst)
    v = to_f64(inst.v_logical[0]).numpy()  # [L, 1, d]
    for r, p in enumerate(pos):
        for h in range(Hq):
            np.testing.assert_allclose(o[r, h], v[:p + 1, 0].mean(axis=0), rtol=0, atol=1e-13)
            assert abs(lse[r, h] - np.log(p + 1)) < 1e-13


def test_identical_keys_give_uniform_weights(oracle_lib):
    """All keys equal k: weights uniform -> o = mean(v_0..v_p) and
    lse = scale * q.k + ln(p+1)."""
    Hq, Hkv, d = 2, 2, 64
    inst = workloads.make_layout(25, [64], [[(10, 5), (40, 3)]], Hq, Hkv, d,
                                 permute_blocks=False)
    inst.k_cache[:] = inst.k_cache[0:1, :, 0:1, :]   # every key = key 0 of its head
    o, lse = oracle_lib.forward(inst)
    _, pos = positions_of(inst)
    q = to_f64(inst.q).numpy()
    k0 = to_f64(inst.k_cache[0, :, 0, :]).numpy()     # [Hkv, d]
    v = to_f64(inst.v_logical[0]).numpy()
    for r, p in enumerate(pos):
        for h in range(Hq):
            np.testing.assert_allclose(o[r, h], v[:p + 1, h].mean(axis=0), rtol=0, atol=1e-13)
            expect = inst.scale * float(np.dot(q[r, h], k0[h])) + np.log(p + 1)
            assert abs(lse[r, h] - expect) < 1e-12


@pytest.mark.parametrize("case", RANDOM_CASES[:4])
def test_physical_permutation_is_bitwise_invariant(oracle_lib, case):
    inst = _rand(case, extra_blocks=3)
    o1, l1 = oracle_lib.forward(inst)
    o2, l2 = oracle_lib.forward(repermute(inst, 99))
    assert np.array_equal(o1, o2) and np.array_equal(l1, l2)


@pytest.mark.parametrize("case", RANDOM_CASES[:4])
def test_segment_split_is_bitwise_invariant(oracle_lib, case):
    inst = _rand(case)
    o1, l1 = oracle_lib.forward(inst)
    o2, l2 = oracle_lib.forward(split_segments(inst, 7))
    assert np.array_equal(o1, o2) and np.array_equal(l1, l2)


def test_eq2_causality_later_keys_do_not_matter(oracle_lib):
    """Two segments: the first segment's output does not depend on K/V at
    positions after its end (its queries attend only to their prefix), the
    second segment's does (Sec. 4.1, Eq. 2)."""
    Hq, Hkv, d, L = 4, 2, 64, 192
    inst = workloads.make_layout(26, [L], [[(40, 24), (150, 20)]], Hq, Hkv, d)
    o1, l1 = oracle_lib.forward(inst)
    mod = copy.copy(inst)
    mod.k_cache = inst.k_cache.copy()
    mod.v_cache = inst.v_cache.copy()
    rng = np.random.Generator(np.random.PCG64(5))
    for j in range(64, L):  # every position after the first segment's end
        blk = inst.block_table[0, j // 16]
        mod.k_cache[blk, :, j % 16, :] = workloads.f32_to_bf16_bits(
            rng.standard_normal((Hkv, d), dtype=np.float32))
        mod.v_cache[blk, :, :, j % 16] = workloads.f32_to_bf16_bits(
            rng.standard_normal((Hkv, d), dtype=np.float32))
    o2, l2 = oracle_lib.forward(mod)
    assert np.array_equal(o1[:24], o2[:24]) and np.array_equal(l1[:24], l2[:24])
    assert np.abs(o1[24:] - o2[24:]).max() > 1e-3


def test_sequences_are_independent(oracle_lib):
    inst = workloads.make_random(31, num_seqs=3, num_q_heads=4, num_kv_heads=2, head_dim=64,
                                 min_len=40, max_len=120, max_segs=3)
    seq, _ = positions_of(inst)
    if not (seq == 1).any():
        pytest.skip("layout has no rows in sequence 1")
    o1, _ = oracle_lib.forward(inst)
    mod = copy.copy(inst)
    mod.k_cache = inst.k_cache.copy()
    mod.v_cache = inst.v_cache.copy()
    for b in (0, 2):
        nb = -(-int(inst.seq_kv_len[b]) // 16)
        for blk in inst.block_table[b, :nb]:
            mod.k_cache[blk] ^= np.uint16(0x0040)
            mod.v_cache[blk] ^= np.uint16(0x0040)
    o2, _ = oracle_lib.forward(mod)
    assert np.array_equal(o1[seq == 1], o2[seq == 1])


def test_gqa_equals_mha_with_repeated_kv_heads(oracle_lib):
    case = (41, 2, 8, 2, 64, 150, 3)
    inst = _rand(case)
    G = inst.num_q_heads // inst.num_kv_heads
    mha = copy.copy(inst)
    mha.num_kv_heads = inst.num_q_heads
    mha.k_cache = np.repeat(inst.k_cache, G, axis=1)   # kv head h -> original h // G
    mha.v_cache = np.repeat(inst.v_cache, G, axis=1)
    o1, l1 = oracle_lib.forward(inst)
    o2, l2 = oracle_lib.forward(mha)
    assert np.array_equal(o1, o2) and np.array_equal(l1, l2)


def test_item_selection_and_threads_are_bitwise_consistent(oracle_lib):
    inst = _rand(RANDOM_CASES[2])
    o, lse = oracle_lib.forward(inst, num_threads=1)
    o8, lse8 = oracle_lib.forward(inst, num_threads=8)
    assert np.array_equal(o, o8) and np.array_equal(lse, lse8)
    rng = np.random.Generator(np.random.PCG64(3))
    rows = rng.integers(0, inst.total_q, size=50)
    heads = rng.integers(0, inst.num_q_heads, size=50)
    so, sl = oracle_lib.forward(inst, rows=rows, heads=heads, num_threads=3)
    assert np.array_equal(so, o[rows, heads]) and np.array_equal(sl, lse[rows, heads])


@pytest.mark.parametrize("bad", ["overlap", "unsorted", "empty", "past_end", "missing_block"])
def test_oracle_rejects_inputs_outside_the_definition(oracle_lib, bad):
    inst = workloads.make_layout(51, [100], [[(10, 20), (50, 10)]], 2, 1, 64)
    if bad == "overlap":
        inst.seg_start = np.asarray([10, 25], np.int32)
    elif bad == "unsorted":
        inst.seg_start = np.asarray([50, 10], np.int32)
        inst.seg_len = np.asarray([10, 20], np.int32)
    elif bad == "empty":
        inst.seg_len = np.asarray([20, 0], np.int32)
        inst.q = inst.q[:20]
    elif bad == "past_end":
        inst.seg_start = np.asarray([10, 95], np.int32)
    elif bad == "missing_block":
        inst.block_table = inst.block_table.copy()
        inst.block_table[0, 2] = -1
    with pytest.raises(ValueError):
        oracle_lib.forward(inst)
