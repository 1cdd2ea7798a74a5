"""Parity of the HIP path (through the C ABI) with the CPU oracle on MI355X.

Bar (bf16 inputs, bf16 output): max-abs <= 1e-2 (plain |stored - ref| where
|ref| < 4; above, where half a bf16 spacing exceeds the bar, on the value
before the output's own rounding, see ``tolerance.py``) and mean-abs <= 1e-3
over every compared element; lse within 2^-9 + 1e-4 (natural log); index handling
bit-exact (permuting physical blocks, poisoning blocks nobody references
and garbage past the context end leave the output bit-identical).
"""
import copy

import numpy as np
import pytest
import torch

import workloads
from msa_pins import repermute

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # collected on a CPU-only host with -m gpu
    pytest.skip("no GPU visible", allow_module_level=True)

from gpu_helpers import (LSE_ABS, MAX_ABS, MEAN_ABS, DeviceInstance, bf16_to_f32,  # noqa: E402
                         check_o, dev_bf16, errors, log_parity, run)
from tolerance import weight_rounding_bound  # noqa: E402
import paper_2606_02964_amd as msa  # noqa: E402


def check_full(inst, oracle_lib, **plan_kw):
    o, lse, plan = run(DeviceInstance(inst), **plan_kw)
    ro, rl = oracle_lib.forward(inst)
    go = bf16_to_f32(o)
    check_o(go, ro, lse.cpu().numpy(), rl)
    return go, lse.cpu().numpy(), plan


def test_config1_full_parity(oracle_lib):
    inst = workloads.make_config(1)
    check_full(inst, oracle_lib)


@pytest.mark.parametrize("seed", [11, 12, 13])
def test_config1_other_seeds(oracle_lib, seed):
    check_full(workloads.make_config(1, seed=seed), oracle_lib)


RANDOM = [
    # seed, B, Hq, Hkv, d, max_len, max_segs
    (101, 3, 4, 4, 64, 700, 5),
    (102, 4, 32, 8, 128, 1500, 8),
    (103, 2, 64, 8, 128, 1200, 3),
    (104, 5, 8, 1, 64, 333, 4),
    (105, 3, 6, 2, 128, 900, 6),     # G = 3: tiles with unused rows
    (106, 6, 2, 2, 128, 70, 3),      # short sequences, ragged last blocks
    (107, 2, 16, 16, 64, 2100, 4),   # MHA, many tiles per sequence
]


# plan flags: automatic tile width, forced 128-row, 256-row and 32-row tiles
TILES = [0, msa.MSA_PLAN_TILE_ROWS_128, msa.MSA_PLAN_TILE_ROWS_256, msa.MSA_PLAN_TILE_ROWS_32]


@pytest.mark.parametrize("tile", TILES)
@pytest.mark.parametrize("case", RANDOM)
@pytest.mark.parametrize("split", [0, 64, 320])
def test_random_full_parity(oracle_lib, case, split, tile):
    seed, B, Hq, Hkv, d, max_len, max_segs = case
    inst = workloads.make_random(seed, num_seqs=B, num_q_heads=Hq, num_kv_heads=Hkv, head_dim=d,
                                 max_len=max_len, max_segs=max_segs, keep_logical=False)
    _, _, plan = check_full(inst, oracle_lib, kv_split_tokens=split, flags=tile)
    max_keys = max((s + n for b in range(inst.num_seqs) for (s, n) in inst.segments(b)), default=0)
    if split and max_keys > split:
        assert plan.info()["num_merge"] > 0


@pytest.mark.parametrize("tile", TILES[1:])
def test_block_aligned_and_adjacent_segments(oracle_lib, tile):
    inst = workloads.make_layout(31, [1024, 777], [[(0, 16), (16, 32), (64, 64), (512, 512)],
                                                  [(0, 1), (1, 1), (400, 377)]], 32, 8, 128)
    check_full(inst, oracle_lib, flags=tile)


@pytest.mark.parametrize("tile", TILES[1:])
def test_prefill_and_decode_layouts(oracle_lib, tile):
    inst = workloads.make_layout(32, [1000, 513, 64], [[(0, 1000)], [(512, 1)], [(63, 1)]], 8, 2, 128)
    check_full(inst, oracle_lib, flags=tile)


@pytest.mark.parametrize("precise", [0, msa.MSA_PLAN_PRECISE_WEIGHTS])
@pytest.mark.parametrize("case", [RANDOM[1], RANDOM[4], RANDOM[6]])
def test_tile_width_is_bitwise_invariant(case, precise):
    """A row's arithmetic does not depend on which rows share its tile, so
    without key splits the 128-row and 256-row kernels agree bit for bit
    (with bf16 or precise weights alike)."""
    seed, B, Hq, Hkv, d, max_len, max_segs = case
    inst = workloads.make_random(seed, num_seqs=B, num_q_heads=Hq, num_kv_heads=Hkv, head_dim=d,
                                 max_len=max_len, max_segs=max_segs, keep_logical=False)
    dinst = DeviceInstance(inst)
    o1, l1, p1 = run(dinst, flags=precise | msa.MSA_PLAN_NO_AUTO_SPLIT | msa.MSA_PLAN_TILE_ROWS_128)
    o2, l2, p2 = run(dinst, flags=precise | msa.MSA_PLAN_NO_AUTO_SPLIT | msa.MSA_PLAN_TILE_ROWS_256)
    assert p1.info()["tile_rows"] == 128 and p2.info()["tile_rows"] == 256
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))
    assert torch.equal(l1, l2)


def test_sequences_sharing_physical_prefix_blocks(oracle_lib):
    """Two sequences whose block tables point at the same physical blocks for
    a shared prefix (prefix caching, Sec. 2.2)."""
    inst = workloads.make_layout(33, [300, 300], [[(100, 50), (250, 50)], [(128, 40), (290, 10)]],
                                 8, 2, 64, permute_blocks=True)
    inst.block_table = inst.block_table.copy()
    inst.block_table[1, :8] = inst.block_table[0, :8]   # first 128 positions shared
    check_full(inst, oracle_lib)


def test_zero_rows_launches_nothing():
    inst = workloads.make_layout(34, [64, 32], [[], []], 4, 2, 64)
    d = DeviceInstance(inst)
    plan = d.plan()
    assert plan.info()["num_work"] == 0
    o = torch.empty((0, 4, 64), dtype=torch.bfloat16, device="cuda")
    msa.msa_forward(plan, d.q, d.k, d.v, d.bt, o, None, None)
    torch.cuda.synchronize()


def _sample_items(inst, n, seed):
    rng = np.random.Generator(np.random.PCG64(seed))
    rows = rng.integers(0, inst.total_q, size=n)
    # first and last rows of every sequence, every row at position 0
    starts = np.cumsum(np.r_[0, [inst.seg_len[inst.seg_indptr[b]:inst.seg_indptr[b + 1]].sum()
                                 for b in range(inst.num_seqs)]])
    extra = [s for s in starts[:-1]] + [e - 1 for e in starts[1:] if e > 0]
    rows = np.r_[rows, np.asarray(extra, dtype=np.int64)]
    rows = rows[(rows >= 0) & (rows < inst.total_q)]
    heads = rng.integers(0, inst.num_q_heads, size=rows.shape[0])
    return rows.astype(np.int64), heads.astype(np.int32)


@pytest.mark.parametrize("split", [0, 4096])
@pytest.mark.parametrize("hq,hkv,d", [(16, 2, 128), (16, 2, 64), (32, 1, 128)])
def test_decode_tiles_long_unsplit_rows(oracle_lib, split, hq, hkv, d):
    """32-row tiles over long key ranges.  Without splits a wave of a tile
    covering 50000 keys runs 391 half-steps, past the 64 whose block ids it
    loads up front, so it also reads ids from the table as it goes.  Rows:
    decode rows at several context lengths (one ending mid-block), two
    tokens of one sequence (a causal mask inside the last half-step); groups
    of 8 and of 32 heads (one token fills a tile), d = 128 and 64."""
    kv = [50000, 8193, 12345, 40, 17]
    segs = [[(49999, 1)], [(8192, 1)], [(12343, 2)], [(39, 1)], [(16, 1)]]
    if hq // hkv == 32:
        segs[2] = [(12344, 1)]  # two tokens x 32 heads would not fit a 32-row tile
    inst = workloads.make_layout(77, kv, segs, hq, hkv, d, keep_logical=False)
    flags = msa.MSA_PLAN_TILE_ROWS_32 | (msa.MSA_PLAN_NO_AUTO_SPLIT if split == 0 else 0)
    _, _, plan = check_full(inst, oracle_lib, kv_split_tokens=split, flags=flags)
    assert plan.info()["tile_rows"] == 32
    assert (plan.info()["num_merge"] > 0) == (split > 0)


@pytest.mark.parametrize("tile", [msa.MSA_PLAN_TILE_ROWS_128, msa.MSA_PLAN_TILE_ROWS_256,
                                  msa.MSA_PLAN_TILE_ROWS_32])
def test_scores_that_start_far_below_and_jump(oracle_lib, tile):
    """Score ranges that exercise the reference max: a rank-one bias along a
    unit vector u puts each sequence's first 64 keys about 150 (log2 units)
    below zero, where a weight against a zero reference would underflow, and
    lifts later keys by about 9 and 25, more than the 2^8 the reference
    allows.  Rows see each jump inside their context, so the reference moves
    mid-row and O is rescaled by factors that underflow to zero."""
    inst = workloads.make_random(4242, num_seqs=3, num_q_heads=8, num_kv_heads=2, head_dim=128,
                                 min_len=200, max_len=700, max_segs=4, keep_logical=True)
    rng = np.random.Generator(np.random.PCG64(7))
    d = inst.head_dim
    u = rng.standard_normal(d)
    u /= np.linalg.norm(u)
    q = workloads.bf16_bits_to_f32(inst.q).astype(np.float64) + 6.0 * u
    inst.q = workloads.f32_to_bf16_bits(q.astype(np.float32))
    # log2-unit shift of a key's score: 6 * a * scale * log2(e)
    a_of = lambda p: np.where(p < 64, -200.0, np.where(p < 160, 0.0, np.where(p < 320, 12.0, 33.0)))
    ks = []
    for kl in inst.k_logical:
        pos = np.arange(kl.shape[0], dtype=np.float64)
        kf = workloads.bf16_bits_to_f32(kl).astype(np.float64) + a_of(pos)[:, None, None] * u
        ks.append(workloads.f32_to_bf16_bits(kf.astype(np.float32)))
    inst.k_logical = ks
    inst.k_cache, inst.v_cache = workloads.layout_cache(inst.block_table, inst.num_blocks, ks, inst.v_logical)
    o, lse, _ = run(DeviceInstance(inst), flags=tile)
    ro, rl = oracle_lib.forward(inst)
    go = bf16_to_f32(o)
    check_o(go, ro)
    # the scores reach ~1200 before scaling: their fp32 accumulation over d
    # products adds up to d * 2^-24 * |q| |k| * scale to lse
    qn = float(np.linalg.norm(q, axis=-1).max())
    kn = max(float(np.linalg.norm(workloads.bf16_bits_to_f32(k).astype(np.float64), axis=-1).max()) for k in ks)
    bound = LSE_ABS + d * 2.0 ** -24 * qn * kn * inst.scale
    assert float(np.abs(lse.cpu().numpy().astype(np.float64) - rl).max()) <= bound


PEAKY = [(303, 3, 32, 8, 128, 1500), (304, 4, 16, 16, 64, 900)]


def _peaky_instance(case):
    seed, B, hq, hkv, d, max_len = case
    inst = workloads.make_random(seed, num_seqs=B, num_q_heads=hq, num_kv_heads=hkv, head_dim=d,
                                 max_len=max_len, max_segs=6, keep_logical=False)
    inst.q = workloads.f32_to_bf16_bits(workloads.bf16_bits_to_f32(inst.q) * np.float32(4.0))
    return inst


@pytest.mark.parametrize("tile", TILES)
@pytest.mark.parametrize("case", PEAKY)
def test_peaky_logits_precise_weights(oracle_lib, case, tile):
    """The peaky-logit inputs below with MSA_PLAN_PRECISE_WEIGHTS: every
    weight enters the PV product as hi + lo bf16 terms, and the plain bar
    holds again."""
    check_full(_peaky_instance(case), oracle_lib, flags=tile | msa.MSA_PLAN_PRECISE_WEIGHTS)


@pytest.mark.parametrize("tile", TILES)
@pytest.mark.parametrize("split", [0, 320])
@pytest.mark.parametrize("case", [RANDOM[1], RANDOM[4], RANDOM[6]])
def test_precise_weights_random(oracle_lib, case, split, tile):
    seed, B, Hq, Hkv, d, max_len, max_segs = case
    inst = workloads.make_random(seed, num_seqs=B, num_q_heads=Hq, num_kv_heads=Hkv, head_dim=d,
                                 max_len=max_len, max_segs=max_segs, keep_logical=False)
    check_full(inst, oracle_lib, kv_split_tokens=split, flags=tile | msa.MSA_PLAN_PRECISE_WEIGHTS)


@pytest.mark.parametrize("tile", TILES)
@pytest.mark.parametrize("case", PEAKY)
def test_peaky_logits(oracle_lib, case, tile):
    """Peaky logits (a stress case outside the five workloads): Q scaled by 4
    (exact in bf16), so the scores of a row spread over about 6 log2 units and
    a few keys carry most of its weight.  The weights of keys before a row's
    diagonal step enter the PV product as bf16 numbers, which moves such a
    row's output by up to 2^-8 sum_j p_j |v_j| before its own rounding; with
    that rounding on top the plain 1e-2 is out of reach here (see
    ``tolerance.weight_rounding_bound``).  Every element must lie within
    that bound, computed from the oracle run on the same instance with |V|;
    the mean-abs and lse bars are the usual ones."""
    inst = _peaky_instance(case)
    o, lse, _ = run(DeviceInstance(inst), flags=tile)
    ro, rl = oracle_lib.forward(inst)
    abs_v = copy.copy(inst)
    abs_v.v_cache = inst.v_cache & np.uint16(0x7FFF)
    ra, _ = oracle_lib.forward(abs_v)
    go = bf16_to_f32(o).astype(np.float64)
    err = np.abs(go - ro)
    bound = weight_rounding_bound(ro, ra)
    lerr = float(np.abs(lse.cpu().numpy().astype(np.float64) - rl).max())
    log_parity(elements=int(go.size), plain_max=float(err.max()), mean=float(err.mean()),
               lse_max=lerr, bound_use=float((err / bound).max()))
    assert np.isfinite(go).all()
    assert np.all(err <= bound), float((err / bound).max())
    assert float(err.mean()) <= MEAN_ABS and lerr <= LSE_ABS


# Oracle results of the last full-size workload, shared by the tests that run
# it with different plans (one instance at a time: config 2 alone is 0.7 GB).
_FULL = {}


def _full_oracle(oracle_lib, cfg):
    if cfg not in _FULL:
        _FULL.clear()
        inst = (workloads.make_config(5, decode_only=True) if cfg == "5-decode"
                else workloads.make_config(cfg))
        if cfg == 4:
            # every row for one query head per KV head, a different head of
            # each group: every work item of the plan is covered
            G = inst.num_q_heads // inst.num_kv_heads
            heads = np.array([g * G + g % G for g in range(inst.num_kv_heads)], dtype=np.int32)
            rows = np.repeat(np.arange(inst.total_q, dtype=np.int64), heads.size)
            hsel = np.tile(heads, inst.total_q)
            ro, rl = oracle_lib.forward(inst, rows=rows, heads=hsel)
            _FULL[cfg] = (inst, ro.reshape(inst.total_q, heads.size, -1),
                          rl.reshape(inst.total_q, heads.size), heads)
        else:
            ro, rl = oracle_lib.forward(inst)
            _FULL[cfg] = (inst, ro, rl, None)
    return _FULL[cfg]


@pytest.mark.parametrize("cfg,tile", [(2, 0), (3, 0), (3, msa.MSA_PLAN_TILE_ROWS_32),
                                      (3, msa.MSA_PLAN_PRECISE_WEIGHTS), (4, 0), (5, 0),
                                      (5, msa.MSA_PLAN_TILE_ROWS_32), ("5-decode", 0),
                                      ("5-decode", msa.MSA_PLAN_PRECISE_WEIGHTS)])
def test_named_workload_full_parity(oracle_lib, cfg, tile):
    """Full-size workloads in the benchmark's launch configuration (automatic
    plan; two of them also forced onto 32-row tiles, whose kernel then takes
    prefill segments at full size; two also with precise weights), compared with the oracle on every output
    element and every lse; the long-context workload on every row for one
    query head per KV head (a different head of each group).  Every output
    is also finite and inside the convex hull of V."""
    inst, ro, rl, heads = _full_oracle(oracle_lib, cfg)
    d = DeviceInstance(inst)
    o, lse, plan = run(d, flags=tile)
    if tile & msa.MSA_PLAN_TILE_ROWS_32:
        assert plan.info()["tile_rows"] == 32
    go = o.float()
    assert torch.isfinite(go).all().item(), "some output rows were not written"
    assert torch.isfinite(lse).all().item()
    vmax = float(np.abs(workloads.bf16_bits_to_f32(inst.v_cache)).max())
    assert float(go.abs().max()) <= vmax * (1 + 2 ** -7)
    if heads is not None:
        hs = torch.from_numpy(heads).long().cuda()
        go, lse = go[:, hs], lse[:, hs]
    check_o(go.cpu().numpy(), ro, lse.cpu().numpy(), rl)


def test_longest_context_sampled_parity(oracle_lib):
    """Llama 3.1's longest context, 131072 keys, at one tensor-parallel
    rank's share of Llama-3.1-8B (8 query heads, 2 KV heads): a 1024-token
    chunk at the end and a 512-token recompute segment in the middle of one
    sequence, plus a decode row over 100000 keys in a second one.  The
    automatic plan splits these long units; sampled (row, head) items against
    the oracle, and the first and last row of every segment."""
    L = 131072
    segs = [[(65536, 512), (L - 1024, 1024)], [(99999, 1)]]
    inst = workloads.make_layout(41, [L, 100000], segs, 8, 2, 128, keep_logical=False)
    o, lse, plan = run(DeviceInstance(inst))
    assert plan.info()["num_merge"] > 0, "expected key splits on 131072-key units"
    go = o.float()
    assert torch.isfinite(go).all().item() and torch.isfinite(lse).all().item()
    rows, heads = _sample_items(inst, 120, seed=41)
    edges = np.array([0, 511, 512, 1535, inst.total_q - 1], dtype=np.int64)
    rows = np.r_[rows, edges]
    heads = np.r_[heads, np.arange(edges.size, dtype=np.int32) * 3 % 8].astype(np.int32)
    ro, rl = oracle_lib.forward(inst, rows=rows, heads=heads)
    gsel = go[torch.from_numpy(rows).cuda(), torch.from_numpy(heads).long().cuda()].cpu().numpy()
    lsel = lse[torch.from_numpy(rows).cuda(), torch.from_numpy(heads).long().cuda()].cpu().numpy()
    check_o(gsel, ro, lsel, rl)


@pytest.mark.parametrize("hq,hkv,d", [(32, 8, 128), (16, 16, 64)])
def test_long_prefill_sampled_parity(oracle_lib, hq, hkv, d):
    """A whole 32768-token prompt as one segment [0, 32768) (plain causal
    prefill, FlashAttention's case, at Llama 3.1's 32K context): every tile
    of the sequence, from the first (a few keys) to the last (the whole
    context), in one launch; sampled items plus the first and last rows."""
    L = 32768
    inst = workloads.make_layout(43, [L], [[(0, L)]], hq, hkv, d, keep_logical=False)
    o, lse, plan = run(DeviceInstance(inst))
    go = o.float()
    assert torch.isfinite(go).all().item() and torch.isfinite(lse).all().item()
    rows, heads = _sample_items(inst, 200, seed=43)
    edges = np.array([0, 1, 63, 64, L // 2, L - 2, L - 1], dtype=np.int64)
    rows = np.r_[rows, edges]
    heads = np.r_[heads, np.arange(edges.size, dtype=np.int32) * 5 % hq].astype(np.int32)
    ro, rl = oracle_lib.forward(inst, rows=rows, heads=heads)
    gsel = go[torch.from_numpy(rows).cuda(), torch.from_numpy(heads).long().cuda()].cpu().numpy()
    lsel = lse[torch.from_numpy(rows).cuda(), torch.from_numpy(heads).long().cuda()].cpu().numpy()
    check_o(gsel, ro, lsel, rl)


def test_large_decode_batch_sampled_parity(oracle_lib):
    """1024 sequences with one decode row each (contexts 64..2048 keys, one
    TP=4 rank of Llama-3.1-8B: 8 query heads, 2 KV heads), plus 4 prefill
    chunks: thousands of work items, narrow tiles, automatic splits.
    Sampled (row, head) items and every sequence's row for head 0 against
    the oracle."""
    rng = np.random.Generator(np.random.PCG64(43))
    lens = [int(x) for x in rng.integers(64, 2049, size=1024)]
    segs = [[(L - 1, 1)] for L in lens]
    for b in (3, 500, 777, 1023):
        segs[b] = [(lens[b] - min(lens[b], 200), min(lens[b], 200))]
    inst = workloads.make_layout(43, lens, segs, 8, 2, 128, keep_logical=False)
    o, lse, plan = run(DeviceInstance(inst))
    assert plan.info()["num_work"] > 1000
    go = o.float()
    assert torch.isfinite(go).all().item() and torch.isfinite(lse).all().item()
    rows, heads = _sample_items(inst, 300, seed=43)
    ro, rl = oracle_lib.forward(inst, rows=rows, heads=heads)
    gsel = go[torch.from_numpy(rows).cuda(), torch.from_numpy(heads).long().cuda()].cpu().numpy()
    lsel = lse[torch.from_numpy(rows).cuda(), torch.from_numpy(heads).long().cuda()].cpu().numpy()
    check_o(gsel, ro, lsel, rl)


def test_config4_forced_split_matches_unsplit(oracle_lib):
    inst = workloads.make_config(4)
    d = DeviceInstance(inst)
    o1, l1, p1 = run(d, flags=msa.MSA_PLAN_NO_AUTO_SPLIT)
    o2, l2, p2 = run(d, kv_split_tokens=4096)
    assert p1.info()["num_merge"] == 0 and p2.info()["num_merge"] > 0
    diff = (o1.float() - o2.float()).abs()
    # both are within one bf16 rounding of the same fp32 value
    assert float(diff.max()) <= 2 ** -7 and float(diff.mean()) <= 1e-4
    # each lse is within LSE_ABS of the exact value; the split path's
    # log-sum-exp merge agrees with the unsplit sum to 1e-6 relative (fp32
    # partial sums in another order; measured 2e-7 here)
    assert float((l1 - l2).abs().max()) <= 2 * LSE_ABS
    assert float(((l1 - l2).abs() / l1.abs().clamp_min(1.0)).max()) <= 1e-6
    rows, heads = _sample_items(inst, 600, seed=44)
    ro, _ = oracle_lib.forward(inst, rows=rows, heads=heads)
    sel = o2.float()[torch.from_numpy(rows).cuda(), torch.from_numpy(heads).long().cuda()]
    check_o(sel.cpu().numpy(), ro)


@pytest.mark.parametrize("tile", [0, msa.MSA_PLAN_TILE_ROWS_32])
@pytest.mark.parametrize("case", [RANDOM[1], RANDOM[2], RANDOM[6]])
def test_forced_splits_match_unsplit(case, tile):
    """Splits of 64 keys (every step its own partial, merged by log-sum-exp)
    against the unsplit plan: lse to 1e-6 relative.  O differs by more than
    the output rounding, since each piece weighs its keys against its own
    reference max and so rounds other bf16 weights; both are checked against
    the oracle elsewhere, here only within 2^-7 of each other."""
    seed, B, Hq, Hkv, d, max_len, max_segs = case
    inst = workloads.make_random(seed, num_seqs=B, num_q_heads=Hq, num_kv_heads=Hkv, head_dim=d,
                                 max_len=max_len, max_segs=max_segs, keep_logical=False)
    dinst = DeviceInstance(inst)
    o1, l1, p1 = run(dinst, flags=msa.MSA_PLAN_NO_AUTO_SPLIT | tile)
    o2, l2, p2 = run(dinst, kv_split_tokens=64, flags=tile)
    assert p1.info()["num_merge"] == 0 and p2.info()["num_merge"] > 0
    assert float(((l1 - l2).abs() / l1.abs().clamp_min(1.0)).max()) <= 1e-6
    assert float((o1.float() - o2.float()).abs().max()) <= 2 ** -7


@pytest.mark.parametrize("tile", [0, msa.MSA_PLAN_TILE_ROWS_32])
def test_physical_permutation_is_bitwise_invariant(tile):
    inst = workloads.make_random(201, num_seqs=3, num_q_heads=32, num_kv_heads=8, head_dim=128,
                                 max_len=1500, max_segs=6, keep_logical=False, extra_blocks=5)
    o1, l1, _ = run(DeviceInstance(inst), flags=tile)
    o2, l2, _ = run(DeviceInstance(repermute(inst, 5)), flags=tile)
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))
    assert torch.equal(l1, l2)


@pytest.mark.parametrize("tile", [0, msa.MSA_PLAN_TILE_ROWS_32])
def test_unreferenced_poison_and_garbage_past_context_end(tile):
    """NaN in blocks no table references and huge finite values past the
    context end inside referenced blocks leave every output bit unchanged."""
    inst = workloads.make_random(202, num_seqs=3, num_q_heads=8, num_kv_heads=2, head_dim=128,
                                 min_len=100, max_len=700, max_segs=4, keep_logical=False,
                                 extra_blocks=4)
    o1, l1, _ = run(DeviceInstance(inst), flags=tile)
    bad = copy.copy(inst)
    bad.k_cache = inst.k_cache.copy()
    bad.v_cache = inst.v_cache.copy()
    nan = np.uint16(0x7FC0)
    big = workloads.f32_to_bf16_bits(np.float32(1e30))
    used = set(int(x) for x in inst.block_table[inst.block_table >= 0].ravel())
    for blk in range(inst.num_blocks):
        if blk not in used:
            bad.k_cache[blk] = nan
            bad.v_cache[blk] = nan
    for b in range(inst.num_seqs):
        L = int(inst.seq_kv_len[b])
        if L % 16:
            blk = inst.block_table[b, L // 16]
            bad.k_cache[blk, :, L % 16:, :] = big
            bad.v_cache[blk, :, :, L % 16:] = big
    o2, l2, _ = run(DeviceInstance(bad), flags=tile)
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))
    assert torch.equal(l1, l2)


def test_strided_output_guard_rows_untouched(oracle_lib):
    """o written through non-contiguous strides; the gaps and guard rows
    around the output stay exactly as they were."""
    inst = workloads.make_random(203, num_seqs=2, num_q_heads=8, num_kv_heads=2, head_dim=64,
                                 max_len=600, max_segs=4, keep_logical=False)
    d = DeviceInstance(inst)
    T, Hq, D = inst.total_q, inst.num_q_heads, inst.head_dim
    tok_stride, head_stride = (Hq + 1) * D + 8, D + 8
    buf = torch.full((T + 2, tok_stride), 7.0, dtype=torch.bfloat16, device="cuda")
    base = buf[1:]
    plan = d.plan(o_strides=(tok_stride, head_stride))
    msa.msa_forward(plan, d.q, d.k, d.v, d.bt, base, None, None)
    torch.cuda.synchronize()
    host = buf.float().cpu().numpy()
    assert (host[0] == 7.0).all() and (host[-1] == 7.0).all()
    rows = host[1:T + 1]
    o = np.stack([rows[:, h * head_stride: h * head_stride + D] for h in range(Hq)], axis=1)
    mask = np.ones(tok_stride, bool)
    for h in range(Hq):
        mask[h * head_stride: h * head_stride + D] = False
    assert (rows[:, mask] == 7.0).all()
    ro, _ = oracle_lib.forward(inst)
    check_o(o, ro)


def test_block_ids_past_2gib_offsets(oracle_lib):
    """Physical block ids whose element offsets exceed 2^31: addressing must
    be 64-bit.  The cache is ~4.3 GB per tensor; the referenced blocks sit at
    its top."""
    inst = workloads.make_random(204, num_seqs=2, num_q_heads=16, num_kv_heads=8, head_dim=128,
                                 min_len=200, max_len=500, max_segs=3, keep_logical=False)
    per_block = inst.num_kv_heads * 16 * inst.head_dim       # elements per block
    top = (2 ** 31) // per_block + 64 + inst.num_blocks      # blocks in the big cache
    off = top - inst.num_blocks
    assert off * per_block > 2 ** 31
    k = torch.zeros((top, inst.num_kv_heads, 16, inst.head_dim), dtype=torch.bfloat16, device="cuda")
    v = torch.zeros((top, inst.num_kv_heads, inst.head_dim, 16), dtype=torch.bfloat16, device="cuda")
    k[off:] = dev_bf16(inst.k_cache)
    v[off:] = dev_bf16(inst.v_cache)
    bt = inst.block_table.copy()
    bt[bt >= 0] += off
    btd = torch.from_numpy(bt).cuda()
    shape = msa.make_shape(inst.num_seqs, inst.num_q_heads, inst.num_kv_heads, inst.head_dim,
                           inst.max_blocks_per_seq, top, inst.scale)
    plan = msa.msa_plan(shape, inst.seq_kv_len, inst.seg_indptr, inst.seg_start, inst.seg_len)
    q = dev_bf16(inst.q)
    o = torch.full((inst.total_q, inst.num_q_heads, inst.head_dim), float("nan"),
                   dtype=torch.bfloat16, device="cuda")
    msa.msa_forward(plan, q, k, v, btd, o, None, None)
    torch.cuda.synchronize()
    del k, v
    ro, _ = oracle_lib.forward(inst)
    check_o(bf16_to_f32(o), ro)


def test_forward_argument_errors():
    inst = workloads.make_config(1)
    d = DeviceInstance(inst)
    plan = d.plan(kv_split_tokens=128)
    need = plan.info()["workspace_bytes"]
    assert need > 0
    o = torch.empty((inst.total_q, inst.num_q_heads, inst.head_dim), dtype=torch.bfloat16,
                    device="cuda")
    small = torch.empty(need - 16, dtype=torch.uint8, device="cuda")
    with pytest.raises(msa.MsaError) as e:
        msa.msa_forward(plan, d.q, d.k, d.v, d.bt, o, None, small)
    assert e.value.status == msa.MSA_ERR_INVALID_ARG and "workspace" in msa.msa_last_error()
    with pytest.raises(msa.MsaError):
        msa.msa_forward(plan, d.q, d.k, d.v, d.bt, None, None, None)
    raw = torch.empty(o.numel() * 2 + 8, dtype=torch.uint8, device="cuda")
    with pytest.raises(msa.MsaError):   # misaligned output pointer
        msa.msa_forward(plan, d.q, d.k, d.v, d.bt, raw.data_ptr() + 2, None, None)


def test_plan_reuse_across_layers_and_streams(oracle_lib):
    """One plan, several 'layers' (different K/V caches) and two streams."""
    inst = workloads.make_random(205, num_seqs=2, num_q_heads=8, num_kv_heads=2, head_dim=128,
                                 max_len=800, max_segs=4, keep_logical=False)
    other = workloads.make_random(205, num_seqs=2, num_q_heads=8, num_kv_heads=2, head_dim=128,
                                  max_len=800, max_segs=4, keep_logical=False)
    rng = np.random.Generator(np.random.PCG64(9))
    other.k_cache = workloads.f32_to_bf16_bits(rng.standard_normal(inst.k_cache.shape, np.float32))
    d1, d2 = DeviceInstance(inst), DeviceInstance(other)
    plan = d1.plan()
    torch.cuda.synchronize()
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    outs = []
    for dd, s in ((d1, s1), (d2, s2)):
        o = torch.empty((inst.total_q, inst.num_q_heads, inst.head_dim), dtype=torch.bfloat16,
                        device="cuda")
        msa.msa_forward(plan, dd.q, dd.k, dd.v, dd.bt, o, None, None, stream=s)
        outs.append(o)
    torch.cuda.synchronize()
    for o, ii in zip(outs, (inst, other)):
        ro, _ = oracle_lib.forward(ii)
        check_o(bf16_to_f32(o), ro)


@pytest.mark.parametrize("hq,hkv,d,tile", [(64, 2, 128, 0), (64, 2, 64, msa.MSA_PLAN_TILE_ROWS_128),
                                           (128, 1, 64, 0), (128, 1, 128, msa.MSA_PLAN_TILE_ROWS_128),
                                           (256, 1, 64, 0)])
def test_large_query_groups(oracle_lib, hq, hkv, d, tile):
    """G = Hq/Hkv of 32, 128 and 256: a tile holds 128/G or 256/G tokens
    (one token per tile at G = 256, which needs the 256-row form)."""
    inst = workloads.make_random(301 + hq + d, num_seqs=2, num_q_heads=hq, num_kv_heads=hkv,
                                 head_dim=d, max_len=300, max_segs=3, keep_logical=False)
    _, _, plan = check_full(inst, oracle_lib, flags=tile)
    expect = 128 if tile == msa.MSA_PLAN_TILE_ROWS_128 else (256 if hq // hkv > 128 else plan.info()["tile_rows"])
    assert plan.info()["tile_rows"] == expect


@pytest.mark.parametrize("tile", [0, msa.MSA_PLAN_TILE_ROWS_32])
def test_hip_graph_replays_match_eager(tile):
    """msa_kv_append and msa_forward (with key splits, so the merge kernel
    runs too) allocate and clear nothing, so a serving loop can capture them
    in a HIP graph.  Every replay, with eager work and synchronisation in
    between, must give the eager outputs bit for bit."""
    inst = workloads.make_random(211, num_seqs=3, num_q_heads=16, num_kv_heads=4, head_dim=128,
                                 max_len=1500, max_segs=5, keep_logical=False)
    d = DeviceInstance(inst)
    plan = d.plan(kv_split_tokens=256, flags=tile)
    info = plan.info()
    assert info["num_merge"] > 0
    kn, vn = (dev_bf16(x) for x in workloads.make_fresh_kv(inst, 5))
    shape_o = (inst.total_q, inst.num_q_heads, inst.head_dim)
    ws = torch.empty(info["workspace_bytes"], dtype=torch.uint8, device="cuda")

    def step(o, lse):
        msa.msa_kv_append(plan, kn, vn, d.bt, d.k, d.v)
        msa.msa_forward(plan, d.q, d.k, d.v, d.bt, o, lse, ws)

    o_ref = torch.empty(shape_o, dtype=torch.bfloat16, device="cuda")
    l_ref = torch.empty(shape_o[:2], dtype=torch.float32, device="cuda")
    step(o_ref, l_ref)
    torch.cuda.synchronize()

    o = torch.empty_like(o_ref)
    lse = torch.empty_like(l_ref)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):  # warm-up on the capture stream
        step(o, lse)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step(o, lse)
    for rep in range(4):
        o.fill_(float("nan"))
        lse.fill_(float("nan"))
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        assert torch.equal(o.view(torch.int16), o_ref.view(torch.int16)), rep
        assert torch.equal(lse.view(torch.int32), l_ref.view(torch.int32)), rep
        (d.q.float() * 2).sum().item()  # unrelated eager work between replays


def test_check_block_table_on_device_tables():
    """The debug validator on device-resident tables: a good table passes; a
    corrupted copy (an entry the plan reads set past the cache, or to -1) is
    reported with its sequence and logical block, on the default and on a
    side stream.  msa_forward never sees the corrupted tables."""
    inst = workloads.make_random(207, num_seqs=4, num_q_heads=8, num_kv_heads=2, head_dim=64,
                                 min_len=100, max_len=600, max_segs=3, keep_logical=False)
    d = DeviceInstance(inst)
    plan = d.plan()
    msa.msa_check_block_table(plan, d.bt)
    # last logical block each sequence's rows read (-1: no rows)
    last = [((lambda sg: (sg[-1][0] + sg[-1][1] - 1) // 16 if sg else -1)(inst.segments(b)))
            for b in range(inst.num_seqs)]
    with_rows = [b for b in range(inst.num_seqs) if last[b] >= 0]
    assert len(with_rows) >= 2
    b0, b1 = with_rows[0], with_rows[-1]
    side = torch.cuda.Stream()
    for b, blk, val, stream in ((b0, 0, inst.num_blocks, None), (b1, last[b1], -1, side),
                                (b1, last[b1] // 2, 2 ** 31 - 1, None)):
        bad = d.bt.clone()
        bad[b, blk] = val
        torch.cuda.synchronize()
        with pytest.raises(msa.MsaError) as e:
            msa.msa_check_block_table(plan, bad, stream=stream)
        assert e.value.status == msa.MSA_ERR_INVALID_ARG
        assert f"sequence {b}, logical block {blk} maps to physical block {val}" in msa.msa_last_error()
    # entries past the last one read are ignored, and so are the rows of
    # sequences without query rows
    ok = d.bt.clone()
    for b in range(inst.num_seqs):
        ok[b, last[b] + 1:] = -1
    msa.msa_check_block_table(plan, ok)
