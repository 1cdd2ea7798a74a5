"""Host-side tests of the C ABI (no GPU needed).

* the library loads and exports every function ``include/msa.h`` declares;
* the planner (run with MSA_PLAN_HOST_ONLY, so nothing touches a device):
  per-row absolute positions are bit-exact, every (row, q head) is covered
  by tiles whose key ranges partition [0, kv_hi) with kv_hi >= position + 1,
  no item reads a block past the last visible one, splits and merge items
  are consistent, plans are deterministic, malformed descriptors get the
  documented status codes;
* a CPU interpreter of the *plan* (per work item partial softmax, then the
  log-sum-exp merge) reproduces the oracle, which pins the planner's key
  ranges and the merge rule without a GPU.
"""
import ctypes
import os
import re
import subprocess
import sys

import numpy as np
import pytest

import workloads

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = [os.path.join(ROOT, "include", h) for h in ("msa.h", "msa_evictor.h")]


@pytest.fixture(scope="module")
def msa():
    import paper_2606_02964_amd as m
    return m


def declared_functions():
    names = set()
    for h in HEADERS:
        text = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        names |= set(re.findall(r"\b(msa_[a-z_]+)\s*\(", text))
    return sorted(names)


def test_library_exports_every_declared_function(msa):
    names = declared_functions()
    assert {"msa_plan", "msa_forward", "msa_plan_info", "msa_plan_destroy",
            "msa_last_error", "msa_plan_export"} <= set(names)
    lib = ctypes.CDLL(msa.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), f"{n} declared in include/ but not exported"
    nm = subprocess.run(["nm", "-D", "--defined-only", msa.LIB_PATH], capture_output=True,
                        text=True, check=True).stdout
    exported = set(re.findall(r"\bT (msa_\w+)", nm))
    assert set(names) <= exported
    assert set(msa.EXPORTED) == set(names)


def shape_of(msa, inst):
    return msa.make_shape(inst.num_seqs, inst.num_q_heads, inst.num_kv_heads, inst.head_dim,
                          inst.max_blocks_per_seq, inst.num_blocks, inst.scale)


def host_plan(msa, inst, **kw):
    flags = kw.pop("flags", 0) | msa.MSA_PLAN_HOST_ONLY
    return msa.msa_plan(shape_of(msa, inst), inst.seq_kv_len, inst.seg_indptr, inst.seg_start,
                        inst.seg_len, flags=flags, **kw)


def expected_positions(inst):
    pos = []
    for b in range(inst.num_seqs):
        for (s, n) in inst.segments(b):
            pos.extend(range(s, s + n))
    return np.asarray(pos, dtype=np.int32)


def row_sequence(inst):
    seq = []
    for b in range(inst.num_seqs):
        seq.extend([b] * int(inst.seg_len[inst.seg_indptr[b]:inst.seg_indptr[b + 1]].sum()))
    return np.asarray(seq, dtype=np.int64)


def check_plan(inst, row_pos, work, merge, info, G):
    """Structural invariants of a plan."""
    total = inst.total_q
    assert np.array_equal(row_pos, expected_positions(inst))
    rseq = row_sequence(inst)
    Hkv = inst.num_kv_heads
    # coverage per (row, kv head): key pieces in order
    pieces = {}
    slots_seen = set()
    for w in work:
        seq, g, row0, nrows, lo, hi, slot, flags = (int(x) for x in w)
        if nrows == 0:
            continue
        assert 0 <= g < Hkv and 0 <= row0 and row0 + nrows <= total
        assert nrows * G <= info["tile_rows"]
        assert (rseq[row0:row0 + nrows] == seq).all(), "tile crosses a sequence"
        assert lo % 64 == 0 and 0 <= lo < hi
        tile_max = int(row_pos[row0:row0 + nrows].max())
        assert hi <= tile_max + 1, "item reads keys past the tile's last visible key"
        assert (hi + 15) // 16 <= (int(inst.seq_kv_len[seq]) + 15) // 16
        if slot >= 0:
            assert slot not in slots_seen
            slots_seen.add(slot)
        key = (row0, nrows, g)
        pieces.setdefault(key, []).append((lo, hi, slot))
    covered = np.zeros((total, Hkv), dtype=np.int32)
    merged = {(int(m[2]), int(m[3]), int(m[1])): m for m in merge}
    for (row0, nrows, g), ps in pieces.items():
        ps.sort()
        assert ps[0][0] == 0
        for a, b in zip(ps, ps[1:]):
            assert a[1] == b[0], "key ranges of a tile must be contiguous"
        hi = ps[-1][1]
        assert (row_pos[row0:row0 + nrows] + 1 <= hi).all()
        if len(ps) == 1:
            assert ps[0][2] == -1
        else:
            m = merged[(row0, nrows, g)]
            assert int(m[4]) == len(ps)
            assert [p[2] for p in ps] == list(range(int(m[5]), int(m[5]) + len(ps)))
        covered[row0:row0 + nrows, g] += 1
    assert (covered == 1).all(), "every (row, kv head) must be in exactly one tile"
    assert len(merged) == len(merge)
    assert info["total_q"] == total
    assert info["tile_rows"] in (32, 128, 256)
    assert info["workspace_bytes"] == len(slots_seen) * info["tile_rows"] * (inst.head_dim + 1) * 4
    useful = 4.0 * inst.head_dim * inst.num_q_heads * float((row_pos.astype(np.float64) + 1).sum())
    assert abs(info["useful_flops"] - useful) <= 1e-9 * max(1.0, useful)


PLAN_CASES = [
    dict(seed=1, num_seqs=3, num_q_heads=4, num_kv_heads=2, head_dim=64, max_len=700, max_segs=6),
    dict(seed=2, num_seqs=5, num_q_heads=32, num_kv_heads=8, head_dim=128, max_len=3000, max_segs=9),
    dict(seed=3, num_seqs=2, num_q_heads=6, num_kv_heads=2, head_dim=128, max_len=500, max_segs=4),
    dict(seed=4, num_seqs=4, num_q_heads=8, num_kv_heads=8, head_dim=64, max_len=129, max_segs=3),
]


@pytest.mark.parametrize("case", PLAN_CASES)
@pytest.mark.parametrize("split", [0, 64, 192, 1024])
@pytest.mark.parametrize("tile_flag", [0, 4, 8, 16])  # auto, 128-row, 256-row, 32-row tiles
def test_plan_structure(msa, case, split, tile_flag):
    inst = workloads.make_random(keep_logical=False, **case)
    plan = host_plan(msa, inst, kv_split_tokens=split, flags=tile_flag)
    info = plan.info()
    row_pos, work, merge = msa.msa_plan_export(plan)
    check_plan(inst, row_pos, work, merge, info, inst.num_q_heads // inst.num_kv_heads)
    if split:
        assert info["num_merge"] > 0 or all(int(w[5]) <= split for w in work if w[3] > 0)


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_plan_structure_named_workloads(msa, cfg):
    inst = make_layout_only(cfg)
    plan = host_plan(msa, inst)
    info = plan.info()
    row_pos, work, merge = msa.msa_plan_export(plan)
    check_plan(inst, row_pos, work, merge, info, inst.num_q_heads // inst.num_kv_heads)
    # a plan's masked waste stays small
    assert info["tile_flops"] <= 1.6 * info["useful_flops"] + 4 * 128 * inst.head_dim * 64 * len(work)


def make_layout_only(cfg):
    """The named workload's descriptors without drawing its (large) tensors."""
    name, layout = workloads.CONFIGS[cfg]
    rng = np.random.Generator(np.random.PCG64(cfg))
    lens, segs, heads = layout(rng)

    class L:
        pass
    inst = L()
    inst.num_seqs = len(lens)
    inst.num_q_heads, inst.num_kv_heads, inst.head_dim = (heads["num_q_heads"],
                                                          heads["num_kv_heads"], heads["head_dim"])
    inst.block_size = 16
    inst.scale = 1.0 / np.sqrt(inst.head_dim)
    inst.seq_kv_len = np.asarray(lens, np.int32)
    starts, ls, indptr = [], [], [0]
    for sg in segs:
        for (s, n) in sg:
            starts.append(s)
            ls.append(n)
        indptr.append(len(starts))
    inst.seg_start = np.asarray(starts, np.int32)
    inst.seg_len = np.asarray(ls, np.int32)
    inst.seg_indptr = np.asarray(indptr, np.int32)
    inst.max_blocks_per_seq = max(-(-L // 16) for L in lens)
    inst.num_blocks = sum(-(-L // 16) for L in lens)
    inst.total_q = int(inst.seg_len.sum())
    inst.segments = lambda b: [(int(inst.seg_start[k]), int(inst.seg_len[k]))
                               for k in range(inst.seg_indptr[b], inst.seg_indptr[b + 1])]
    return inst


def test_named_workload_sizes():
    """Row counts of the named workloads match their definitions."""
    assert make_layout_only(1).total_q == 128
    assert make_layout_only(2).total_q == 8 * (128 * 16 + 512)
    assert make_layout_only(3).total_q == 16 * 64 * 32
    assert make_layout_only(4).total_q == 2 * (2048 + 4096)


def test_plan_is_deterministic(msa):
    inst = workloads.make_random(keep_logical=False, **PLAN_CASES[1])
    a = msa.msa_plan_export(host_plan(msa, inst))
    b = msa.msa_plan_export(host_plan(msa, inst))
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


@pytest.mark.parametrize("tile_flag", [0, 4, 8, 16])
def test_precise_weights_flag_leaves_the_plan_unchanged(msa, tile_flag):
    """MSA_PLAN_PRECISE_WEIGHTS changes only the kernels' arithmetic: the
    exported plan (positions, work items, merges) is the same; flag bits
    beyond the documented ones are still refused."""
    inst = workloads.make_random(keep_logical=False, **PLAN_CASES[1])
    a = msa.msa_plan_export(host_plan(msa, inst, flags=tile_flag))
    b = msa.msa_plan_export(host_plan(msa, inst, flags=tile_flag | msa.MSA_PLAN_PRECISE_WEIGHTS))
    for x, y in zip(a, b):
        assert np.array_equal(x, y)
    with pytest.raises(msa.MsaError) as e:
        host_plan(msa, inst, flags=msa.MSA_PLAN_PRECISE_WEIGHTS << 1)
    assert e.value.status == msa.MSA_ERR_INVALID_ARG


def test_empty_and_zero_segment_sequences(msa):
    inst = workloads.make_layout(5, [10, 40, 0], [[], [(3, 5)], []], 4, 2, 64)
    plan = host_plan(msa, inst)
    info = plan.info()
    row_pos, work, merge = msa.msa_plan_export(plan)
    assert info["total_q"] == 5 and list(row_pos) == [3, 4, 5, 6, 7]
    check_plan(inst, row_pos, work, merge, info, 2)
    none = workloads.make_layout(6, [16], [[]], 2, 2, 64)
    p2 = host_plan(msa, none)
    assert p2.info()["total_q"] == 0 and p2.info()["num_work"] == 0


def test_forward_rejects_host_only_plan_and_null_plan(msa):
    inst = workloads.make_config(1)
    plan = host_plan(msa, inst)
    with pytest.raises(msa.MsaError) as e:
        msa.msa_forward(plan, 16, 16, 16, 16, 16, stream=0)
    assert e.value.status == msa.MSA_ERR_INVALID_ARG
    assert "HOST_ONLY" in msa.msa_last_error()
    null = msa.Plan(None, None)
    with pytest.raises(msa.MsaError):
        msa.msa_forward(null, 16, 16, 16, 16, 16, stream=0)


def test_kv_append_rejects_bad_arguments(msa):
    inst = workloads.make_config(1)
    plan = host_plan(msa, inst)
    for bad in [(0, 64), (8 * 64, 0), (-64, 64), (260, 64), (256, 12)]:
        with pytest.raises(msa.MsaError) as e:
            msa.msa_kv_append(plan, 16, 16, 16, 16, 16, k_new_strides=bad, stream=0)
        assert e.value.status == msa.MSA_ERR_INVALID_ARG
        assert "strides" in msa.msa_last_error()
    with pytest.raises(msa.MsaError) as e:
        msa.msa_kv_append(plan, 16, 16, 16, 16, 16, stream=0)
    assert e.value.status == msa.MSA_ERR_INVALID_ARG
    assert "HOST_ONLY" in msa.msa_last_error()
    with pytest.raises(msa.MsaError):
        msa.msa_kv_append(msa.Plan(None, None), 16, 16, 16, 16, 16, stream=0)


def _bad(inst, what):
    kv = inst.seq_kv_len.copy()
    ip = inst.seg_indptr.copy()
    ss = inst.seg_start.copy()
    sl = inst.seg_len.copy()
    if what == "overlap":
        ss[1] = ss[0] + sl[0] - 1
    elif what == "unsorted":
        ss[0], ss[1] = ss[1], ss[0]
        sl[0], sl[1] = sl[1], sl[0]
    elif what == "empty":
        sl[1] = 0
    elif what == "past_end":
        ss[1] = kv[0] - sl[1] + 1
    elif what == "negative_start":
        ss[0] = -1
    elif what == "kv_len_too_big":
        kv[0] = inst.max_blocks_per_seq * 16 + 1
    elif what == "indptr":
        ip[0] = 1
    return kv, ip, ss, sl


@pytest.mark.parametrize("what", ["overlap", "unsorted", "empty", "past_end", "negative_start",
                                  "kv_len_too_big", "indptr"])
def test_plan_rejects_malformed_segments(msa, what):
    inst = workloads.make_layout(7, [256], [[(10, 30), (100, 40)]], 4, 2, 64)
    kv, ip, ss, sl = _bad(inst, what)
    with pytest.raises(msa.MsaError) as e:
        msa.msa_plan(shape_of(msa, inst), kv, ip, ss, sl, flags=msa.MSA_PLAN_HOST_ONLY)
    assert e.value.status == msa.MSA_ERR_INVALID_ARG
    assert msa.msa_last_error()


@pytest.mark.parametrize("field,value,status", [
    ("head_dim", 96, 2), ("head_dim", 0, 1), ("block_size", 32, 2), ("block_size", 0, 1),
    ("num_kv_heads", 3, 1), ("num_q_heads", 0, 1), ("q_stride_tok", 12, 1),
    ("v_stride_dim", 0, 1), ("scale", float("nan"), 1), ("scale", 0.0, 1), ("scale", -0.5, 1),
    ("num_seqs", -1, 1)])
def test_plan_rejects_bad_shapes(msa, field, value, status):
    inst = workloads.make_layout(8, [256], [[(10, 30)]], 4, 2, 64)
    sh = shape_of(msa, inst)
    setattr(sh, field, value)
    with pytest.raises(msa.MsaError) as e:
        msa.msa_plan(sh, inst.seq_kv_len, inst.seg_indptr, inst.seg_start, inst.seg_len,
                     flags=msa.MSA_PLAN_HOST_ONLY)
    assert e.value.status == status


def _blocks_read(inst):
    """Block-table entries a plan reads per sequence: logical blocks up to
    the one holding the sequence's largest query position."""
    out = []
    for b in range(inst.num_seqs):
        segs = inst.segments(b)
        out.append(0 if not segs else (segs[-1][0] + segs[-1][1] - 1) // 16 + 1)
    return out


@pytest.mark.parametrize("case", PLAN_CASES)
@pytest.mark.parametrize("tile_flag", [0, 16])
def test_check_block_table_covers_every_entry_the_kernels_read(msa, case, tile_flag):
    """The validator's range contains every block a work item (and an append
    slice) touches, and holds exactly the entries the model above names."""
    inst = workloads.make_random(keep_logical=False, **case)
    plan = host_plan(msa, inst, kv_split_tokens=64, flags=tile_flag)
    _, work, _ = msa.msa_plan_export(plan)
    nread = _blocks_read(inst)
    for w in work:
        if w[3] > 0:
            assert (int(w[5]) - 1) // 16 < nread[int(w[0])]
    msa.msa_check_block_table(plan, inst.block_table)
    rng = np.random.default_rng(case["seed"])
    # a bad value at each read entry is found and named; unread entries are ignored
    for b in range(inst.num_seqs):
        for i in sorted(set(rng.integers(0, max(nread[b], 1), size=3).tolist())) if nread[b] else []:
            for bad in (-1, inst.num_blocks, 2 ** 31 - 1):
                bt = inst.block_table.copy()
                bt[b, i] = bad
                with pytest.raises(msa.MsaError) as e:
                    msa.msa_check_block_table(plan, bt)
                assert e.value.status == msa.MSA_ERR_INVALID_ARG
                assert f"sequence {b}, logical block {i} maps to physical block {bad}" in msa.msa_last_error()
        if nread[b] < inst.max_blocks_per_seq:
            bt = inst.block_table.copy()
            bt[b, nread[b]:] = -7
            msa.msa_check_block_table(plan, bt)


def test_check_block_table_reports_the_first_bad_entry(msa):
    inst = workloads.make_layout(35, [100, 64, 300], [[(10, 5), (90, 10)], [], [(200, 1)]], 4, 2, 64,
                                 keep_logical=False, permute_blocks=True)
    plan = host_plan(msa, inst)
    assert _blocks_read(inst) == [7, 0, 13]
    bt = inst.block_table.copy()
    bt[1, :] = -1            # sequence 1 has no query rows: nothing read
    msa.msa_check_block_table(plan, bt)
    bt[2, 12] = -3
    bt[2, 4] = 10 ** 6
    bt[0, 6] = -1
    with pytest.raises(msa.MsaError):
        msa.msa_check_block_table(plan, bt)
    assert "sequence 0, logical block 6 maps to physical block -1" in msa.msa_last_error()
    bt[0, 6] = 0
    with pytest.raises(msa.MsaError):
        msa.msa_check_block_table(plan, bt)
    assert "sequence 2, logical block 4 maps to physical block 1000000" in msa.msa_last_error()


def test_check_block_table_arguments(msa):
    inst = workloads.make_config(1)
    plan = host_plan(msa, inst)
    lib = msa._lib
    assert lib.msa_check_block_table(None, inst.block_table.ctypes.data, msa.MSA_TABLE_HOST, None) \
        == msa.MSA_ERR_INVALID_ARG
    assert lib.msa_check_block_table(plan.handle, None, msa.MSA_TABLE_HOST, None) == msa.MSA_ERR_INVALID_ARG
    assert lib.msa_check_block_table(plan.handle, inst.block_table.ctypes.data, 7, None) \
        == msa.MSA_ERR_INVALID_ARG
    # a plan without query rows reads no entry: even a null table passes
    empty = workloads.make_layout(36, [64], [[]], 4, 2, 64, keep_logical=False)
    assert lib.msa_check_block_table(host_plan(msa, empty).handle, None, msa.MSA_TABLE_HOST, None) == msa.MSA_OK


def test_plan_rejects_bad_options(msa):
    inst = workloads.make_layout(9, [256], [[(10, 30)]], 4, 2, 64)
    for kw in (dict(kv_split_tokens=100), dict(q_tile_tokens=65), dict(kv_split_tokens=-64)):
        with pytest.raises(msa.MsaError) as e:
            host_plan(msa, inst, **kw)
        assert e.value.status == msa.MSA_ERR_INVALID_ARG
    too_big_group = workloads.make_layout(10, [64], [[(0, 4)]], 512, 1, 64)
    with pytest.raises(msa.MsaError) as e:
        host_plan(msa, too_big_group)
    assert e.value.status == msa.MSA_ERR_UNSUPPORTED
    big_group = workloads.make_layout(10, [64], [[(0, 4)]], 256, 1, 64)
    assert host_plan(msa, big_group).info()["tile_rows"] == 256
    with pytest.raises(msa.MsaError) as e:
        host_plan(msa, big_group, flags=msa.MSA_PLAN_TILE_ROWS_128)
    assert e.value.status == msa.MSA_ERR_UNSUPPORTED
    for both in (msa.MSA_PLAN_TILE_ROWS_128 | msa.MSA_PLAN_TILE_ROWS_256,
                 msa.MSA_PLAN_TILE_ROWS_32 | msa.MSA_PLAN_TILE_ROWS_128,
                 msa.MSA_PLAN_TILE_ROWS_32 | msa.MSA_PLAN_TILE_ROWS_256):
        with pytest.raises(msa.MsaError) as e:
            host_plan(msa, inst, flags=both)
        assert e.value.status == msa.MSA_ERR_INVALID_ARG
    # 32-row tiles hold at most 32 rows: Hq / Hkv <= 32
    g64 = workloads.make_layout(10, [64], [[(63, 1)]], 64, 1, 64)
    with pytest.raises(msa.MsaError) as e:
        host_plan(msa, g64, flags=msa.MSA_PLAN_TILE_ROWS_32)
    assert e.value.status == msa.MSA_ERR_UNSUPPORTED
    g32 = workloads.make_layout(10, [64], [[(63, 1)]], 32, 1, 64)
    assert host_plan(msa, g32, flags=msa.MSA_PLAN_TILE_ROWS_32).info()["tile_rows"] == 32
    # the token cap follows the tile width: 128 / 2 = 64 narrow, 128 wide
    assert host_plan(msa, inst, q_tile_tokens=65, flags=msa.MSA_PLAN_TILE_ROWS_256).info()["tile_rows"] == 256


# --------------------------------------------------------------------------
# CPU interpreter of a plan (float64), compared with the oracle
# --------------------------------------------------------------------------

def interpret_plan(inst, row_pos, work, merge):
    """Run the plan's work items with exact float64 math: each item gives a
    partial (o, lse) over its key range per row; split tiles are combined by
    log-sum-exp.  Reads K/V through the block table like the kernel does."""
    from workloads import bf16_bits_to_f32
    G = inst.num_q_heads // inst.num_kv_heads
    d = inst.head_dim
    q = bf16_bits_to_f32(inst.q).astype(np.float64)
    out_o = np.full((inst.total_q, inst.num_q_heads, d), np.nan)
    out_l = np.full((inst.total_q, inst.num_q_heads), np.nan)
    partial = {}
    for w in work:
        seq, g, row0, nrows, lo, hi, slot, _ = (int(x) for x in w)
        if nrows == 0:
            continue
        keys = np.arange(lo, hi)
        blk = inst.block_table[seq, keys // 16]
        K = bf16_bits_to_f32(inst.k_cache[blk, g, keys % 16, :]).astype(np.float64)
        V = bf16_bits_to_f32(inst.v_cache[blk, g, :, keys % 16]).astype(np.float64)
        for t in range(nrows):
            row = row0 + t
            vis = keys <= row_pos[row]
            for hh in range(G):
                h = g * G + hh
                s = inst.scale * (K @ q[row, h])
                s = np.where(vis, s, -np.inf)
                m = s.max()
                if m == -np.inf:
                    o, l = np.zeros(d), -np.inf
                else:
                    e = np.exp(s - m)
                    o, l = (e @ V) / e.sum(), m + np.log(e.sum())
                if slot < 0:
                    out_o[row, h], out_l[row, h] = o, l
                else:
                    partial[(slot, row, h)] = (o, l)
    for m in merge:
        seq, g, row0, nrows, nsplit, slot0 = (int(x) for x in m[:6])
        for t in range(nrows):
            row = row0 + t
            for hh in range(G):
                h = g * G + hh
                parts = [partial[(slot0 + k, row, h)] for k in range(nsplit)]
                ls = np.array([p[1] for p in parts])
                mx = ls.max()
                wts = np.exp(ls - mx)
                out_o[row, h] = sum(wt * p[0] for wt, p in zip(wts, parts)) / wts.sum()
                out_l[row, h] = mx + np.log(wts.sum())
    return out_o, out_l


@pytest.mark.parametrize("tile_flag", [4, 8, 16])
@pytest.mark.parametrize("split", [0, 64, 128])
@pytest.mark.parametrize("case", PLAN_CASES[:2] + PLAN_CASES[3:])
def test_plan_interpreter_matches_oracle(msa, oracle_lib, case, split, tile_flag):
    case = dict(case, max_len=min(case["max_len"], 400))
    inst = workloads.make_random(keep_logical=False, **case)
    plan = host_plan(msa, inst, kv_split_tokens=split, flags=tile_flag)
    row_pos, work, merge = msa.msa_plan_export(plan)
    io, il = interpret_plan(inst, row_pos, work, merge)
    o, l = oracle_lib.forward(inst)
    np.testing.assert_allclose(io, o, rtol=0, atol=1e-12)
    np.testing.assert_allclose(il, l, rtol=0, atol=1e-12)


def test_fused_ablation_layouts():
    """Prefix and suffix placements of the same cached run compute the same
    number of tokens; the suffix layout's segments are valid and end with the
    128 new tokens (Sec. 6.3)."""
    for ctx in (1024, 10240):
        step = (ctx - 128) // 7 // 16 * 16
        for cached in [i * step for i in range(7)] + [ctx - 128]:
            pre = workloads.fused_ablation_layout(ctx, cached, "prefix")
            suf = workloads.fused_ablation_layout(ctx, cached, "suffix")
            assert sum(n for _, n in pre) == sum(n for _, n in suf) == ctx - cached
            assert pre == [(cached, ctx - cached)]
            assert suf[-1] == (ctx - 128, 128)
            end = 0
            for (s, n) in suf:
                assert s >= end and n >= 1
                end = s + n
            assert end == ctx
            if cached < ctx - 128:
                assert suf[0] == (0, ctx - 128 - cached)


def check_workgroups(work, info, num_kv_heads):
    """The persistent launch: items grouped by workgroup (adjacent, ascending),
    workgroup i on XCD i % 8; inside a workgroup items run in XCD-queue
    order (groups by decreasing longest piece, then id; a group's pieces by
    decreasing cost, cost = key steps + 1); per XCD the workgroups' loads
    differ by at most the largest item cost of that XCD (greedy
    least-loaded assignment); a (sequence, KV head) group's items share one
    XCD unless the group alone is more than half of an XCD's share."""
    wg = work[:, 7].astype(np.int64)
    nwg = info["num_workgroups"]
    slots = 256 if info["tile_rows"] == 256 else 512
    assert 0 < nwg <= slots and (np.diff(wg) >= 0).all() and wg.min() >= 0 and wg.max() == nwg - 1
    cost = (work[:, 5] - work[:, 4] + 63) // 64 + 1
    groups = work[:, 0].astype(np.int64) * num_kv_heads + work[:, 1]
    gmax = {g: cost[groups == g].max() for g in np.unique(groups)}
    key = [(-gmax[g], g, -c) for g, c in zip(groups, cost)]
    for w in np.unique(wg):
        k = [key[i] for i in np.where(wg == w)[0]]
        assert all(a <= b for a, b in zip(k, k[1:])), "a workgroup's items are out of queue order"
    load = np.bincount(wg, weights=cost, minlength=nwg)
    for x in range(8):
        mine = np.arange(x, nwg, 8)
        if mine.size == 0:
            continue
        on_x = (wg % 8) == x
        if on_x.any():
            assert load[mine].max() - load[mine].min() <= cost[on_x].max()
    total = cost.sum()
    for gr in np.unique(groups):
        sel = groups == gr
        if cost[sel].sum() <= 0.5 * total / 8:
            assert len(np.unique(wg[sel] % 8)) == 1, "a group's items are spread over XCDs"
    if len(work) <= nwg:
        assert len(np.unique(wg)) == len(work), "one item per workgroup when they fit"


@pytest.mark.parametrize("cfg", [1, 2, 3, 4, 5])
def test_workgroup_assignment_named_workloads(msa, cfg):
    inst = make_layout_only(cfg)
    plan = host_plan(msa, inst)
    _, work, _ = msa.msa_plan_export(plan)
    check_workgroups(work, plan.info(), inst.num_kv_heads)


@pytest.mark.parametrize("case", PLAN_CASES)
@pytest.mark.parametrize("split", [0, 64, 1024])
@pytest.mark.parametrize("tile_flag", [0, 4, 8, 16])
def test_workgroup_assignment_random(msa, case, split, tile_flag):
    inst = workloads.make_random(keep_logical=False, **case)
    plan = host_plan(msa, inst, kv_split_tokens=split, flags=tile_flag)
    _, work, _ = msa.msa_plan_export(plan)
    if len(work):
        check_workgroups(work, plan.info(), inst.num_kv_heads)


def _descriptors(kv_lens, segs, hq, hkv, d):
    """Plan descriptors of a layout, without drawing its tensors."""
    class L:
        pass
    inst = L()
    inst.num_seqs, inst.num_q_heads, inst.num_kv_heads, inst.head_dim = len(kv_lens), hq, hkv, d
    inst.scale = 1.0 / np.sqrt(d)
    inst.seq_kv_len = np.asarray(kv_lens, np.int32)
    inst.seg_start = np.asarray([st for sg in segs for (st, n) in sg], np.int32)
    inst.seg_len = np.asarray([n for sg in segs for (st, n) in sg], np.int32)
    inst.seg_indptr = np.cumsum([0] + [len(sg) for sg in segs]).astype(np.int32)
    inst.max_blocks_per_seq = max(-(-x // 16) for x in kv_lens)
    inst.num_blocks = sum(-(-x // 16) for x in kv_lens)
    return inst


def test_tile_width_choice(msa):
    """Wide (256-row) tiles for plans with many tiles and a long run of key
    steps per workgroup slot; 32-row tiles when no 128-row tile would hold
    more than 32 rows (decode-only plans); narrow (128-row) tiles for the
    other small and short plans; flags force each."""
    for cfg, rows in ((1, 128), (2, 256), (3, 256), (4, 256), (5, 256)):
        assert host_plan(msa, make_layout_only(cfg)).info()["tile_rows"] == rows, cfg
    # many narrow tiles, little work per slot: 8 x 1024-token requests whose
    # first 896 tokens and last 128 are computed (2048 narrow tiles, ~34
    # steps per slot) stay narrow; the same layout at 10240 tokens goes wide
    for ctx, rows in ((1024, 128), (10240, 256)):
        segs = workloads.fused_ablation_layout(ctx, 0, "suffix")
        inst = _descriptors([ctx] * 8, [segs] * 8, 32, 8, 128)
        assert host_plan(msa, inst).info()["tile_rows"] == rows, ctx
    _, layout = workloads.CONFIGS[5]
    lens, segs, heads = layout(np.random.Generator(np.random.PCG64(5)))
    keep = [b for b in range(len(lens)) if segs[b] == [(lens[b] - 1, 1)]]  # the decode rows
    decode = _descriptors([lens[b] for b in keep], [segs[b] for b in keep], heads["num_q_heads"],
                          heads["num_kv_heads"], heads["head_dim"])
    assert host_plan(msa, decode).info()["tile_rows"] == 32
    assert host_plan(msa, decode, flags=msa.MSA_PLAN_TILE_ROWS_256).info()["tile_rows"] == 256
    assert host_plan(msa, decode, flags=msa.MSA_PLAN_TILE_ROWS_128).info()["tile_rows"] == 128
    # one more decode token per sequence: 2 tokens x 4 heads = 8 rows, still 32-row tiles;
    # a 16-token chunk in one sequence (64 rows) takes the plan back to 128-row tiles
    two = _descriptors([lens[b] for b in keep], [[(lens[b] - 2, 2)] for b in keep], heads["num_q_heads"],
                       heads["num_kv_heads"], heads["head_dim"])
    assert host_plan(msa, two).info()["tile_rows"] == 32
    chunk = _descriptors([lens[b] for b in keep], [[(lens[b] - 16, 16)] if i == 0 else [(lens[b] - 1, 1)]
                                                   for i, b in enumerate(keep)],
                         heads["num_q_heads"], heads["num_kv_heads"], heads["head_dim"])
    assert host_plan(msa, chunk).info()["tile_rows"] == 128
    assert host_plan(msa, make_layout_only(2), flags=msa.MSA_PLAN_TILE_ROWS_128).info()["tile_rows"] == 128


def test_decode_split_fits_one_round(msa):
    """32-row plans cut their units at the shortest 64-aligned length whose
    pieces all fit one round of the 512 workgroup slots (two per CU)."""
    _, layout = workloads.CONFIGS[5]
    lens, segs, heads = layout(np.random.Generator(np.random.PCG64(5)))
    keep = [b for b in range(len(lens)) if segs[b] == [(lens[b] - 1, 1)]]
    decode = _descriptors([lens[b] for b in keep], [segs[b] for b in keep], heads["num_q_heads"],
                          heads["num_kv_heads"], heads["head_dim"])
    plan = host_plan(msa, decode)
    _, work, _ = msa.msa_plan_export(plan)
    assert plan.info()["tile_rows"] == 32
    slots = 2 * 256
    units = [lens[b] for b in keep for _ in range(heads["num_kv_heads"])]
    count = lambda n: sum(-(-u // n) for u in units)
    longest = int((work[:, 5] - work[:, 4]).max())
    assert len(work) == count(longest) <= slots
    assert longest % 64 == 0 and count(longest - 64) > slots
    # more units than slots: no split
    many = _descriptors([2000] * 200, [[(1999, 1)]] * 200, 32, 8, 128)
    p2 = host_plan(msa, many)
    assert p2.info()["tile_rows"] == 32 and p2.info()["num_merge"] == 0


@pytest.mark.parametrize("seed", range(12))
def test_decode_split_rule_on_random_batches(msa, seed):
    """Random decode batches: the pieces of a 32-row plan fit one round of
    the 512 workgroup slots whenever the units alone do, and no shorter
    64-aligned cut (above the 1024-key floor) would still fit."""
    rng = np.random.default_rng(seed)
    B = int(rng.integers(1, 96))
    hkv = int(rng.choice([1, 2, 4, 8]))
    G = int(rng.choice([1, 2, 4, 8]))
    lens = [int(x) for x in rng.integers(1, 40000, size=B)]
    inst = _descriptors(lens, [[(L - 1, 1)] for L in lens], G * hkv, hkv, 128)
    plan = host_plan(msa, inst)
    info = plan.info()
    assert info["tile_rows"] == 32
    _, work, _ = msa.msa_plan_export(plan)
    work = work[work[:, 3] > 0]  # padding items (empty, they exit at once) even out the XCD queues
    units = [L for L in lens for _ in range(hkv)]
    slots = 512
    if len(units) > slots:
        assert info["num_merge"] == 0 and len(work) == len(units)
        return
    assert len(work) <= slots
    if info["num_merge"]:
        # every piece is at most the cut length, so rounding the longest one
        # up to 64 keys gives at most the cut; one step shorter must not fit
        longest = int((work[:, 5] - work[:, 4]).max())
        at_most_cut = -(-longest // 64) * 64
        count = lambda n: sum(-(-u // n) for u in units)
        if at_most_cut - 64 >= 1024:
            assert count(at_most_cut - 64) > slots


def test_one_hip_runtime_per_process():
    """Importing the package before torch must not load a second HIP runtime
    (torch's streams and device pointers belong to torch's runtime)."""
    code = ("import paper_2606_02964_amd, torch\n"
            "maps = open('/proc/self/maps').read().split('\\n')\n"
            "paths = {l.split()[-1] for l in maps if 'libamdhip64' in l}\n"
            "print(len(paths))\n")
    out = subprocess.run([sys.executable, "-c", code], cwd=ROOT, capture_output=True, text=True,
                         check=True).stdout.strip()
    assert out == "1", out


C_CONSUMER = r"""
#include <stdio.h>
#include <string.h>
#include "msa.h"
#include "msa_evictor.h"

int main(void) {
  /* two sequences: [40, 72) of 100 keys; [0, 16) and [33, 34) of 50 keys */
  const int32_t kv[2] = {100, 50}, indptr[3] = {0, 1, 3};
  const int32_t start[3] = {40, 0, 33}, len[3] = {32, 16, 1};
  msa_shape s;
  memset(&s, 0, sizeof s);
  s.num_seqs = 2; s.num_q_heads = 8; s.num_kv_heads = 2; s.head_dim = 128; s.block_size = 16;
  s.max_blocks_per_seq = 7; s.num_blocks = 11; s.scale = 0.0883883476f;
  s.q_stride_tok = 8 * 128; s.q_stride_head = 128; s.o_stride_tok = 8 * 128; s.o_stride_head = 128;
  s.k_stride_block = 2 * 16 * 128; s.k_stride_head = 16 * 128; s.k_stride_tok = 128;
  s.v_stride_block = 2 * 128 * 16; s.v_stride_head = 128 * 16; s.v_stride_dim = 16;
  msa_plan_opts o;
  memset(&o, 0, sizeof o);
  o.flags = MSA_PLAN_HOST_ONLY;
  msa_plan_t plan = NULL;
  if (msa_plan(&s, kv, indptr, start, len, &o, NULL, &plan) != MSA_OK) {
    printf("plan failed: %s\n", msa_last_error());
    return 1;
  }
  msa_plan_info_t info;
  if (msa_plan_info(plan, &info) != MSA_OK) return 2;
  int32_t row_pos[49];
  if (msa_plan_export(plan, row_pos, NULL, NULL) != MSA_OK) return 3;
  printf("%lld %lld %lld %lld %d %d %d\n", (long long)info.total_q, (long long)info.num_tiles,
         (long long)info.tile_rows, (long long)info.num_work, row_pos[0], row_pos[32], row_pos[48]);
  /* a malformed plan reports through msa_last_error */
  s.head_dim = 96;
  msa_plan_t bad = NULL;
  const msa_status st = msa_plan(&s, kv, indptr, start, len, &o, NULL, &bad);
  printf("%d %d\n", (int)st, bad == NULL);
  msa_plan_destroy(plan);

  msa_evictor_params p;
  memset(&p, 0, sizeof p);
  p.alpha = 10.0; p.beta = 1.0; p.tau0 = 9.0; p.lambda = 1.0;
  msa_evictor_t ev = NULL;
  if (msa_evictor_create(&p, &ev) != MSA_OK) return 4;
  msa_evictor_add(ev, 0, 0.0, 3.0);
  msa_evictor_add(ev, 1, 5.0, 1.0);
  int64_t id = -1;
  msa_evictor_evict(ev, 6.0, &id);
  printf("%lld %lld\n", (long long)id, (long long)msa_evictor_size(ev));
  msa_evictor_destroy(ev);
  return 0;
}
"""


def test_plain_c_consumer(msa, tmp_path):
    """The headers compile as strict C11 and a C program linked against the
    library plans (host only), reports errors and drives the evictor, with
    the same results as the Python binding."""
    src = tmp_path / "consumer.c"
    exe = tmp_path / "consumer"
    src.write_text(C_CONSUMER)
    libdir = os.path.dirname(msa.LIB_PATH)
    subprocess.check_call(["gcc", "-std=c11", "-Wall", "-Wextra", "-Werror", "-pedantic",
                           "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe),
                           "-L", libdir, "-lmsa", f"-Wl,-rpath,{libdir}"])
    out = subprocess.run([str(exe)], capture_output=True, text=True, check=True).stdout.split("\n")
    inst = _descriptors([100, 50], [[(40, 32)], [(0, 16), (33, 1)]], 8, 2, 128)
    plan = host_plan(msa, inst)
    info = plan.info()
    row_pos, _, _ = msa.msa_plan_export(plan)
    assert out[0].split() == [str(x) for x in (info["total_q"], info["num_tiles"], info["tile_rows"],
                                                info["num_work"], row_pos[0], row_pos[32], row_pos[48])]
    assert out[1].split() == [str(msa.MSA_ERR_UNSUPPORTED), "1"]
    assert out[2].split() == ["1", "1"]  # Eq. 9 example: B (released at 5, cost 1) goes first at t = 6
