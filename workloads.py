"""Seeded synthetic inputs for Multi-Segment Attention (MSA).

This module only *generates inputs*: segment layouts, block tables, a paged
K/V cache and packed queries.  It holds none of the attention arithmetic and
is the one piece of code shared by the CPU oracle's tests and the GPU path.

Value recipe: every Q/K/V element is drawn as float32 N(0, 1) and rounded to
bfloat16 with round-to-nearest-even; arrays hold the bf16 *bit patterns*
(uint16).  One ``numpy.random.Generator(PCG64(seed))`` per instance, drawn in
a fixed order: layout, physical block permutation, Q, K, V.

Layouts (what the consumer of this module must accept):

* ``q``        [total_q, Hq, d]            packed query rows.  Sequences in
  order; inside a sequence, segments ascending; inside a segment, ascending
  position.
* ``k_cache``  [num_blocks, Hkv, bs, d]    token-major block, d contiguous.
* ``v_cache``  [num_blocks, Hkv, d, bs]    channel-major block (the value
  vectors of one block stored transposed, tokens contiguous), the layout
  vLLM's paged-attention kernels use for V.
* ``block_table`` [B, max_blocks] int32; unused entries are -1.
* Physical block ids are a seeded random permutation of
  ``0 .. sum_b ceil(L_b / bs) - 1``.

The five named workloads follow the paper's setting: long contexts whose
middle blocks were evicted while both ends stay cached (Sec. 3, Observation
2), multi-turn fragmentation, a 70B-class layer on one GPU, and a mixed
chunked-prefill + decode batch in one launch (Sec. 5.1, adaptive chunking).
They stand in for the LongBench / LooGLE / BFCL traces of Sec. 6, which are
not reproduced here.
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional, Sequence, Tuple

import numpy as np

BLOCK_SIZE = 16


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (round-to-nearest-even); returns uint16 bits.

    Inputs are finite N(0,1) draws, so the NaN/overflow branches of a general
    converter are not needed; they are rejected instead.
    """
    x = np.ascontiguousarray(x, dtype=np.float32)
    if not np.isfinite(x).all():
        raise ValueError("generator values must be finite")
    u = x.view(np.uint32)
    rounded = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return rounded.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to float32."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


@dataclasses.dataclass
class Instance:
    name: str
    num_seqs: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    block_size: int
    scale: float
    seq_kv_len: np.ndarray      # int32 [B]
    seg_indptr: np.ndarray      # int32 [B+1]
    seg_start: np.ndarray       # int32 [nseg]
    seg_len: np.ndarray         # int32 [nseg]
    block_table: np.ndarray     # int32 [B, max_blocks]
    num_blocks: int
    q: np.ndarray               # uint16 [total_q, Hq, d]
    k_cache: np.ndarray         # uint16 [num_blocks, Hkv, bs, d]
    v_cache: np.ndarray         # uint16 [num_blocks, Hkv, d, bs]
    k_logical: Optional[List[np.ndarray]] = None  # per sequence uint16 [L_b, Hkv, d]
    v_logical: Optional[List[np.ndarray]] = None

    @property
    def total_q(self) -> int:
        return int(self.seg_len.sum())

    @property
    def max_blocks_per_seq(self) -> int:
        return int(self.block_table.shape[1])

    def segments(self, b: int) -> List[Tuple[int, int]]:
        lo, hi = int(self.seg_indptr[b]), int(self.seg_indptr[b + 1])
        return [(int(self.seg_start[s]), int(self.seg_len[s])) for s in range(lo, hi)]


def _bf16_normal(rng: np.random.Generator, shape) -> np.ndarray:
    return f32_to_bf16_bits(rng.standard_normal(size=shape, dtype=np.float32))


def layout_cache(block_table: np.ndarray, num_blocks: int, k_logical, v_logical,
                 block_size: int = BLOCK_SIZE) -> Tuple[np.ndarray, np.ndarray]:
    """Place per-sequence logical K/V ([L_b, Hkv, d] bf16 bits) into zeroed
    paged caches K [num_blocks, Hkv, bs, d] and V [num_blocks, Hkv, d, bs]
    through ``block_table`` (whole blocks at a time: reshape + transpose)."""
    B = len(k_logical)
    Hkv, d = (k_logical[0].shape[1], k_logical[0].shape[2]) if B else (1, 1)
    k_cache = np.zeros((num_blocks, Hkv, block_size, d), dtype=np.uint16)
    v_cache = np.zeros((num_blocks, Hkv, d, block_size), dtype=np.uint16)
    for b in range(B):
        L = int(k_logical[b].shape[0])
        nb = -(-L // block_size)
        pad = nb * block_size - L
        kb = np.concatenate([k_logical[b], np.zeros((pad, Hkv, d), np.uint16)])
        vb = np.concatenate([v_logical[b], np.zeros((pad, Hkv, d), np.uint16)])
        kb = kb.reshape(nb, block_size, Hkv, d)
        vb = vb.reshape(nb, block_size, Hkv, d)
        phys = block_table[b, :nb]
        k_cache[phys] = kb.transpose(0, 2, 1, 3)
        v_cache[phys] = vb.transpose(0, 2, 3, 1)
    return k_cache, v_cache


def make_fresh_kv(inst: Instance, seed: int) -> Tuple[np.ndarray, np.ndarray]:
    """Seeded fresh keys and values of every packed row: bf16 bits
    [total_q, Hkv, d] each, drawn N(0, 1) like the rest of the inputs."""
    rng = np.random.Generator(np.random.PCG64(seed))
    shape = (inst.total_q, inst.num_kv_heads, inst.head_dim)
    return _bf16_normal(rng, shape), _bf16_normal(rng, shape)


def build_instance(name: str, rng: np.random.Generator, kv_lens: Sequence[int],
                   segments: Sequence[Sequence[Tuple[int, int]]], num_q_heads: int,
                   num_kv_heads: int, head_dim: int, block_size: int = BLOCK_SIZE,
                   keep_logical: bool = False, extra_blocks: int = 0,
                   permute_blocks: bool = True) -> Instance:
    """Draw Q/K/V for a given layout and lay K/V out in a paged cache.

    ``segments[b]`` is the list of (start, length) query segments of sequence
    b.  ``extra_blocks`` appends that many physical blocks that no block table
    references (callers may poison them).
    """
    B = len(kv_lens)
    assert len(segments) == B
    blocks_per_seq = [-(-int(L) // block_size) for L in kv_lens]
    n_logical = int(sum(blocks_per_seq))
    num_blocks = n_logical + int(extra_blocks)
    perm = rng.permutation(n_logical) if permute_blocks else np.arange(n_logical)
    max_blocks = max(1, max(blocks_per_seq) if blocks_per_seq else 1)
    block_table = np.full((B, max_blocks), -1, dtype=np.int32)
    nxt = 0
    for b in range(B):
        for j in range(blocks_per_seq[b]):
            block_table[b, j] = perm[nxt]
            nxt += 1

    seg_indptr = np.zeros(B + 1, dtype=np.int32)
    starts, lens = [], []
    for b in range(B):
        for (s, n) in segments[b]:
            starts.append(int(s))
            lens.append(int(n))
        seg_indptr[b + 1] = len(starts)
    seg_start = np.asarray(starts, dtype=np.int32)
    seg_len = np.asarray(lens, dtype=np.int32)
    total_q = int(seg_len.sum())

    q = _bf16_normal(rng, (total_q, num_q_heads, head_dim))
    # K and V are drawn per sequence in logical (position) order, then placed
    # into their physical blocks; positions past L_b inside the last block
    # are zero.
    k_log = [_bf16_normal(rng, (int(L), num_kv_heads, head_dim)) for L in kv_lens]
    v_log = [_bf16_normal(rng, (int(L), num_kv_heads, head_dim)) for L in kv_lens]
    k_cache, v_cache = layout_cache(block_table, num_blocks, k_log, v_log, block_size)
    return Instance(
        name=name, num_seqs=B, num_q_heads=num_q_heads, num_kv_heads=num_kv_heads,
        head_dim=head_dim, block_size=block_size, scale=float(1.0 / np.sqrt(head_dim)),
        seq_kv_len=np.asarray(kv_lens, dtype=np.int32), seg_indptr=seg_indptr,
        seg_start=seg_start, seg_len=seg_len, block_table=block_table,
        num_blocks=num_blocks, q=q, k_cache=k_cache, v_cache=v_cache,
        k_logical=k_log if keep_logical else None,
        v_logical=v_log if keep_logical else None)


# ---------------------------------------------------------------------------
# layouts of the five named workloads
# ---------------------------------------------------------------------------

def _runs(blocks: np.ndarray) -> List[Tuple[int, int]]:
    """Maximal runs of consecutive block ids -> (first_block, n_blocks)."""
    out: List[Tuple[int, int]] = []
    for blk in np.sort(blocks):
        blk = int(blk)
        if out and out[-1][0] + out[-1][1] == blk:
            out[-1] = (out[-1][0], out[-1][1] + 1)
        else:
            out.append((blk, 1))
    return out


def layout_tiny(rng):
    return [512], [[(128, 64), (384, 64)]], dict(num_q_heads=4, num_kv_heads=4, head_dim=64)


def layout_llama8b(rng, batch=8, ctx=8192, tail=512, frac=0.25):
    """25% of the blocks before the final 512-token prompt are evicted; the
    evicted runs are the recompute segments; a run that reaches the prompt
    merges with it."""
    bs = BLOCK_SIZE
    nblk = ctx // bs
    tail_blk = tail // bs
    pool = nblk - tail_blk
    n_evict = int(round(frac * nblk))
    segs = []
    for _ in range(batch):
        ev = rng.choice(pool, size=n_evict, replace=False)
        ev = np.concatenate([ev, np.arange(pool, nblk)])
        segs.append([(f * bs, n * bs) for (f, n) in _runs(ev)])
    return [ctx] * batch, segs, dict(num_q_heads=32, num_kv_heads=8, head_dim=128)


def layout_fragmented(rng, batch=16, ctx=4096, nseg=64, seg_blocks=2):
    """64 block-aligned 32-token segments per sequence, uniform over the
    non-overlapping placements (stars and bars); adjacent segments stay
    separate descriptors."""
    bs = BLOCK_SIZE
    nblk = ctx // bs
    free = nblk - nseg * seg_blocks
    segs = []
    for _ in range(batch):
        c = np.sort(rng.choice(free + nseg, size=nseg, replace=False))
        starts = [int(c[k]) + k * (seg_blocks - 1) for k in range(nseg)]
        segs.append([(s * bs, seg_blocks * bs) for s in starts])
    return [ctx] * batch, segs, dict(num_q_heads=32, num_kv_heads=8, head_dim=128)


def layout_long70b(rng, batch=2, ctx=32768, num_q_heads=64, num_kv_heads=8):
    segs = [[(8192, 2048), (ctx - 4096, 4096)] for _ in range(batch)]
    return [ctx] * batch, segs, dict(num_q_heads=num_q_heads, num_kv_heads=num_kv_heads,
                                      head_dim=128)


def layout_mixed(rng, batch=32, n_prefill=8):
    """Adaptive-chunk batch: decode rows beside prefill chunks that end the
    sequence, plus 0-4 block-aligned recompute segments earlier on."""
    bs = BLOCK_SIZE
    lens = [int(x) for x in rng.integers(1024, 16384, size=batch, endpoint=True)]
    prefill = set(int(i) for i in rng.permutation(batch)[:n_prefill])
    segs = []
    for b in range(batch):
        L = lens[b]
        if b not in prefill:
            segs.append([(L - 1, 1)])
            continue
        c = min(int(rng.integers(256, 2048, endpoint=True)), L)
        k = int(rng.integers(0, 4, endpoint=True))
        room = (L - c) // bs  # recompute segments live in blocks [0, room)
        chosen: List[Tuple[int, int]] = []
        tries = 0
        while len(chosen) < k and tries < 1000:
            tries += 1
            nb = int(rng.integers(1, 16, endpoint=True))
            if nb > room:
                continue
            s = int(rng.integers(0, room - nb, endpoint=True))
            # non-overlapping and non-adjacent to every chosen segment
            if all(s + nb < f or f + n < s for (f, n) in chosen):
                chosen.append((s, nb))
        chosen.sort()
        segs.append([(f * bs, n * bs) for (f, n) in chosen] + [(L - c, c)])
    return lens, segs, dict(num_q_heads=32, num_kv_heads=8, head_dim=128)


CONFIGS = {
    1: ("tiny", layout_tiny),
    2: ("llama8b", layout_llama8b),
    3: ("fragmented", layout_fragmented),
    4: ("long70b", layout_long70b),
    5: ("mixed", layout_mixed),
}

CONFIG_DESCRIPTIONS = {
    1: "tiny: B=1, L=512, 4q/4kv, d=64, segments [128,192) and [384,448)",
    2: "llama8b: B=8, L=8192, 32q/8kv, d=128, 25% blocks evicted + 512-token prompt",
    3: "fragmented: B=16, L=4096, 32q/8kv, d=128, 64 x 32-token segments per sequence",
    4: "long70b: B=2, L=32768, 64q/8kv, d=128, [8192,10240) + 4096-token tail",
    5: "mixed: B=32, L~U[1024,16384], 32q/8kv, d=128, 24 decode + 8 prefill/recompute",
}


def fused_ablation_layout(ctx: int, cached: int, layout: str, new_tokens: int = 128):
    """Query segments of one request in the paper's fused-kernel ablation
    (Sec. 6.3): a context of ``ctx`` tokens that ends with ``new_tokens``
    uncached tokens, of which ``cached`` earlier tokens are in the cache.

    * ``"prefix"``: the cached tokens are the prefix [0, cached); one segment
      [cached, ctx) is computed.
    * ``"suffix"``: the cached tokens sit right before the new ones,
      [ctx - new - cached, ctx - new); the evicted head [0, ctx - new - cached)
      and the new tokens [ctx - new, ctx) are computed: two segments (one when
      nothing before the cached run is evicted).
    """
    assert 0 <= cached <= ctx - new_tokens
    if layout == "prefix":
        return [(cached, ctx - cached)]
    if layout == "suffix":
        head = ctx - new_tokens - cached
        return ([(0, head)] if head > 0 else []) + [(ctx - new_tokens, new_tokens)]
    raise ValueError(layout)


def cost_model_grid(seed: int, n: int, contexts=(2048, 4096, 8192, 12288, 16384),
                    new_tokens=(64, 128, 256, 512, 1024)):
    """Seeded two-segment layouts (l1, q1, l2, q2) for fitting the cost model
    of Sec. 4.3: context [l1 cached][q1 computed][l2 cached][q2 computed]; the
    context length and q2 are drawn from the given sets, the rest is cut at
    two uniform block boundaries."""
    rng = np.random.Generator(np.random.PCG64(seed))
    pts = []
    for _ in range(n):
        N = int(rng.choice(contexts))
        q2 = int(rng.choice(new_tokens))
        rest_blocks = (N - q2) // BLOCK_SIZE
        a, b = sorted(int(x) for x in rng.integers(0, rest_blocks + 1, 2))
        l1, q1 = a * BLOCK_SIZE, (b - a) * BLOCK_SIZE
        l2 = N - q2 - l1 - q1
        pts.append((l1, q1, l2, q2))
    return pts


def two_segment_layout(l1: int, q1: int, l2: int, q2: int):
    """Query segments of the cost model's layout (the q1 segment only if non-empty)."""
    return ([(l1, q1)] if q1 > 0 else []) + [(l1 + q1 + l2, q2)]


# ---------------------------------------------------------------------------
# block-cache traces for the evictor (Sec. 4.2, 4.5)
# ---------------------------------------------------------------------------

@dataclasses.dataclass
class EvictorTrace:
    """Operations recorded from a block-cache simulation (codes 0 add,
    1 remove, 2 evict, 3 lifespan), with the evicted ids the driving evictor
    returned and the cache statistics of the run."""
    op: np.ndarray
    ids: np.ndarray
    t: np.ndarray
    cost: np.ndarray
    evicted: np.ndarray
    requests: int
    hits: int
    misses: int
    capacity: int


def block_cost(index, tok_cost: float = 1.0, pair_cost: float = 1.0 / 4096,
               block_size: int = BLOCK_SIZE):
    """Synthetic recomputation cost of logical block ``index`` of a request:
    a per-token part plus attention over every earlier key, summed over the
    block's tokens (the position-linear form of Sec. 4.3).  By default
    attention costs as much as the rest of the layer at 4K context."""
    index = np.asarray(index, dtype=np.float64)
    first = index * block_size
    pairs = block_size * (first + 1) + block_size * (block_size - 1) / 2.0
    return tok_cost * block_size + pair_cost * pairs


def simulate_block_cache(evictor, seed: int, capacity: int = 8192, conversations: int = 300,
                         turns: int = 8, first_prompt=(1024, 8192), turn_tokens=(200, 2048),
                         max_tokens: int = 32768, think_time: float = 60.0,
                         span: float = 3600.0, tokens_per_s: float = 20000.0,
                         lifespan_every: int = 0) -> EvictorTrace:
    """Multi-turn serving on a cache of ``capacity`` blocks, one request at a
    time in arrival order.  Each conversation's context grows turn by turn;
    the blocks of a request are held while it runs and handed to the evictor
    (``add``) when it finishes.  A request takes its cached blocks back
    (``remove``, a hit) and gets a fresh block for every missing one,
    evicting (``evict``) when no free block is left.  Conversations start
    uniformly over ``span`` seconds; turns follow after exponential think
    times; a request runs ``tokens / tokens_per_s`` seconds.  With
    ``lifespan_every`` = k > 0, every k-th request reports the mean observed
    reuse gap as the lifespan (Sec. 5.1, Eq. 10)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    bs = BLOCK_SIZE
    arrivals = []
    for c in range(conversations):
        t = float(rng.uniform(0.0, span))
        ctx = int(rng.integers(first_prompt[0], first_prompt[1] + 1))
        for k in range(turns):
            arrivals.append((t, c, min(ctx, max_tokens)))
            t += float(rng.exponential(think_time))
            ctx += int(rng.integers(turn_tokens[0], turn_tokens[1] + 1))
    arrivals.sort()
    ops, ids, ts, costs, ev_out = [], [], [], [], []
    cached = set()
    released = {}
    free = capacity
    clock = 0.0
    hits = misses = 0
    gaps = []

    def record(o, i, t, c, e=-1):
        ops.append(o)
        ids.append(i)
        ts.append(t)
        costs.append(c)
        ev_out.append(e)

    for n_req, (t_arr, c, ctx) in enumerate(arrivals):
        clock = max(clock, t_arr)
        n = -(-ctx // bs)
        assert n <= capacity, "a request larger than the cache"
        blocks = [c * (max_tokens // bs + 1) + i for i in range(n)]
        want = []
        for b in blocks:
            if b in cached:
                evictor.remove(b)
                record(1, b, 0.0, 0.0)
                gaps.append(clock - released[b])
                hits += 1
            else:
                want.append(b)
        misses += len(want)
        while free < len(want):
            victim = evictor.evict(clock)
            record(2, -1, clock, 0.0, victim)
            cached.discard(victim)
            free += 1
        free -= len(want)
        cached.update(want)
        clock += ctx / tokens_per_s
        for i, b in enumerate(blocks):
            cost = float(block_cost(i))
            evictor.add(b, clock, cost)
            record(0, b, clock, cost)
            released[b] = clock
        if lifespan_every and (n_req + 1) % lifespan_every == 0 and gaps:
            tau = float(np.mean(gaps[-4096:]))
            evictor.set_lifespan(tau)
            record(3, -1, tau, 0.0)
    return EvictorTrace(np.asarray(ops, np.int32), np.asarray(ids, np.int64),
                        np.asarray(ts, np.float64), np.asarray(costs, np.float64),
                        np.asarray(ev_out, np.int64), len(arrivals), hits, misses, capacity)


def make_config(cfg: int, seed: Optional[int] = None, keep_logical: bool = False,
                decode_only: bool = False, **layout_kw) -> Instance:
    """Instance of named workload ``cfg`` (1..5).  Default seed = cfg.

    ``decode_only`` keeps just the sequences whose only segment is their last
    token (the decode rows of the mixed workload) with the same context
    lengths; their values are drawn afresh.
    """
    name, layout = CONFIGS[cfg]
    rng = np.random.Generator(np.random.PCG64(cfg if seed is None else seed))
    lens, segs, heads = layout(rng, **layout_kw)
    if decode_only:
        keep = [b for b in range(len(lens)) if segs[b] == [(lens[b] - 1, 1)]]
        lens = [lens[b] for b in keep]
        segs = [segs[b] for b in keep]
        name += "-decode"
    return build_instance(name, rng, lens, segs, keep_logical=keep_logical, **heads)


def make_random(seed: int, num_seqs: int = 2, num_q_heads: int = 4, num_kv_heads: int = 2,
                head_dim: int = 64, min_len: int = 1, max_len: int = 300,
                max_segs: int = 4, keep_logical: bool = True, extra_blocks: int = 0,
                aligned: bool = False, min_segs: int = 1) -> Instance:
    """Small random instance: random lengths, 0..max_segs random disjoint
    segments per sequence at arbitrary (or block-aligned) token boundaries;
    the first sequence gets at least ``min_segs`` of them."""
    rng = np.random.Generator(np.random.PCG64(seed))
    bs = BLOCK_SIZE
    lens = [int(x) for x in rng.integers(min_len, max_len, size=num_seqs, endpoint=True)]
    segs = []
    for i, L in enumerate(lens):
        lo = min(min_segs, max_segs) if i == 0 else 0
        k = int(rng.integers(lo, max_segs, endpoint=True))
        if aligned:
            nb = -(-L // bs)
            cuts = np.sort(rng.choice(nb + 1, size=min(2 * k, nb + 1), replace=False)) * bs
            cuts = np.minimum(cuts, L)
        else:
            cuts = np.sort(rng.choice(L + 1, size=min(2 * k, L + 1), replace=False))
        cur = []
        for i in range(0, len(cuts) - 1, 2):
            s, e = int(cuts[i]), int(cuts[i + 1])
            if e > s:
                cur.append((s, e - s))
        segs.append(cur)
    return build_instance(f"random{seed}", rng, lens, segs, num_q_heads, num_kv_heads,
                          head_dim, keep_logical=keep_logical, extra_blocks=extra_blocks)


def make_layout(seed: int, kv_lens: Sequence[int], segments, num_q_heads: int,
                num_kv_heads: int, head_dim: int, keep_logical: bool = True,
                extra_blocks: int = 0, permute_blocks: bool = True) -> Instance:
    """Instance for an explicit layout (edge cases)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    return build_instance(f"layout{seed}", rng, list(kv_lens), segments, num_q_heads,
                          num_kv_heads, head_dim, keep_logical=keep_logical,
                          extra_blocks=extra_blocks, permute_blocks=permute_blocks)
