"""Independent references used to pin the CPU oracle (CPU only).

Nothing here touches the oracle's code or the GPU library.  The routes are
deliberately different from the oracle's:

* ``dense_reference`` never reads the paged cache or the block table: it
  starts from the per-sequence logical K/V the generator drew, places the
  query rows at their absolute positions in a dense [L, Hq, d] tensor, and
  runs PyTorch's ``scaled_dot_product_attention(is_causal=True)`` in float64
  (a library routine for plain causal attention, Sec. 2.1 Eq. 1), with the
  K/V heads repeated G times for grouped-query attention.  The log-sum-exp
  comes from ``torch.logsumexp`` over the masked dense score matrix.
"""
from __future__ import annotations

import numpy as np
import torch

from workloads import bf16_bits_to_f32


def to_f64(bits: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(bf16_bits_to_f32(bits).astype(np.float64))


def positions_of(inst):
    """Packed row -> (sequence, absolute position), from the descriptors."""
    seq, pos = [], []
    for b in range(inst.num_seqs):
        for (s, n) in inst.segments(b):
            seq.extend([b] * n)
            pos.extend(range(s, s + n))
    return np.asarray(seq, dtype=np.int64), np.asarray(pos, dtype=np.int64)


def dense_reference(inst):
    """(o [total_q, Hq, d], lse [total_q, Hq]) in float64 via dense causal SDPA."""
    assert inst.k_logical is not None, "instance must keep its logical K/V"
    Hq, Hkv, d = inst.num_q_heads, inst.num_kv_heads, inst.head_dim
    G = Hq // Hkv
    q_all = to_f64(inst.q)
    o = torch.zeros((inst.total_q, Hq, d), dtype=torch.float64)
    lse = torch.zeros((inst.total_q, Hq), dtype=torch.float64)
    r = 0
    for b in range(inst.num_seqs):
        segs = inst.segments(b)
        pos = [s + t for (s, n) in segs for t in range(n)]
        if not pos:
            continue
        L = int(inst.seq_kv_len[b])
        n = len(pos)
        qd = torch.zeros((L, Hq, d), dtype=torch.float64)
        qd[pos] = q_all[r:r + n]
        k = to_f64(inst.k_logical[b]).repeat_interleave(G, dim=1)  # [L, Hq, d]
        v = to_f64(inst.v_logical[b]).repeat_interleave(G, dim=1)
        qh, kh, vh = (x.permute(1, 0, 2).unsqueeze(0) for x in (qd, k, v))
        out = torch.nn.functional.scaled_dot_product_attention(
            qh, kh, vh, is_causal=True, scale=inst.scale)[0]      # [Hq, L, d]
        scores = inst.scale * torch.matmul(qh[0], kh[0].transpose(1, 2))  # [Hq, L, L]
        causal = torch.ones((L, L), dtype=torch.bool).tril()
        scores = scores.masked_fill(~causal, float("-inf"))
        l = torch.logsumexp(scores, dim=-1)                        # [Hq, L]
        idx = torch.tensor(pos)
        o[r:r + n] = out[:, idx, :].permute(1, 0, 2)
        lse[r:r + n] = l[:, idx].permute(1, 0)
        r += n
    return o.numpy(), lse.numpy()


def repermute(inst, seed: int):
    """Same logical content, different physical block ids (and block table)."""
    import copy
    rng = np.random.Generator(np.random.PCG64(seed))
    new = copy.copy(inst)
    nb = inst.num_blocks
    perm = rng.permutation(nb)            # old physical id -> new physical id
    k = np.empty_like(inst.k_cache)
    v = np.empty_like(inst.v_cache)
    k[perm] = inst.k_cache
    v[perm] = inst.v_cache
    bt = inst.block_table.copy()
    m = bt >= 0
    bt[m] = perm[bt[m]]
    new.k_cache, new.v_cache, new.block_table = k, v, bt
    return new


def split_segments(inst, seed: int):
    """Split every segment of length >= 2 into two adjacent segments."""
    import copy
    rng = np.random.Generator(np.random.PCG64(seed))
    starts, lens, indptr = [], [], [0]
    for b in range(inst.num_seqs):
        for (s, n) in inst.segments(b):
            if n >= 2:
                c = int(rng.integers(1, n))
                starts += [s, s + c]
                lens += [c, n - c]
            else:
                starts.append(s)
                lens.append(n)
        indptr.append(len(starts))
    new = copy.copy(inst)
    new.seg_start = np.asarray(starts, dtype=np.int32)
    new.seg_len = np.asarray(lens, dtype=np.int32)
    new.seg_indptr = np.asarray(indptr, dtype=np.int32)
    return new
