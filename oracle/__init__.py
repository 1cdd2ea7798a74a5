"""CPU oracle for Multi-Segment Attention -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the benchmark's CPU-baseline
leg may import this package.  The product (``paper_2606_02964_amd``) never
does, and this package never imports the product.

``kv_append`` is the paged cache write of the rows' fresh K/V (Sec. 4.1, 5.3).
``evictor_replay`` is the block-eviction policy (Sec. 4.2, Eq. 3, Eq. 9,
Alg. 1's lambda, Eq. 10) evaluated by scanning every block at each eviction.
``forward`` is exact MSA (Sec. 2.1 Eq. 1 + Sec. 4.1 Eq. 2, causal by absolute
position, GQA grouping h -> h / (Hq/Hkv)), computed in IEEE double by the
plain C routine in ``msa_oracle.c``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Tuple

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "msa_oracle.c")
_SRC_EVICTOR = os.path.join(_HERE, "evictor_oracle.c")
# MSA_ORACLE_LIBRARY names another build of the same oracle (the
# host-sanitizer test loads an instrumented build this way)
_LIB = os.environ.get("MSA_ORACLE_LIBRARY") or os.path.join(_HERE, "libmsa_oracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (no fast-math, no FMA contraction)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
                               "-fno-fast-math", "-pthread", _SRC, _SRC_EVICTOR, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def load_library(path: str):
    """ctypes handle on an oracle shared library at ``path``."""
    lib = ctypes.CDLL(path)
    _declare(lib)
    return lib


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=True)
        _lib = load_library(_LIB)
    return _lib


def _declare(lib):
    P = ctypes.c_void_p
    i32, i64, f64 = ctypes.c_int32, ctypes.c_int64, ctypes.c_double
    lib.msa_oracle_forward.restype = ctypes.c_int
    lib.msa_oracle_forward.argtypes = [
        i32, i32, i32, i32, i32, i32, i32, f64,  # shapes, scale
        P, P, P, P,                              # seq_kv_len, seg_indptr, seg_start, seg_len
        P, i64, i64,                             # q
        P, i64, i64, i64,                        # k cache
        P, i64, i64, i64,                        # v cache
        P,                                       # block table
        P, P, i64,                               # items
        P, P, i32]                               # outputs, threads
    lib.msa_oracle_kv_append.restype = ctypes.c_int
    lib.msa_oracle_kv_append.argtypes = [
        i32, i32, i32, i32, i32, i32,            # shapes
        P, P, P, P,                              # seq_kv_len, seg_indptr, seg_start, seg_len
        P, i64, i64,                             # k_new
        P, i64, i64,                             # v_new
        P, i64, i64, i64,                        # k cache (written)
        P, i64, i64, i64,                        # v cache (written)
        P]                                       # block table
    if hasattr(lib, "msa_oracle_evictor_replay"):  # absent from single-file test builds
        lib.msa_oracle_evictor_replay.restype = i64
        lib.msa_oracle_evictor_replay.argtypes = [f64, f64, f64, f64, i64, P, P, P, P, P]
    lib.msa_oracle_total_rows.restype = i64
    lib.msa_oracle_total_rows.argtypes = [i32, P, P]


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def default_threads() -> int:
    return max(1, len(os.sched_getaffinity(0)))


def forward(inst, rows: Optional[np.ndarray] = None, heads: Optional[np.ndarray] = None,
            num_threads: Optional[int] = None, lib=None) -> Tuple[np.ndarray, np.ndarray]:
    """Exact MSA in float64.

    Without ``rows``/``heads``: returns o [total_q, Hq, d], lse [total_q, Hq].
    With them (equal-length int arrays): o [n, d], lse [n] for the items
    (rows[i], heads[i]).  ``lib`` overrides the library handle (tests load
    deliberately broken copies to show that the pins catch them).
    """
    lib = _load() if lib is None else lib
    c = np.ascontiguousarray
    seq_kv_len = c(inst.seq_kv_len, dtype=np.int32)
    seg_indptr = c(inst.seg_indptr, dtype=np.int32)
    seg_start = c(inst.seg_start, dtype=np.int32)
    seg_len = c(inst.seg_len, dtype=np.int32)
    q = c(inst.q, dtype=np.uint16)
    k = c(inst.k_cache, dtype=np.uint16)
    v = c(inst.v_cache, dtype=np.uint16)
    bt = c(inst.block_table, dtype=np.int32)
    B, Hq, Hkv, d = inst.num_seqs, inst.num_q_heads, inst.num_kv_heads, inst.head_dim
    total = int(seg_len.sum())
    assert q.shape == (total, Hq, d)
    assert k.ndim == 4 and v.ndim == 4
    if rows is None:
        n = total * Hq
        item_row = item_head = None
        o = np.empty((total, Hq, d), dtype=np.float64)
        lse = np.empty((total, Hq), dtype=np.float64)
    else:
        item_row = c(rows, dtype=np.int64)
        item_head = c(heads, dtype=np.int32)
        assert item_row.shape == item_head.shape and item_row.ndim == 1
        n = item_row.shape[0]
        o = np.empty((n, d), dtype=np.float64)
        lse = np.empty((n,), dtype=np.float64)
    if num_threads is None:
        num_threads = default_threads()
    rc = lib.msa_oracle_forward(
        B, Hq, Hkv, d, inst.block_size, bt.shape[1], k.shape[0], float(inst.scale),
        _ptr(seq_kv_len), _ptr(seg_indptr), _ptr(seg_start), _ptr(seg_len),
        _ptr(q), Hq * d, d,
        _ptr(k), Hkv * k.shape[2] * d, k.shape[2] * d, d,
        _ptr(v), Hkv * d * v.shape[3], d * v.shape[3], v.shape[3],
        _ptr(bt),
        _ptr(item_row) if item_row is not None else None,
        _ptr(item_head) if item_head is not None else None,
        n, _ptr(o), _ptr(lse), int(num_threads))
    if rc != 0:
        raise ValueError(f"msa_oracle_forward rejected its inputs (code {rc})")
    return o, lse


def kv_append(inst, k_new: np.ndarray, v_new: np.ndarray, lib=None) -> Tuple[np.ndarray, np.ndarray]:
    """Paged cache write of the rows' K/V: returns copies of ``inst``'s caches
    with k_new / v_new ([total_q, Hkv, d] bf16 bits) stored at every row's
    absolute position.  ``inst``'s own caches are not modified."""
    lib = _load() if lib is None else lib
    c = np.ascontiguousarray
    seq_kv_len = c(inst.seq_kv_len, dtype=np.int32)
    seg_indptr = c(inst.seg_indptr, dtype=np.int32)
    seg_start = c(inst.seg_start, dtype=np.int32)
    seg_len = c(inst.seg_len, dtype=np.int32)
    kn = c(k_new, dtype=np.uint16)
    vn = c(v_new, dtype=np.uint16)
    k = np.array(inst.k_cache, dtype=np.uint16, copy=True, order="C")
    v = np.array(inst.v_cache, dtype=np.uint16, copy=True, order="C")
    bt = c(inst.block_table, dtype=np.int32)
    Hkv, d = inst.num_kv_heads, inst.head_dim
    total = int(seg_len.sum())
    assert kn.shape == (total, Hkv, d) and vn.shape == (total, Hkv, d)
    rc = lib.msa_oracle_kv_append(
        inst.num_seqs, Hkv, d, inst.block_size, bt.shape[1], k.shape[0],
        _ptr(seq_kv_len), _ptr(seg_indptr), _ptr(seg_start), _ptr(seg_len),
        _ptr(kn), Hkv * d, d, _ptr(vn), Hkv * d, d,
        _ptr(k), Hkv * k.shape[2] * d, k.shape[2] * d, d,
        _ptr(v), Hkv * d * v.shape[3], d * v.shape[3], v.shape[3],
        _ptr(bt))
    if rc != 0:
        raise ValueError(f"msa_oracle_kv_append rejected its inputs (code {rc})")
    return k, v


def evictor_replay(alpha: float, beta: float, tau0: float, lam: float, op, ids, t, cost,
                   lib=None) -> np.ndarray:
    """Replay evictor operations (codes 0 add, 1 remove, 2 evict, 3 lifespan);
    returns the evicted id per op (-1 for non-evict ops).  Raises ValueError
    naming the first operation the definition cannot apply."""
    lib = _load() if lib is None else lib
    c = np.ascontiguousarray
    op = c(op, dtype=np.int32)
    ids = c(ids, dtype=np.int64)
    t = c(t, dtype=np.float64)
    cost = c(cost, dtype=np.float64)
    n = op.shape[0]
    assert ids.shape == t.shape == cost.shape == (n,)
    out = np.empty(n, dtype=np.int64)
    rc = lib.msa_oracle_evictor_replay(float(alpha), float(beta), float(tau0), float(lam), n,
                                       _ptr(op), _ptr(ids), _ptr(t), _ptr(cost), _ptr(out))
    if rc != 0:
        raise ValueError(f"msa_oracle_evictor_replay: operation {rc - 1} cannot be applied")
    return out
