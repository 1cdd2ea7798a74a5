"""Multi-Segment Attention (MSA) for AMD Instinct MI355X (gfx950).

Thin ctypes binding of ``libmsa.so`` (C ABI in ``include/msa.h``).  It only
marshals arguments: planning runs in the library's C++ planner and every
step of the attention runs in the library's HIP kernels.  There is no CPU
fallback: importing this package without a built library raises.

Functions carry the C names: ``msa_plan``, ``msa_plan_info``,
``msa_forward``, ``msa_kv_append``, ``msa_plan_destroy``,
``msa_last_error``, ``msa_plan_export``, ``msa_check_block_table``,
``msa_forward_noalloc``.  Device buffers are passed as objects with a
``data_ptr()`` method (e.g. torch tensors) or as integer addresses; streams
as ``hipStream_t`` integers or objects with ``cuda_stream`` (torch streams).
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# MSA_LIBRARY names another build of the same library (the host-sanitizer
# test loads an instrumented build of the planner this way)
LIB_PATH = os.environ.get("MSA_LIBRARY") or os.path.join(_HERE, "libmsa.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2606_02964_amd.build`")
# Device buffers and streams come from PyTorch: load it first so that the
# library binds to the HIP runtime torch already holds (a second runtime in
# the process would see other streams, and possibly no device).
try:
    import torch  # noqa: F401
except ImportError:  # plain C users: the system HIP runtime
    pass
_lib = ctypes.CDLL(LIB_PATH)

MSA_OK = 0
MSA_ERR_INVALID_ARG = 1
MSA_ERR_UNSUPPORTED = 2
MSA_ERR_OUT_OF_MEMORY = 3
MSA_ERR_DEVICE = 4
MSA_PLAN_HOST_ONLY = 1
MSA_PLAN_NO_AUTO_SPLIT = 2
MSA_PLAN_TILE_ROWS_128 = 4
MSA_PLAN_TILE_ROWS_256 = 8
MSA_PLAN_TILE_ROWS_32 = 16
MSA_PLAN_PRECISE_WEIGHTS = 32
MSA_TABLE_HOST = 0
MSA_TABLE_DEVICE = 1
MSA_NOALLOC_WORKSPACE_BYTES = 64 << 20

_i32, _i64, _f32, _f64, _P = ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_double, ctypes.c_void_p


class msa_shape(ctypes.Structure):
    _fields_ = [("num_seqs", _i32), ("num_q_heads", _i32), ("num_kv_heads", _i32),
                ("head_dim", _i32), ("block_size", _i32), ("max_blocks_per_seq", _i32),
                ("num_blocks", _i32), ("scale", _f32),
                ("q_stride_tok", _i64), ("q_stride_head", _i64),
                ("o_stride_tok", _i64), ("o_stride_head", _i64),
                ("k_stride_block", _i64), ("k_stride_head", _i64), ("k_stride_tok", _i64),
                ("v_stride_block", _i64), ("v_stride_head", _i64), ("v_stride_dim", _i64)]


class msa_plan_opts(ctypes.Structure):
    _fields_ = [("q_tile_tokens", _i32), ("kv_split_tokens", _i32), ("flags", _i32),
                ("reserved", _i32 * 5)]


class msa_plan_info_t(ctypes.Structure):
    _fields_ = [("total_q", _i64), ("num_work", _i64), ("num_tiles", _i64), ("num_merge", _i64),
                ("max_splits", _i64), ("workspace_bytes", _i64), ("useful_flops", _f64),
                ("tile_flops", _f64), ("planned_bytes", _f64), ("min_bytes", _f64),
                ("tile_rows", _i64), ("num_workgroups", _i64)]

    def as_dict(self):
        return {name: getattr(self, name) for name, _ in self._fields_}


_lib.msa_plan.restype = _i32
_lib.msa_plan.argtypes = [ctypes.POINTER(msa_shape), _P, _P, _P, _P,
                          ctypes.POINTER(msa_plan_opts), _P, ctypes.POINTER(_P)]
_lib.msa_plan_info.restype = _i32
_lib.msa_plan_info.argtypes = [_P, ctypes.POINTER(msa_plan_info_t)]
_lib.msa_forward.restype = _i32
_lib.msa_forward.argtypes = [_P, _P, _P, _P, _P, _P, _P, _P, ctypes.c_size_t, _P]
_lib.msa_kv_append.restype = _i32
_lib.msa_kv_append.argtypes = [_P, _P, _P, _i64, _i64, _i64, _i64, _P, _P, _P, _P]
_lib.msa_plan_destroy.restype = None
_lib.msa_plan_destroy.argtypes = [_P]
_lib.msa_last_error.restype = ctypes.c_char_p
_lib.msa_last_error.argtypes = []
_lib.msa_plan_export.restype = _i32
_lib.msa_plan_export.argtypes = [_P, _P, _P, _P]
_lib.msa_forward_noalloc.restype = _i32
_lib.msa_forward_noalloc.argtypes = [_P, _P, _P, _P, _P, _P, _P, _P]
_lib.msa_check_block_table.restype = _i32
_lib.msa_check_block_table.argtypes = [_P, _P, _i32, _P]

_lib.msa_evictor_create.restype = _i32
_lib.msa_evictor_create.argtypes = [_P, ctypes.POINTER(_P)]
_lib.msa_evictor_destroy.restype = None
_lib.msa_evictor_destroy.argtypes = [_P]
_lib.msa_evictor_add.restype = _i32
_lib.msa_evictor_add.argtypes = [_P, _i64, _f64, _f64]
_lib.msa_evictor_remove.restype = _i32
_lib.msa_evictor_remove.argtypes = [_P, _i64]
_lib.msa_evictor_evict.restype = _i32
_lib.msa_evictor_evict.argtypes = [_P, _f64, ctypes.POINTER(_i64)]
_lib.msa_evictor_set_lambda.restype = _i32
_lib.msa_evictor_set_lambda.argtypes = [_P, _f64]
_lib.msa_evictor_set_lifespan.restype = _i32
_lib.msa_evictor_set_lifespan.argtypes = [_P, _f64, ctypes.POINTER(_f64)]
_lib.msa_evictor_size.restype = _i64
_lib.msa_evictor_size.argtypes = [_P]
_lib.msa_evictor_log_weight.restype = _i32
_lib.msa_evictor_log_weight.argtypes = [_P, _i64, _f64, ctypes.POINTER(_f64)]
_lib.msa_evictor_replay.restype = _i32
_lib.msa_evictor_replay.argtypes = [_P, _i64, _P, _P, _P, _P, _P, ctypes.POINTER(_i64)]

EXPORTED = ("msa_plan", "msa_plan_info", "msa_forward", "msa_kv_append", "msa_plan_destroy",
            "msa_last_error", "msa_plan_export", "msa_check_block_table", "msa_forward_noalloc",
            "msa_evictor_create", "msa_evictor_destroy", "msa_evictor_add", "msa_evictor_remove",
            "msa_evictor_evict", "msa_evictor_set_lambda", "msa_evictor_set_lifespan",
            "msa_evictor_size", "msa_evictor_log_weight", "msa_evictor_replay")

MSA_EVICTOR_LINEAR = 1
EVICTOR_OP_ADD, EVICTOR_OP_REMOVE, EVICTOR_OP_EVICT, EVICTOR_OP_LIFESPAN = 0, 1, 2, 3


class MsaError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"[status {status}] {message}")
        self.status = status


def _check(status: int):
    if status != MSA_OK:
        raise MsaError(status, msa_last_error())


def _addr(x) -> Optional[int]:
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return int(x.data_ptr())


def _stream(s) -> Optional[int]:
    if s is None:
        try:
            import torch
            return int(torch.cuda.current_stream().cuda_stream)
        except Exception:
            return None
    if isinstance(s, int):
        return s
    return int(s.cuda_stream)


def _host_i32(a) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(a), dtype=np.int32)


def msa_last_error() -> str:
    return _lib.msa_last_error().decode()


class Plan:
    """Owning wrapper of an ``msa_plan_t`` handle."""

    def __init__(self, handle: int, shape: msa_shape):
        self.handle = handle
        self.shape = shape

    def info(self) -> dict:
        return msa_plan_info(self)

    def close(self):
        if self.handle:
            _lib.msa_plan_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def msa_plan(shape: msa_shape, seq_kv_len: Sequence[int], seg_indptr: Sequence[int],
             seg_start: Sequence[int], seg_len: Sequence[int], q_tile_tokens: int = 0,
             kv_split_tokens: int = 0, flags: int = 0, stream=None) -> Plan:
    """Validate the descriptors and build a plan (host arrays in, plan out)."""
    kv = _host_i32(seq_kv_len)
    ip = _host_i32(seg_indptr)
    ss = _host_i32(seg_start)
    sl = _host_i32(seg_len)
    opts = msa_plan_opts(q_tile_tokens, kv_split_tokens, flags)
    handle = _P()
    st = _lib.msa_plan(ctypes.byref(shape), kv.ctypes.data, ip.ctypes.data,
                       ss.ctypes.data if ss.size else None, sl.ctypes.data if sl.size else None,
                       ctypes.byref(opts), None if flags & MSA_PLAN_HOST_ONLY else _stream(stream),
                       ctypes.byref(handle))
    _check(st)
    return Plan(handle.value, shape)


def msa_plan_info(plan: Plan) -> dict:
    info = msa_plan_info_t()
    _check(_lib.msa_plan_info(plan.handle, ctypes.byref(info)))
    return info.as_dict()


def msa_plan_export(plan: Plan):
    """(row_pos [total_q], work [num_work, 8], merge [num_merge, 8]) as int32 arrays."""
    info = msa_plan_info(plan)
    row_pos = np.zeros(info["total_q"], np.int32)
    work = np.zeros((info["num_work"], 8), np.int32)
    merge = np.zeros((info["num_merge"], 8), np.int32)
    _check(_lib.msa_plan_export(plan.handle, row_pos.ctypes.data if row_pos.size else None,
                                work.ctypes.data if work.size else None,
                                merge.ctypes.data if merge.size else None))
    return row_pos, work, merge


def msa_check_block_table(plan: Plan, block_table, stream=None) -> None:
    """Debug check of the block-table entries the plan reads (raises MsaError
    naming the first bad entry).  A numpy array is checked as a host table,
    anything else (a device tensor, an integer address) as a device table."""
    if isinstance(block_table, np.ndarray):
        bt = np.ascontiguousarray(block_table, dtype=np.int32)
        _check(_lib.msa_check_block_table(plan.handle, bt.ctypes.data if bt.size else None,
                                          MSA_TABLE_HOST, None))
    else:
        _check(_lib.msa_check_block_table(plan.handle, _addr(block_table), MSA_TABLE_DEVICE,
                                          _stream(stream)))


def msa_forward(plan: Plan, q, k_cache, v_cache, block_table, o, lse=None, workspace=None,
                workspace_bytes: int = 0, stream=None) -> None:
    """Enqueue MSA for one layer on ``stream`` (torch's current stream if None)."""
    if workspace is not None and not workspace_bytes:
        workspace_bytes = int(workspace.numel() * workspace.element_size())
    _check(_lib.msa_forward(plan.handle, _addr(q), _addr(k_cache), _addr(v_cache),
                            _addr(block_table), _addr(o), _addr(lse), _addr(workspace),
                            int(workspace_bytes), _stream(stream)))


def msa_forward_noalloc(plan: Plan, q, k_cache, v_cache, block_table, o, lse=None,
                        stream=None) -> None:
    """msa_forward with the library's own scratch workspace (no allocation;
    calls that overlap on one device race, see include/msa.h)."""
    _check(_lib.msa_forward_noalloc(plan.handle, _addr(q), _addr(k_cache), _addr(v_cache),
                                    _addr(block_table), _addr(o), _addr(lse), _stream(stream)))


def msa_kv_append(plan: Plan, k_new, v_new, block_table, k_cache, v_cache,
                  k_new_strides=None, v_new_strides=None, stream=None) -> None:
    """Enqueue the write of the rows' fresh K/V ([total_q, Hkv, d]) into the paged cache.

    Strides (tok, head) in elements default to those of a tensor argument
    (``.stride()``), else to the contiguous layout."""
    def strides(x, given):
        if given is not None:
            return int(given[0]), int(given[1])
        if hasattr(x, "stride"):
            st = x.stride()
            return int(st[0]), int(st[1])
        sh = plan.shape
        if sh is None:  # no plan: the library reports that
            return 0, 0
        return sh.num_kv_heads * sh.head_dim, sh.head_dim
    kst, ksh = strides(k_new, k_new_strides)
    vst, vsh = strides(v_new, v_new_strides)
    _check(_lib.msa_kv_append(plan.handle, _addr(k_new), _addr(v_new), kst, ksh, vst, vsh,
                              _addr(block_table), _addr(k_cache), _addr(v_cache), _stream(stream)))


def msa_plan_destroy(plan: Plan) -> None:
    plan.close()


def make_shape(num_seqs: int, num_q_heads: int, num_kv_heads: int, head_dim: int,
               max_blocks_per_seq: int, num_blocks: int, scale: float,
               q_strides=None, o_strides=None, k_strides=None, v_strides=None,
               block_size: int = 16) -> msa_shape:
    """msa_shape with contiguous defaults: q/o [total_q, Hq, d], K [blocks, Hkv, bs, d],
    V [blocks, Hkv, d, bs].  Strides are (tok, head), (block, head, tok), (block, head, dim)."""
    d, bs = head_dim, block_size
    qs = q_strides or (num_q_heads * d, d)
    os_ = o_strides or (num_q_heads * d, d)
    ks = k_strides or (num_kv_heads * bs * d, bs * d, d)
    vs = v_strides or (num_kv_heads * d * bs, d * bs, bs)
    return msa_shape(num_seqs, num_q_heads, num_kv_heads, head_dim, block_size,
                     max_blocks_per_seq, num_blocks, scale, qs[0], qs[1], os_[0], os_[1],
                     ks[0], ks[1], ks[2], vs[0], vs[1], vs[2])


class msa_evictor_params(ctypes.Structure):
    _fields_ = [("alpha", _f64), ("beta", _f64), ("tau0", _f64), ("lambda_", _f64),
                ("flags", _i32), ("reserved", _i32 * 3)]


class Evictor:
    """Owning wrapper of an ``msa_evictor_t`` (include/msa_evictor.h): the
    computation-aware block evictor (Sec. 4.2, Alg. 1)."""

    def __init__(self, alpha: float, beta: float, tau0: float, lam: float = 1.0,
                 linear: bool = False):
        params = msa_evictor_params(alpha, beta, tau0, lam, MSA_EVICTOR_LINEAR if linear else 0)
        h = _P()
        _check(_lib.msa_evictor_create(ctypes.byref(params), ctypes.byref(h)))
        self.handle = h.value

    def close(self):
        if getattr(self, "handle", None):
            _lib.msa_evictor_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def add(self, block_id: int, t_last: float, cost: float) -> None:
        _check(_lib.msa_evictor_add(self.handle, int(block_id), float(t_last), float(cost)))

    def remove(self, block_id: int) -> None:
        _check(_lib.msa_evictor_remove(self.handle, int(block_id)))

    def evict(self, t_now: float) -> int:
        out = _i64()
        _check(_lib.msa_evictor_evict(self.handle, float(t_now), ctypes.byref(out)))
        return out.value

    def set_lambda(self, lam: float) -> None:
        _check(_lib.msa_evictor_set_lambda(self.handle, float(lam)))

    def set_lifespan(self, tau: float) -> float:
        out = _f64()
        _check(_lib.msa_evictor_set_lifespan(self.handle, float(tau), ctypes.byref(out)))
        return out.value

    def __len__(self) -> int:
        return int(_lib.msa_evictor_size(self.handle))

    def log_weight(self, block_id: int, t: float) -> float:
        out = _f64()
        _check(_lib.msa_evictor_log_weight(self.handle, int(block_id), float(t), ctypes.byref(out)))
        return out.value

    def replay(self, op, ids, t, cost) -> np.ndarray:
        """Apply a trace (codes EVICTOR_OP_*); returns the evicted id per op (-1 otherwise)."""
        c = np.ascontiguousarray
        op, ids = c(op, dtype=np.int32), c(ids, dtype=np.int64)
        t, cost = c(t, dtype=np.float64), c(cost, dtype=np.float64)
        n = op.shape[0]
        out = np.empty(n, dtype=np.int64)
        failed = _i64()
        st = _lib.msa_evictor_replay(self.handle, n, op.ctypes.data, ids.ctypes.data,
                                     t.ctypes.data, cost.ctypes.data, out.ctypes.data,
                                     ctypes.byref(failed))
        if st != MSA_OK:
            raise MsaError(st, f"op {failed.value}: {msa_last_error()}")
        return out
