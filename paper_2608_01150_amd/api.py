"""Thin Python binding of the C ABI in include/zl_attn.h (ctypes).

Argument marshalling only: tensors become raw device pointers, the current
torch stream becomes the hipStream_t, descriptors become ``zl_seg_desc``.
Every computation runs in the HIP library; if it is not built, importing this
module raises.  PyTorch supplies device memory and streams.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional, Sequence

import numpy as np
import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libzl_attn.so")

ZL_OK, ZL_ERR_INVALID_ARG, ZL_ERR_UNSUPPORTED, ZL_ERR_WORKSPACE, ZL_ERR_HIP, ZL_ERR_INFEASIBLE = range(6)
ZL_WHOLE, ZL_SHARD = 0, 1
ZL_BF16, ZL_FP32 = 0, 1
ZL_OP_FWD, ZL_OP_BWD, ZL_OP_BWD_DQ = 0, 1, 2
ZL_STEP_FIRST, ZL_STEP_LAST = 1, 2


class ZlError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"zl status {status}: {message}")
        self.status = status


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build the HIP library first (python -c "
                          "'import __graft_entry__ as g; g.build()')")
    return ctypes.CDLL(LIB_PATH)


_lib = _load()

_i32p = ctypes.POINTER(ctypes.c_int32)
_i64p = ctypes.POINTER(ctypes.c_int64)
_u8p = ctypes.POINTER(ctypes.c_uint8)
_vp = ctypes.c_void_p


class _CDesc(ctypes.Structure):
    _fields_ = [
        ("num_q_segs", ctypes.c_int32),
        ("cu_seqlens_q", _i32p),
        ("kind", _u8p),
        ("q_offset", _i64p),
        ("kv_first", _i32p),
        ("kv_count", _i32p),
        ("num_kv_ranges", ctypes.c_int32),
        ("cu_seqlens_k", _i32p),
        ("k_offset", _i64p),
        ("block_index", _i32p),
        ("num_slots", ctypes.c_int32),
    ]


def _sig(name, res, *args):
    fn = getattr(_lib, name)
    fn.restype = res
    fn.argtypes = list(args)
    return fn


_DP = ctypes.POINTER(_CDesc)
_abi_version = _sig("zl_abi_version", ctypes.c_int32)
_last_error = _sig("zl_last_error", ctypes.c_char_p)
_workspace_size = _sig("zl_workspace_size", ctypes.c_int, _DP, ctypes.c_int32, ctypes.c_int32, ctypes.c_int,
                       ctypes.c_int32, ctypes.POINTER(ctypes.c_size_t))
_fwd = _sig("zl_attn_fwd", ctypes.c_int, _DP, ctypes.c_int32, ctypes.c_int32, ctypes.c_int, ctypes.c_float,
            _vp, _vp, _vp, _vp, _vp, _vp, _vp, ctypes.c_int32, _vp)
_fwd_ex = _sig("zl_attn_fwd_ex", ctypes.c_int, _DP, ctypes.c_int32, ctypes.c_int32, ctypes.c_int, ctypes.c_float,
               _vp, _vp, _vp, _vp, _vp, _vp, ctypes.c_int, _vp, ctypes.c_int32, _vp)
_fwd_step = _sig("zl_attn_fwd_step", ctypes.c_int, _DP, ctypes.c_int32, ctypes.c_int32, ctypes.c_int, ctypes.c_float,
                 _vp, _vp, _vp, _vp, _vp, _vp, _vp, ctypes.c_uint32, _vp)
_u_pack_qkv = _sig("zl_ulysses_pack_qkv", ctypes.c_int, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                   ctypes.c_int, _vp, _vp, _vp, _vp, _vp)
_u_unpack_qkv = _sig("zl_ulysses_unpack_qkv", ctypes.c_int, ctypes.c_int32, ctypes.c_int32, _i32p, ctypes.c_int32,
                     ctypes.c_int32, ctypes.c_int, _vp, _vp, _vp, _vp, _vp)
_u_pack_out = _sig("zl_ulysses_pack_out", ctypes.c_int, ctypes.c_int32, ctypes.c_int32, _i32p, ctypes.c_int32,
                   ctypes.c_int32, ctypes.c_int, _vp, _vp, _vp)
_u_unpack_out = _sig("zl_ulysses_unpack_out", ctypes.c_int, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                     ctypes.c_int32, ctypes.c_int, _vp, _vp, _vp)
_merge = _sig("zl_lse_merge", ctypes.c_int, _DP, ctypes.c_int32, ctypes.c_int32, ctypes.c_int, _vp, _vp,
              ctypes.c_int32, _vp, _vp, _vp)
_merge_ex = _sig("zl_lse_merge_ex", ctypes.c_int, _DP, ctypes.c_int32, ctypes.c_int32, ctypes.c_int, _vp, ctypes.c_int,
                 _vp, ctypes.c_int32, _vp, _vp, _vp)
_bwd = _sig("zl_attn_bwd", ctypes.c_int, _DP, ctypes.c_int32, ctypes.c_int32, ctypes.c_int, ctypes.c_float,
            _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, ctypes.c_uint32, _vp, ctypes.c_size_t, _vp)
_bwd_noalloc = _sig("zl_attn_bwd_noalloc", ctypes.c_int, _DP, ctypes.c_int32, ctypes.c_int32, ctypes.c_int,
                    ctypes.c_float, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp)
_bwd_step = _sig("zl_attn_bwd_step", ctypes.c_int, _DP, ctypes.c_int32, ctypes.c_int32, ctypes.c_int, ctypes.c_float,
                 _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, ctypes.c_uint32, _vp, ctypes.c_size_t, _vp)
_plan_dump = _sig("zl_plan_dump", ctypes.c_int, _DP, ctypes.c_int32, ctypes.c_int32, ctypes.c_int, ctypes.c_int32,
                  _i32p, ctypes.c_size_t, ctypes.POINTER(ctypes.c_size_t), _i32p, _i32p)
_f64p = ctypes.POINTER(ctypes.c_double)
_fill_pack = _sig("zl_fill_pack", ctypes.c_int, ctypes.c_int32, ctypes.c_int32, _f64p, _f64p, ctypes.c_double,
                  ctypes.c_double, _f64p, _f64p, _i32p, ctypes.POINTER(ctypes.c_int32))
_shutdown = _sig("zl_shutdown", None)
_prof_enable = _sig("zl_profile_enable", ctypes.c_int, ctypes.c_int32)
_prof_read = _sig("zl_profile_read", ctypes.c_int, ctypes.c_int32, ctypes.POINTER(ctypes.c_double),
                  ctypes.POINTER(ctypes.c_int64))
_prof_reset = _sig("zl_profile_reset", None)

ZL_K_FWD, ZL_K_MERGE, ZL_K_BWD_PRE, ZL_K_BWD_DKDV, ZL_K_BWD_DQ, ZL_K_ULYSSES = range(6)
KERNEL_NAMES = {ZL_K_FWD: "fwd", ZL_K_MERGE: "merge", ZL_K_BWD_PRE: "bwd_pre", ZL_K_BWD_DKDV: "bwd_dkdv",
                ZL_K_BWD_DQ: "bwd_dq", ZL_K_ULYSSES: "ulysses"}


def profile_enable(on: bool) -> None:
    _check(_prof_enable(1 if on else 0))


def profile_reset() -> None:
    _prof_reset()


def profile_read(kernel_id: int):
    """(total milliseconds, launches) of one kernel family since the last reset."""
    ms, n = ctypes.c_double(0), ctypes.c_int64(0)
    _check(_prof_read(kernel_id, ctypes.byref(ms), ctypes.byref(n)))
    return ms.value, n.value


def abi_version() -> int:
    return int(_abi_version())


def last_error() -> str:
    return _last_error().decode()


def shutdown() -> None:
    _shutdown()


def _check(st: int) -> None:
    if st != ZL_OK:
        raise ZlError(st, last_error())


class SegDesc:
    """Host-side ``zl_seg_desc`` with its arrays kept alive.

    Built from any object with the descriptor fields (a ``Workload``, a dict
    wrapper) or from keyword arrays.  ``q_offset`` / ``k_offset`` may be None.
    """

    def __init__(self, cu_seqlens_q, kind, kv_first, kv_count, cu_seqlens_k, block_index, num_slots,
                 q_offset=None, k_offset=None):
        self._a = {
            "cu_seqlens_q": np.ascontiguousarray(cu_seqlens_q, dtype=np.int32),
            "kind": np.ascontiguousarray(kind, dtype=np.uint8),
            "kv_first": np.ascontiguousarray(kv_first, dtype=np.int32),
            "kv_count": np.ascontiguousarray(kv_count, dtype=np.int32),
            "cu_seqlens_k": np.ascontiguousarray(cu_seqlens_k, dtype=np.int32),
            "block_index": np.ascontiguousarray(block_index, dtype=np.int32),
        }
        if q_offset is not None:
            self._a["q_offset"] = np.ascontiguousarray(q_offset, dtype=np.int64)
        if k_offset is not None:
            self._a["k_offset"] = np.ascontiguousarray(k_offset, dtype=np.int64)
        a = self._a
        self.c = _CDesc()
        self.c.num_q_segs = len(a["kind"])
        self.c.num_kv_ranges = len(a["cu_seqlens_k"]) - 1
        self.c.num_slots = int(num_slots)
        for name, ptype in (("cu_seqlens_q", _i32p), ("kind", _u8p), ("kv_first", _i32p), ("kv_count", _i32p),
                            ("cu_seqlens_k", _i32p), ("block_index", _i32p), ("q_offset", _i64p),
                            ("k_offset", _i64p)):
            arr = a.get(name)
            setattr(self.c, name, arr.ctypes.data_as(ptype) if arr is not None and arr.size else ptype())
        self.num_slots = int(num_slots)
        self.total_q = int(a["cu_seqlens_q"][-1])
        self.total_k = int(a["cu_seqlens_k"][-1])
        # one past the last packed row of any SHARD segment: the rows a ring
        # accumulator must cover
        ends = [int(a["cu_seqlens_q"][s + 1]) for s in range(len(a["kind"])) if int(a["kind"][s]) == ZL_SHARD]
        self.shard_rows_end = max(ends, default=0)

    @classmethod
    def of(cls, w) -> "SegDesc":
        get = (lambda n: w[n]) if isinstance(w, dict) else (lambda n: getattr(w, n))
        return cls(get("cu_seqlens_q"), get("kind"), get("kv_first"), get("kv_count"), get("cu_seqlens_k"),
                   get("block_index"), get("num_slots"), q_offset=get("q_offset"), k_offset=get("k_offset"))

    def ptr(self):
        return ctypes.byref(self.c)


def _dtype_code(t: torch.dtype) -> int:
    if t == torch.bfloat16:
        return ZL_BF16
    if t == torch.float32:
        return ZL_FP32
    raise ZlError(ZL_ERR_UNSUPPORTED, f"dtype {t} unsupported")


def _p(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_contiguous():
        raise ZlError(ZL_ERR_INVALID_ARG, "tensors must be contiguous")
    return t.data_ptr()


def _need(t: Optional[torch.Tensor], name: str, shape, dtype: torch.dtype, min_rows: bool = False) -> None:
    """Raises ZlError unless `t` (when given) has `shape` (with min_rows: at
    least shape[0] rows and the rest equal) and `dtype`.  The library reads
    and writes through raw pointers whose extents follow from the descriptor,
    so a mismatched tensor must be stopped here."""
    if t is None:
        return
    shape = tuple(int(x) for x in shape)
    got = tuple(t.shape)
    if min_rows:
        ok = len(got) == len(shape) and got[1:] == shape[1:] and got[0] >= shape[0]
    else:
        ok = got == shape
    if not ok:
        want = f"at least {shape[0]} rows of {shape[1:]}" if min_rows else str(shape)
        raise ZlError(ZL_ERR_INVALID_ARG, f"{name} has shape {got}, expected {want}")
    if t.dtype != dtype:
        raise ZlError(ZL_ERR_INVALID_ARG, f"{name} has dtype {t.dtype}, expected {dtype}")


def _same_gpu(*ts) -> torch.device:
    """The one CUDA device every given tensor is on (raises otherwise)."""
    devs = {t.device for t in ts if t is not None}
    if len(devs) != 1 or next(iter(devs)).type != "cuda":
        raise ZlError(ZL_ERR_INVALID_ARG, f"tensors must all be on one GPU (got {sorted(map(str, devs))})")
    return next(iter(devs))


def _qkv(desc: SegDesc, q, k, v):
    """Checks q [Tq, H, d] and k, v [Tk, H, d] against the descriptor; returns (H, d)."""
    if q.dim() != 3:
        raise ZlError(ZL_ERR_INVALID_ARG, f"q must be [Tq, H, d], got shape {tuple(q.shape)}")
    _, h, d = q.shape
    _need(q, "q", (desc.total_q, h, d), q.dtype)
    _need(k, "k", (desc.total_k, h, d), q.dtype)
    _need(v, "v", (desc.total_k, h, d), q.dtype)
    return h, d


def _stream(device) -> int:
    return torch.cuda.current_stream(device).cuda_stream


def workspace_size(desc: SegDesc, num_heads: int, head_dim: int, dtype: torch.dtype, op: int) -> int:
    n = ctypes.c_size_t(0)
    _check(_workspace_size(desc.ptr(), num_heads, head_dim, _dtype_code(dtype), op, ctypes.byref(n)))
    return int(n.value)


def plan_dump(desc: SegDesc, num_heads: int, head_dim: int, dtype: torch.dtype, op: int):
    """Work items of a launch in issue order: int32 [n, 8] and (tile_m, tile_n)."""
    n = ctypes.c_size_t(0)
    tm, tn = ctypes.c_int32(0), ctypes.c_int32(0)
    _check(_plan_dump(desc.ptr(), num_heads, head_dim, _dtype_code(dtype), op, None, 0, ctypes.byref(n),
                      ctypes.byref(tm), ctypes.byref(tn)))
    items = np.zeros((int(n.value), 8), dtype=np.int32)
    if items.size:
        _check(_plan_dump(desc.ptr(), num_heads, head_dim, _dtype_code(dtype), op, items.ctypes.data_as(_i32p),
                          items.shape[0], ctypes.byref(n), None, None))
    return items, (tm.value, tn.value)


def fill_pack(price, mem, load, mem_used, load_floor: float, mem_cap: float):
    """zl_fill_pack (Filler Packing, Eq. 8) on host arrays.

    price [n], mem [n, N], load [N] and mem_used [N] (the ledgers after anchor
    placement).  Returns (rank_of int32 [n], load [N], mem_used [N], failed),
    failed = index of the first filler that fit nowhere, or None.  Raises
    ZlError for invalid arguments.
    """
    price = np.ascontiguousarray(price, dtype=np.float64)
    n = price.shape[0]
    ld = np.array(load, dtype=np.float64)
    mu = np.array(mem_used, dtype=np.float64)
    N = ld.shape[0]
    mem = np.ascontiguousarray(np.asarray(mem, dtype=np.float64).reshape(n, N))
    rank_of = np.full(n, -1, dtype=np.int32)
    failed = ctypes.c_int32(-1)
    st = _fill_pack(N, n, price.ctypes.data_as(_f64p), mem.ctypes.data_as(_f64p), float(load_floor), float(mem_cap),
                    ld.ctypes.data_as(_f64p), mu.ctypes.data_as(_f64p), rank_of.ctypes.data_as(_i32p),
                    ctypes.byref(failed))
    if st not in (ZL_OK, ZL_ERR_INFEASIBLE):
        _check(st)
    return rank_of, ld, mu, (None if failed.value < 0 else int(failed.value))


def attn_fwd(desc: SegDesc, q, k, v, scale: float, out=None, lse=None, o_part=None, lse_part=None,
             part_dtype: Optional[torch.dtype] = None):
    """zl_attn_fwd (fp32 partials) or zl_attn_fwd_ex (bf16 partials).  The partials' dtype is o_part's,
    else part_dtype (default fp32).  Allocates the outputs it is not given; returns (out, lse, o_part,
    lse_part)."""
    h, d = _qkv(desc, q, k, v)
    tq = desc.total_q
    pdt = o_part.dtype if o_part is not None else (part_dtype or torch.float32)
    if pdt not in (torch.float32, torch.bfloat16):
        raise ZlError(ZL_ERR_INVALID_ARG, f"partials must be float32 or bfloat16, got {pdt}")
    _need(out, "out", (tq, h, d), q.dtype)
    _need(lse, "lse", (tq, h), torch.float32)
    _need(o_part, "o_part", (desc.num_slots, tq, h, d), pdt)
    _need(lse_part, "lse_part", (desc.num_slots, tq, h), torch.float32)
    dev = _same_gpu(q, k, v, out, lse, o_part, lse_part)
    if out is None:
        out = torch.empty_like(q)
    if lse is None:
        lse = torch.empty((tq, h), dtype=torch.float32, device=dev)
    if o_part is None and desc.num_slots > 0:
        o_part = torch.empty((desc.num_slots, tq, h, d), dtype=pdt, device=dev)
    if lse_part is None and desc.num_slots > 0:
        lse_part = torch.empty((desc.num_slots, tq, h), dtype=torch.float32, device=dev)
    if pdt == torch.float32:
        _check(_fwd(desc.ptr(), h, d, _dtype_code(q.dtype), float(scale), _p(q), _p(k), _p(v), _p(out), _p(lse),
                    _p(o_part), _p(lse_part), desc.num_slots, _stream(dev)))
    else:
        _check(_fwd_ex(desc.ptr(), h, d, _dtype_code(q.dtype), float(scale), _p(q), _p(k), _p(v), _p(out), _p(lse),
                       _p(o_part), ZL_BF16, _p(lse_part), desc.num_slots, _stream(dev)))
    return out, lse, o_part, lse_part


def attn_fwd_step(desc: SegDesc, q, k, v, scale: float, out, lse, o_acc, lse_acc, flags: int):
    """zl_attn_fwd_step: one ring step; SHARD rows fold this call's block into (o_acc, lse_acc), and with
    ZL_STEP_LAST write the final out / lse.  Every tensor is caller-provided (o_acc / lse_acc may be None only
    when no SHARD rows need them)."""
    h, d = _qkv(desc, q, k, v)
    tq, r = desc.total_q, desc.shard_rows_end
    _need(out, "out", (tq, h, d), q.dtype)
    _need(lse, "lse", (tq, h), torch.float32)
    _need(o_acc, "o_acc", (r, h, d), torch.float32, min_rows=True)
    _need(lse_acc, "lse_acc", (r, h), torch.float32, min_rows=True)
    _same_gpu(q, k, v, out, lse, o_acc, lse_acc)
    _check(_fwd_step(desc.ptr(), h, d, _dtype_code(q.dtype), float(scale), _p(q), _p(k), _p(v), _p(out), _p(lse),
                     _p(o_acc), _p(lse_acc), int(flags), _stream(q.device)))
    return out, lse


def _cu_rank(cu_rank):
    a = np.ascontiguousarray(np.asarray(cu_rank, dtype=np.int32))
    if a.ndim != 2:
        raise ZlError(ZL_ERR_INVALID_ARG, "cu_rank must be [group, num_seqs + 1]")
    return a


def ulysses_pack_qkv(group: int, q, k, v, send=None):
    """zl_ulysses_pack_qkv: local q, k, v [T, H, d] -> send [group, T, H/group, 3, d]."""
    if q.dim() != 3:
        raise ZlError(ZL_ERR_INVALID_ARG, f"q must be [T, H, d], got shape {tuple(q.shape)}")
    t, h, d = q.shape
    if send is None and group >= 1 and h % group == 0:
        send = torch.empty((group, t, h // group, 3, d), dtype=q.dtype, device=q.device)
    if group >= 1 and h % group == 0:  # otherwise the library reports the bad group
        _need(k, "k", (t, h, d), q.dtype)
        _need(v, "v", (t, h, d), q.dtype)
        _need(send, "send", (group, t, h // group, 3, d), q.dtype)
        _same_gpu(q, k, v, send)
    _check(_u_pack_qkv(group, t, h, d, _dtype_code(q.dtype), _p(q), _p(k), _p(v), _p(send), _stream(q.device)))
    return send


def ulysses_unpack_qkv(group: int, cu_rank, recv, num_heads: int, q=None, k=None, v=None):
    """zl_ulysses_unpack_qkv: rank-major recv [T_full, H/group, 3, d] -> q, k, v [T_full, H/group, d]."""
    cu = _cu_rank(cu_rank)
    if recv.dim() != 4:
        raise ZlError(ZL_ERR_INVALID_ARG, f"recv must be [T_full, H/group, 3, d], got shape {tuple(recv.shape)}")
    tf, hl, _, d = recv.shape
    q = torch.empty((tf, hl, d), dtype=recv.dtype, device=recv.device) if q is None else q
    k = torch.empty_like(q) if k is None else k
    v = torch.empty_like(q) if v is None else v
    if group >= 1 and num_heads % group == 0 and cu.shape[0] == group:
        t_full = int(cu[:, -1].sum())
        _need(recv, "recv", (t_full, num_heads // group, 3, d), recv.dtype)
        for t, name in ((q, "q"), (k, "k"), (v, "v")):
            _need(t, name, (t_full, num_heads // group, d), recv.dtype)
        _same_gpu(recv, q, k, v)
    _check(_u_unpack_qkv(group, cu.shape[1] - 1, cu.ctypes.data_as(_i32p), num_heads, d, _dtype_code(recv.dtype),
                         _p(recv), _p(q), _p(k), _p(v), _stream(recv.device)))
    return q, k, v


def ulysses_pack_out(group: int, cu_rank, out, num_heads: int, send=None):
    """zl_ulysses_pack_out: out [T_full, H/group, d] -> rank-major send [T_full, H/group, d]."""
    cu = _cu_rank(cu_rank)
    if out.dim() != 3:
        raise ZlError(ZL_ERR_INVALID_ARG, f"out must be [T_full, H/group, d], got shape {tuple(out.shape)}")
    send = torch.empty_like(out) if send is None else send
    if group >= 1 and num_heads % group == 0 and cu.shape[0] == group:
        shape = (int(cu[:, -1].sum()), num_heads // group, out.shape[2])
        _need(out, "out", shape, out.dtype)
        _need(send, "send", shape, out.dtype)
        _same_gpu(out, send)
    _check(_u_pack_out(group, cu.shape[1] - 1, cu.ctypes.data_as(_i32p), num_heads, out.shape[2],
                       _dtype_code(out.dtype), _p(out), _p(send), _stream(out.device)))
    return send


def ulysses_unpack_out(group: int, recv, num_heads: int, out_local=None):
    """zl_ulysses_unpack_out: recv [group, T, H/group, d] -> out_local [T, H, d]."""
    if recv.dim() != 4:
        raise ZlError(ZL_ERR_INVALID_ARG, f"recv must be [group, T, H/group, d], got shape {tuple(recv.shape)}")
    g, t, hl, d = recv.shape
    if out_local is None:
        out_local = torch.empty((t, num_heads, d), dtype=recv.dtype, device=recv.device)
    if group >= 1 and num_heads % group == 0:
        _need(recv, "recv", (group, t, num_heads // group, d), recv.dtype)
        _need(out_local, "out_local", (t, num_heads, d), recv.dtype)
        _same_gpu(recv, out_local)
    _check(_u_unpack_out(group, t, num_heads, d, _dtype_code(recv.dtype), _p(recv), _p(out_local),
                         _stream(recv.device)))
    return out_local


def lse_merge(desc: SegDesc, o_part, lse_part, out, lse):
    """zl_lse_merge (zl_lse_merge_ex for bf16 o_part): writes the SHARD rows of out / lse."""
    if out.dim() != 3:
        raise ZlError(ZL_ERR_INVALID_ARG, f"out must be [Tq, H, d], got shape {tuple(out.shape)}")
    _, h, d = out.shape
    tq = desc.total_q
    _need(out, "out", (tq, h, d), out.dtype)
    _need(lse, "lse", (tq, h), torch.float32)
    pdt = o_part.dtype if o_part is not None else torch.float32
    if pdt not in (torch.float32, torch.bfloat16):
        raise ZlError(ZL_ERR_INVALID_ARG, f"partials must be float32 or bfloat16, got {pdt}")
    _need(o_part, "o_part", (desc.num_slots, tq, h, d), pdt)
    _need(lse_part, "lse_part", (desc.num_slots, tq, h), torch.float32)
    _same_gpu(out, lse, o_part, lse_part)
    if pdt == torch.float32:
        _check(_merge(desc.ptr(), h, d, _dtype_code(out.dtype), _p(o_part), _p(lse_part), desc.num_slots, _p(out),
                      _p(lse), _stream(out.device)))
    else:
        _check(_merge_ex(desc.ptr(), h, d, _dtype_code(out.dtype), _p(o_part), ZL_BF16, _p(lse_part), desc.num_slots,
                         _p(out), _p(lse), _stream(out.device)))
    return out, lse


def attn_bwd(desc: SegDesc, q, k, v, out, lse, dout, scale: float, dq=None, dk=None, dv=None, workspace=None):
    """zl_attn_bwd.  Allocates dq/dk/dv/workspace it is not given; returns (dq, dk, dv)."""
    h, d = _qkv(desc, q, k, v)
    tq, tk = desc.total_q, desc.total_k
    for t, name in ((out, "out"), (dout, "dout"), (dq, "dq")):
        _need(t, name, (tq, h, d), q.dtype)
    for t, name in ((dk, "dk"), (dv, "dv")):
        _need(t, name, (tk, h, d), q.dtype)
    _need(lse, "lse", (tq, h), torch.float32)
    dev = _same_gpu(q, k, v, out, lse, dout, dq, dk, dv, workspace)
    dq = torch.empty_like(q) if dq is None else dq
    dk = torch.zeros_like(k) if dk is None else dk
    dv = torch.zeros_like(v) if dv is None else dv
    if workspace is None:
        workspace = torch.empty(workspace_size(desc, h, d, q.dtype, ZL_OP_BWD), dtype=torch.uint8, device=dev)
    _check(_bwd(desc.ptr(), h, d, _dtype_code(q.dtype), float(scale), _p(q), _p(k), _p(v), _p(out), _p(lse),
                _p(dout), _p(dq), _p(dk), _p(dv), 0, _p(workspace), workspace.numel() * workspace.element_size(), _stream(dev)))
    return dq, dk, dv


def attn_bwd_noalloc(desc: SegDesc, q, k, v, out, lse, dout, scale: float, dq, dk, dv):
    """zl_attn_bwd_noalloc: zl_attn_bwd with no allocation anywhere (the library's static scratch
    holds its tables and workspace).  Every output is caller-provided; returns (dq, dk, dv)."""
    h, d = _qkv(desc, q, k, v)
    tq, tk = desc.total_q, desc.total_k
    for t, name in ((out, "out"), (dout, "dout"), (dq, "dq")):
        _need(t, name, (tq, h, d), q.dtype)
    for t, name in ((dk, "dk"), (dv, "dv")):
        _need(t, name, (tk, h, d), q.dtype)
    _need(lse, "lse", (tq, h), torch.float32)
    dev = _same_gpu(q, k, v, out, lse, dout, dq, dk, dv)
    _check(_bwd_noalloc(desc.ptr(), h, d, _dtype_code(q.dtype), float(scale), _p(q), _p(k), _p(v), _p(out), _p(lse),
                        _p(dout), _p(dq), _p(dk), _p(dv), _stream(dev)))
    return dq, dk, dv


def attn_bwd_step(desc: SegDesc, q, k, v, out, lse, dout, scale: float, dq, dk, dv, dq_acc, flags: int,
                  workspace=None):
    """zl_attn_bwd_step: one ring step of the backward (see the header); returns (dq, dk, dv)."""
    h, d = _qkv(desc, q, k, v)
    tq, tk = desc.total_q, desc.total_k
    for t, name in ((out, "out"), (dout, "dout"), (dq, "dq")):
        _need(t, name, (tq, h, d), q.dtype)
    for t, name in ((dk, "dk"), (dv, "dv")):
        _need(t, name, (tk, h, d), q.dtype)
    _need(lse, "lse", (tq, h), torch.float32)
    _need(dq_acc, "dq_acc", (desc.shard_rows_end, h, d), torch.float32, min_rows=True)
    _same_gpu(q, k, v, out, lse, dout, dq, dk, dv, dq_acc, workspace)
    if workspace is None:
        workspace = torch.empty(workspace_size(desc, h, d, q.dtype, ZL_OP_BWD), dtype=torch.uint8, device=q.device)
    _check(_bwd_step(desc.ptr(), h, d, _dtype_code(q.dtype), float(scale), _p(q), _p(k), _p(v), _p(out), _p(lse),
                     _p(dout), _p(dq), _p(dk), _p(dv), _p(dq_acc), int(flags), _p(workspace), workspace.numel() * workspace.element_size(),
                     _stream(q.device)))
    return dq, dk, dv


def header_symbols(header_path: Optional[str] = None) -> Sequence[str]:
    """Function names declared in include/zl_attn.h."""
    import re
    if header_path is None:
        header_path = os.path.join(os.path.dirname(_PKG), "include", "zl_attn.h")
    text = open(header_path).read()
    return sorted(set(re.findall(r"\b(zl_[a-z_]+)\s*\(", text)))
