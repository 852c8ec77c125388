"""Topology-biased graph attention for AMD Instinct MI355X (gfx950).

Thin Python binding of libgtattn.so. Every function here only marshals
arguments: it checks tensors, allocates outputs with torch (device memory
only) and calls the C ABI of the same name on the current HIP stream. All
computation runs in the library's HIP kernels; there is no fallback path.
If the library is missing or cannot be loaded, every call raises.

    o, lse = gt_attn_fwd(q, k, v, spd, table)                     # [H,N,d], [H,N]
    dq, dk, dv, dtable = gt_attn_bwd(q, k, v, spd, table, o, lse, d_o)
    o, lse = gt_attn_fwd_batch(q_b, k_b, v_b, spd_b, table)      # [B,H,N,d], spd [B,N,N]
    o_p, lse_p = gt_attn_ring_step(q_sh, k_sh, v_sh, spd_shard, row_off, col_off, table)
    o, lse = gt_attn_merge(o_parts, lse_parts, dtype=torch.bfloat16)
    state = gt_attn_ring_step(...)                      # first step: a running state
    gt_attn_ring_step_acc(q_sh, k_sh, v_sh, spd_shard, row_off, col_off, table, state)
    dq, dk, dv, dt = gt_attn_bwd_ring_step(q_sh, o_sh, lse_sh, do_sh, k_blk, v_blk, spd_shard,
                                           row_off, col_off, table, acc=(dq, dk, dv, dt))
"""
from __future__ import annotations

import ctypes
import math
from pathlib import Path

import torch

__all__ = ["gt_attn_fwd", "gt_attn_bwd", "gt_attn_bwd_phase", "gt_attn_bwd_noalloc",
           "gt_attn_bwd_noalloc_max_bytes", "gt_attn_ring_step",
           "gt_attn_ring_step_acc", "gt_attn_merge",
           "gt_attn_bwd_ring_step", "gt_attn_bwd_workspace_size", "gt_attn_bwd_ring_workspace_size",
           "gt_status_string", "gt_attn_version",
           "GTError", "lib", "LIB_PATH"]

LIB_PATH = Path(__file__).resolve().parent / "libgtattn.so"

GT_F32, GT_BF16 = 0, 1
_STATUS = {0: "GT_OK", 1: "GT_ERR_INVALID", 2: "GT_ERR_UNSUPPORTED", 3: "GT_ERR_WORKSPACE",
           4: "GT_ERR_LAUNCH"}


class GTError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what}: {_STATUS.get(status, status)} ({gt_status_string(status)})")


_lib = None
_P = ctypes.c_void_p
_I32 = ctypes.c_int32
_I64 = ctypes.c_int64
_F = ctypes.c_float


def lib() -> ctypes.CDLL:
    """The loaded libgtattn.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not LIB_PATH.exists():
            raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() "
                              "or python -m paper_2609_34420_amd.build_lib")
        L = ctypes.CDLL(str(LIB_PATH))
        L.gt_attn_fwd.restype = _I32
        L.gt_attn_fwd.argtypes = [_P, _P, _P, _P, _P, _I32, _P, _P, _I32, _I64, _I32, _I32, _F, _P]
        L.gt_attn_bwd_workspace_size.restype = ctypes.c_size_t
        L.gt_attn_bwd_workspace_size.argtypes = [_I32, _I64, _I32, _I32]
        L.gt_attn_bwd.restype = _I32
        L.gt_attn_bwd.argtypes = [_P, _P, _P, _P, _P, _P, _I32, _P, _P, _P, _P, _P, _P, _P, _P,
                                  ctypes.c_size_t, _I32, _I64, _I32, _I32, _F, _P]
        L.gt_attn_bwd_noalloc.restype = _I32
        L.gt_attn_bwd_noalloc.argtypes = [_P, _P, _P, _P, _P, _P, _I32, _P, _P, _P, _P, _P, _P, _P,
                                          _I32, _I64, _I32, _I32, _F, _P]
        L.gt_attn_bwd_noalloc_max_bytes.restype = ctypes.c_size_t
        L.gt_attn_bwd_noalloc_max_bytes.argtypes = []
        L.gt_attn_bwd_phase.restype = _I32
        L.gt_attn_bwd_phase.argtypes = [_I32] + L.gt_attn_bwd.argtypes
        L.gt_attn_ring_step.restype = _I32
        L.gt_attn_ring_step.argtypes = [_P, _I64, _P, _P, _I64, _P, _I64, _I64, _I64, _P, _I32,
                                        _P, _P, _I32, _I32, _I32, _F, _P]
        L.gt_attn_ring_step_acc.restype = _I32
        L.gt_attn_ring_step_acc.argtypes = L.gt_attn_ring_step.argtypes
        L.gt_attn_fwd_batch.restype = _I32
        L.gt_attn_fwd_batch.argtypes = [_P, _P, _P, _P, _I64, _P, _I32, _P, _P, _I32, _I32, _I64,
                                        _I32, _I32, _F, _P]
        L.gt_attn_bwd_batch.restype = _I32
        L.gt_attn_bwd_batch.argtypes = [_P, _P, _P, _P, _P, _I64, _P, _I32, _P, _P, _P, _P, _P, _P,
                                        _P, _P, ctypes.c_size_t, _I32, _I32, _I64, _I32, _I32, _F,
                                        _P]
        L.gt_attn_bwd_ring_workspace_size.restype = ctypes.c_size_t
        L.gt_attn_bwd_ring_workspace_size.argtypes = [_I32, _I64, _I64, _I32, _I32]
        L.gt_attn_bwd_ring_step.restype = _I32
        L.gt_attn_bwd_ring_step.argtypes = [_P, _P, _P, _P, _I64, _P, _P, _I64, _P, _I64, _I64, _I64,
                                            _P, _I32, _P, _P, _P, _P, _P, ctypes.c_size_t,
                                            _I32, _I32, _I32, _F, _P]
        L.gt_attn_merge.restype = _I32
        L.gt_attn_merge.argtypes = [_P, _P, _I32, _P, _P, _I32, _I64, _I32, _I32, _P]
        L.gt_status_string.restype = ctypes.c_char_p
        L.gt_status_string.argtypes = [_I32]
        L.gt_attn_version.restype = _I32
        L.gt_attn_version.argtypes = []
        _lib = L
    return _lib


def gt_status_string(status: int) -> str:
    return lib().gt_status_string(int(status)).decode()


def gt_attn_version() -> int:
    return int(lib().gt_attn_version())


def _dt(x: torch.Tensor) -> int:
    if x.dtype == torch.bfloat16:
        return GT_BF16
    if x.dtype == torch.float32:
        return GT_F32
    raise TypeError(f"unsupported dtype {x.dtype}")


def _ptr(x) -> int | None:
    return None if x is None else x.data_ptr()


def _stream(stream) -> int | None:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


def _check(status: int, what: str):
    if status != 0:
        raise GTError(status, what)


def _need(cond: bool, msg: str):
    if not cond:
        raise ValueError(msg)


# Argument checks. Every entry point checks each tensor's shape and dtype
# against q (and table) first, then that all tensors are contiguous tensors
# on q's device, all before anything is launched: a wrong shape raises
# ValueError instead of becoming an out-of-bounds device access.

_HEAD_DIMS = (8, 16, 32, 64)


def _shape(t, name: str, shape, dtype=None):
    _need(isinstance(t, torch.Tensor), f"{name} must be a tensor")
    _need(tuple(t.shape) == tuple(shape), f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if dtype is not None:
        _need(t.dtype == dtype, f"{name} must be {dtype}, got {t.dtype}")


def _qdims(q, name: str, ndim: int):
    _need(isinstance(q, torch.Tensor) and q.dim() == ndim, f"{name} must be a {ndim}-D tensor")
    _need(q.dtype in (torch.bfloat16, torch.float32), f"{name} must be bfloat16 or float32, got {q.dtype}")
    _need(q.shape[-1] in _HEAD_DIMS, f"head dim must be one of {_HEAD_DIMS}, got {q.shape[-1]}")
    _need(all(n >= 1 for n in q.shape), f"{name} must not be empty")
    return q.dtype


def _table(table, H: int):
    _need(isinstance(table, torch.Tensor) and table.dim() == 2 and table.shape[0] == H
          and table.dtype == torch.float32, f"table must be fp32 [H={H}, n_buckets]")
    _need(1 <= table.shape[1] <= 256, f"table must have 1..256 buckets, got {table.shape[1]}")


def _devices(ref, *ts, contiguous=True):
    """Every tensor is a device tensor on ref's device (and contiguous)."""
    _need(ref.is_cuda, "tensors must be device tensors")
    for t in ts:
        if t is None:
            continue
        _need(t.is_cuda and t.device == ref.device, "tensors must be device tensors on one device")
        if contiguous:
            _need(t.is_contiguous(), "tensors must be contiguous")


def _spd_view(spd, rows_needed: int, cols_needed: int, name: str = "spd"):
    """A 2-D uint8 spd shard with unit column stride that holds rows
    [0, rows_needed) and columns [0, cols_needed) of what the step reads
    (the row stride is passed on as ld_spd, so a column-sliced view must
    not let the step read past its last column)."""
    _need(isinstance(spd, torch.Tensor) and spd.dtype == torch.uint8 and spd.dim() == 2
          and spd.stride(1) == 1, f"{name} must be a uint8 2-D tensor with unit column stride")
    _need(rows_needed <= spd.shape[0], f"{name} has {spd.shape[0]} rows; the step reads rows up to {rows_needed}")
    _need(cols_needed <= spd.shape[1],
          f"{name} has {spd.shape[1]} columns; the step reads columns up to {cols_needed}")


def _workspace(ws, need: int, ref):
    _need(isinstance(ws, torch.Tensor) and ws.dtype == torch.uint8 and ws.dim() == 1
          and ws.is_contiguous(), "workspace must be a contiguous uint8 1-D tensor")
    _need(ws.numel() >= need, f"workspace holds {ws.numel()} bytes; {need} are needed")
    _need(ws.is_cuda and ws.device == ref.device, "workspace must be on the tensors' device")
    _need(ws.data_ptr() % 256 == 0, "workspace must be 256-byte aligned")


def gt_attn_fwd(q, k, v, spd, table, scale: float | None = None, out=None, lse=None,
                stream=None):
    """O, LSE of biased attention over all N nodes (C ABI gt_attn_fwd).
    q, k, v [H, N, d] bf16|fp32; spd [N, N] uint8; table [H, n_buckets] fp32."""
    dt = _qdims(q, "q", 3)
    H, N, d = q.shape
    _shape(k, "k", q.shape, dt)
    _shape(v, "v", q.shape, dt)
    _shape(spd, "spd", (N, N), torch.uint8)
    _table(table, H)
    if out is not None:
        _shape(out, "out", q.shape, dt)
    if lse is not None:
        _shape(lse, "lse", (H, N), torch.float32)
    _devices(q, k, v, spd, table, out, lse)
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    if out is None:
        out = torch.empty_like(q)
    if lse is None:
        lse = torch.empty((H, N), device=q.device, dtype=torch.float32)
    st = lib().gt_attn_fwd(_ptr(q), _ptr(k), _ptr(v), _ptr(spd), _ptr(table), table.shape[1],
                           _ptr(out), _ptr(lse), H, N, d, _dt(q), scale, _stream(stream))
    _check(st, "gt_attn_fwd")
    return out, lse


def gt_attn_bwd_workspace_size(H: int, N: int, d: int, dtype=torch.bfloat16) -> int:
    return int(lib().gt_attn_bwd_workspace_size(H, N, d, GT_BF16 if dtype == torch.bfloat16 else GT_F32))


def gt_attn_bwd(q, k, v, spd, table, o, lse, d_o, scale: float | None = None,
                workspace=None, grads=None, stream=None, spd_t=None):
    """dQ, dK, dV, dTable (C ABI gt_attn_bwd). `grads` may hold preallocated
    (dq, dk, dv, dtable); `workspace` a uint8 device tensor of at least
    gt_attn_bwd_workspace_size bytes; `spd_t` the transpose of spd (spd itself
    for a symmetric matrix) or None."""
    return gt_attn_bwd_phase(-1, q, k, v, spd, table, o, lse, d_o, scale, workspace, grads, stream,
                             spd_t)


def _check_bwd(q, k, v, spd, table, o, lse, d_o, grads, spd_t, lead):
    """Shapes of a (batched) backward: q [*lead, N, d]; spd [N, N] (or
    [B, N, N] / [N, N] for a batch, checked by the caller)."""
    dt = q.dtype
    N = q.shape[-2]
    for name, t in (("k", k), ("v", v), ("o", o), ("d_o", d_o)):
        _shape(t, name, q.shape, dt)
    _shape(lse, "lse", tuple(q.shape[:-1]), torch.float32)
    H = q.shape[-3]
    _table(table, H)
    if spd_t is not None:
        _need(isinstance(spd_t, torch.Tensor) and tuple(spd_t.shape) == tuple(spd.shape)
              and spd_t.dtype == spd.dtype and spd_t.stride() == spd.stride(),
              "spd_t must have the shape and layout of spd")
    if grads is not None:
        _need(len(grads) == 4, "grads must be (dq, dk, dv, dtable)")
        for name, t in zip(("dq", "dk", "dv"), grads[:3]):
            _shape(t, name, q.shape, dt)
        _shape(grads[3], "dtable", table.shape, torch.float32)
    return N


def gt_attn_bwd_phase(phase: int, q, k, v, spd, table, o, lse, d_o, scale: float | None = None,
                      workspace=None, grads=None, stream=None, spd_t=None):
    """One stage of the backward (C ABI gt_attn_bwd_phase): 0 prepare,
    1 dK/dV/dtable, 2 dQ; phase -1 runs gt_attn_bwd (all three)."""
    _need(phase in (-1, 0, 1, 2), f"phase must be -1, 0, 1 or 2, got {phase}")
    _qdims(q, "q", 3)
    H, N, d = q.shape
    _shape(spd, "spd", (N, N), torch.uint8)
    _check_bwd(q, k, v, spd, table, o, lse, d_o, grads, spd_t, (H,))
    need = gt_attn_bwd_workspace_size(H, N, d, q.dtype)
    _devices(q, k, v, spd, table, o, lse, d_o, spd_t, *(grads or ()))
    if workspace is not None:
        _workspace(workspace, need, q)
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    if grads is None:
        grads = (torch.empty_like(q), torch.empty_like(k), torch.empty_like(v),
                 torch.empty_like(table))
    dq, dk, dv, dtable = grads
    if workspace is None:
        workspace = torch.empty(need, device=q.device, dtype=torch.uint8)
    args = (_ptr(q), _ptr(k), _ptr(v), _ptr(spd), None if spd_t is None else _ptr(spd_t),
            _ptr(table), table.shape[1],
            _ptr(o), _ptr(lse), _ptr(d_o), _ptr(dq), _ptr(dk), _ptr(dv),
            _ptr(dtable), _ptr(workspace), workspace.numel() * workspace.element_size(),
            H, N, d, _dt(q), scale, _stream(stream))
    if phase == -1:
        _check(lib().gt_attn_bwd(*args), "gt_attn_bwd")
    else:
        _check(lib().gt_attn_bwd_phase(int(phase), *args), "gt_attn_bwd_phase")
    return dq, dk, dv, dtable


def gt_attn_bwd_noalloc_max_bytes() -> int:
    return int(lib().gt_attn_bwd_noalloc_max_bytes())


def gt_attn_bwd_noalloc(q, k, v, spd, table, o, lse, d_o, grads, scale: float | None = None,
                        stream=None, spd_t=None):
    """gt_attn_bwd with the library's fixed device scratch instead of a
    workspace (C ABI gt_attn_bwd_noalloc): the call allocates nothing, so the
    outputs `grads` = (dq, dk, dv, dtable) must be given. Calls that overlap
    on one GPU share the scratch and race."""
    _qdims(q, "q", 3)
    H, N, d = q.shape
    _shape(spd, "spd", (N, N), torch.uint8)
    _need(grads is not None, "grads (dq, dk, dv, dtable) must be given: the call allocates nothing")
    _check_bwd(q, k, v, spd, table, o, lse, d_o, grads, spd_t, (H,))
    _devices(q, k, v, spd, table, o, lse, d_o, spd_t, *grads)
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    dq, dk, dv, dtable = grads
    st = lib().gt_attn_bwd_noalloc(_ptr(q), _ptr(k), _ptr(v), _ptr(spd),
                                   None if spd_t is None else _ptr(spd_t), _ptr(table),
                                   table.shape[1], _ptr(o), _ptr(lse), _ptr(d_o), _ptr(dq), _ptr(dk),
                                   _ptr(dv), _ptr(dtable), H, N, d, _dt(q), scale, _stream(stream))
    _check(st, "gt_attn_bwd_noalloc")
    return dq, dk, dv, dtable


def _batch_spd(spd, B, N):
    _need(isinstance(spd, torch.Tensor) and spd.dtype == torch.uint8 and spd.dim() in (2, 3)
          and tuple(spd.shape[-2:]) == (N, N), "spd must be uint8 [B, N, N] or [N, N] (shared by the batch)")
    if spd.dim() == 2:
        return 0
    _need(spd.shape[0] == B, "spd must hold one [N, N] matrix per graph")
    return spd.stride(0) if B > 1 else 0


def gt_attn_fwd_batch(q, k, v, spd, table, scale: float | None = None, out=None, lse=None,
                      stream=None):
    """O, LSE of a batch of graphs (C ABI gt_attn_fwd_batch). q, k, v
    [B, H, N, d]; spd [B, N, N] uint8 (or [N, N] shared); table [H, nb]."""
    dt = _qdims(q, "q", 4)
    B, H, N, d = q.shape
    _shape(k, "k", q.shape, dt)
    _shape(v, "v", q.shape, dt)
    stride = _batch_spd(spd, B, N)
    _table(table, H)
    if out is not None:
        _shape(out, "out", q.shape, dt)
    if lse is not None:
        _shape(lse, "lse", (B, H, N), torch.float32)
    _devices(q, k, v, spd, table, out, lse)
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    if out is None:
        out = torch.empty_like(q)
    if lse is None:
        lse = torch.empty((B, H, N), device=q.device, dtype=torch.float32)
    st = lib().gt_attn_fwd_batch(_ptr(q), _ptr(k), _ptr(v), _ptr(spd), stride, _ptr(table),
                                 table.shape[1], _ptr(out), _ptr(lse), B, H, N, d, _dt(q), scale,
                                 _stream(stream))
    _check(st, "gt_attn_fwd_batch")
    return out, lse


def gt_attn_bwd_batch(q, k, v, spd, table, o, lse, d_o, scale: float | None = None,
                      workspace=None, grads=None, stream=None, spd_t=None):
    """dQ, dK, dV [B, H, N, d] and dTable [H, nb] summed over the batch (C ABI
    gt_attn_bwd_batch); spd_t, if given, has spd's shape."""
    _qdims(q, "q", 4)
    B, H, N, d = q.shape
    stride = _batch_spd(spd, B, N)
    _check_bwd(q, k, v, spd, table, o, lse, d_o, grads, spd_t, (B, H))
    need = gt_attn_bwd_workspace_size(B * H, N, d, q.dtype)
    _devices(q, k, v, spd, table, o, lse, d_o, spd_t, *(grads or ()))
    if workspace is not None:
        _workspace(workspace, need, q)
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    if grads is None:
        grads = (torch.empty_like(q), torch.empty_like(k), torch.empty_like(v),
                 torch.empty_like(table))
    dq, dk, dv, dtable = grads
    if workspace is None:
        workspace = torch.empty(need, device=q.device, dtype=torch.uint8)
    st = lib().gt_attn_bwd_batch(_ptr(q), _ptr(k), _ptr(v), _ptr(spd),
                                 None if spd_t is None else _ptr(spd_t), stride, _ptr(table),
                                 table.shape[1], _ptr(o), _ptr(lse), _ptr(d_o), _ptr(dq), _ptr(dk),
                                 _ptr(dv), _ptr(dtable), _ptr(workspace),
                                 workspace.numel() * workspace.element_size(), B, H, N, d, _dt(q),
                                 scale, _stream(stream))
    _check(st, "gt_attn_bwd_batch")
    return dq, dk, dv, dtable


def _check_kv_block(q_shard, k_shard, v_shard):
    """KV block [H, Sk, d] of q_shard's dtype, or None for an empty block;
    returns Sk."""
    if k_shard is None and v_shard is None:
        return 0
    H, _, d = q_shard.shape
    _need(isinstance(k_shard, torch.Tensor) and k_shard.dim() == 3, "k_shard must be [H, Sk, d]")
    Sk = k_shard.shape[1]
    _shape(k_shard, "k_shard", (H, Sk, d), q_shard.dtype)
    _shape(v_shard, "v_shard", (H, Sk, d), q_shard.dtype)
    return Sk


def gt_attn_ring_step(q_shard, k_shard, v_shard, spd, row_off: int, col_off: int, table,
                      scale: float | None = None, out=None, lse=None, stream=None):
    """Partial (O_p fp32, LSE_p) of one context-parallel step (C ABI
    gt_attn_ring_step). spd: uint8 2-D tensor, element (r, c) = spd[r, c];
    its row stride is ld_spd, and it must hold rows row_off .. row_off + Sq - 1
    and columns col_off .. col_off + Sk - 1."""
    _qdims(q_shard, "q_shard", 3)
    H, Sq, d = q_shard.shape
    Sk = _check_kv_block(q_shard, k_shard, v_shard)
    _need(int(row_off) >= 0 and int(col_off) >= 0, "row_off and col_off must be >= 0")
    if Sk > 0:
        _spd_view(spd, int(row_off) + Sq, int(col_off) + Sk)
    _table(table, H)
    if out is not None:
        _shape(out, "out", (H, Sq, d), torch.float32)
    if lse is not None:
        _shape(lse, "lse", (H, Sq), torch.float32)
    _devices(q_shard, k_shard, v_shard, table, out, lse)
    if Sk > 0:
        _devices(q_shard, spd, contiguous=False)
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    if out is None:
        out = torch.empty((H, Sq, d), device=q_shard.device, dtype=torch.float32)
    if lse is None:
        lse = torch.empty((H, Sq), device=q_shard.device, dtype=torch.float32)
    ld = spd.stride(0) if (spd is not None and Sk > 0) else 0
    st = lib().gt_attn_ring_step(_ptr(q_shard), Sq, _ptr(k_shard), _ptr(v_shard), Sk,
                                 _ptr(spd) if Sk > 0 else None, ld, int(row_off), int(col_off),
                                 _ptr(table), table.shape[1], _ptr(out), _ptr(lse), H, d,
                                 _dt(q_shard), scale, _stream(stream))
    _check(st, "gt_attn_ring_step")
    return out, lse


def gt_attn_ring_step_acc(q_shard, k_shard, v_shard, spd, row_off: int, col_off: int, table,
                          state, scale: float | None = None, stream=None):
    """One context-parallel step merged in place into the running state
    (o_acc fp32 [H, Sq, d], lse_acc fp32 [H, Sq]) (C ABI
    gt_attn_ring_step_acc); returns the state. The first step's
    gt_attn_ring_step output is a valid starting state."""
    _qdims(q_shard, "q_shard", 3)
    H, Sq, d = q_shard.shape
    Sk = _check_kv_block(q_shard, k_shard, v_shard)
    _need(int(row_off) >= 0 and int(col_off) >= 0, "row_off and col_off must be >= 0")
    if Sk > 0:
        _spd_view(spd, int(row_off) + Sq, int(col_off) + Sk)
    _table(table, H)
    _need(len(state) == 2, "state must be (o_acc, lse_acc)")
    o_acc, lse_acc = state
    _shape(o_acc, "o_acc", (H, Sq, d), torch.float32)
    _shape(lse_acc, "lse_acc", (H, Sq), torch.float32)
    _devices(q_shard, k_shard, v_shard, table, o_acc, lse_acc)
    if Sk > 0:
        _devices(q_shard, spd, contiguous=False)
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    ld = spd.stride(0) if (spd is not None and Sk > 0) else 0
    st = lib().gt_attn_ring_step_acc(_ptr(q_shard), Sq, _ptr(k_shard), _ptr(v_shard), Sk,
                                     _ptr(spd) if Sk > 0 else None, ld, int(row_off), int(col_off),
                                     _ptr(table), table.shape[1], _ptr(o_acc), _ptr(lse_acc), H, d,
                                     _dt(q_shard), scale, _stream(stream))
    _check(st, "gt_attn_ring_step_acc")
    return o_acc, lse_acc


def gt_attn_bwd_ring_workspace_size(H: int, Sq: int, Sk: int, d: int, dtype=torch.bfloat16) -> int:
    return int(lib().gt_attn_bwd_ring_workspace_size(
        H, Sq, Sk, d, GT_BF16 if dtype == torch.bfloat16 else GT_F32))


def gt_attn_bwd_ring_step(q_shard, o_shard, lse_shard, d_o_shard, k_blk, v_blk, spd,
                          row_off: int, col_off: int, table, scale: float | None = None,
                          acc=None, workspace=None, stream=None):
    """Add one ring step's gradients (C ABI gt_attn_bwd_ring_step) into the
    fp32 accumulators acc = (dq [H,Sq,d], dk [H,Sk,d], dv [H,Sk,d],
    dtable [H,n_buckets]); acc=None starts them at zero. o_shard / lse_shard
    are the merged forward results of the shard's rows."""
    dt = _qdims(q_shard, "q_shard", 3)
    H, Sq, d = q_shard.shape
    _shape(o_shard, "o_shard", q_shard.shape, dt)
    _shape(d_o_shard, "d_o_shard", q_shard.shape, dt)
    _shape(lse_shard, "lse_shard", (H, Sq), torch.float32)
    Sk = _check_kv_block(q_shard, k_blk, v_blk)
    _need(int(row_off) >= 0 and int(col_off) >= 0, "row_off and col_off must be >= 0")
    if Sk > 0:
        _spd_view(spd, int(row_off) + Sq, int(col_off) + Sk)
    _table(table, H)
    if acc is not None:
        _need(len(acc) == 4, "acc must be (dq, dk, dv, dtable)")
        _shape(acc[0], "dq accumulator", (H, Sq, d), torch.float32)
        _shape(acc[1], "dk accumulator", (H, Sk, d), torch.float32)
        _shape(acc[2], "dv accumulator", (H, Sk, d), torch.float32)
        _shape(acc[3], "dtable accumulator", table.shape, torch.float32)
    need = gt_attn_bwd_ring_workspace_size(H, Sq, Sk, d, q_shard.dtype)
    _devices(q_shard, o_shard, lse_shard, d_o_shard, k_blk, v_blk, table, *(acc or ()))
    if Sk > 0:
        _devices(q_shard, spd, contiguous=False)
    if workspace is not None:
        _workspace(workspace, need, q_shard)
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    dev = q_shard.device
    if acc is None:
        acc = (torch.zeros((H, Sq, d), device=dev, dtype=torch.float32),
               torch.zeros((H, Sk, d), device=dev, dtype=torch.float32),
               torch.zeros((H, Sk, d), device=dev, dtype=torch.float32),
               torch.zeros_like(table))
    dq, dk, dv, dtable = acc
    if workspace is None:
        workspace = torch.empty(max(need, 1), device=dev, dtype=torch.uint8)
    ld = spd.stride(0) if (spd is not None and Sk > 0) else 0
    st = lib().gt_attn_bwd_ring_step(
        _ptr(q_shard), _ptr(o_shard), _ptr(lse_shard), _ptr(d_o_shard), Sq,
        _ptr(k_blk), _ptr(v_blk), Sk, _ptr(spd) if Sk > 0 else None, ld, int(row_off), int(col_off),
        _ptr(table), table.shape[1], _ptr(dq), _ptr(dk), _ptr(dv), _ptr(dtable),
        _ptr(workspace), workspace.numel() * workspace.element_size(), H, d, _dt(q_shard),
        scale, _stream(stream))
    _check(st, "gt_attn_bwd_ring_step")
    return dq, dk, dv, dtable


def gt_attn_merge(o_parts, lse_parts, dtype=torch.bfloat16, out=None, lse=None, stream=None):
    """Combine partials [P, H, S, d] / [P, H, S] (C ABI gt_attn_merge)."""
    _need(isinstance(o_parts, torch.Tensor) and o_parts.dim() == 4 and o_parts.dtype == torch.float32,
          "o_parts must be fp32 [P, H, S, d]")
    P, H, S, d = o_parts.shape
    _need(d in _HEAD_DIMS, f"head dim must be one of {_HEAD_DIMS}, got {d}")
    _need(P >= 1 and H >= 1 and S >= 1, "o_parts must not be empty")
    _shape(lse_parts, "lse_parts", (P, H, S), torch.float32)
    if out is not None:
        _need(out.dtype in (torch.bfloat16, torch.float32), "out must be bfloat16 or float32")
        _shape(out, "out", (H, S, d))
    else:
        _need(dtype in (torch.bfloat16, torch.float32), "dtype must be bfloat16 or float32")
    if lse is not None:
        _shape(lse, "lse", (H, S), torch.float32)
    _devices(o_parts, lse_parts, out, lse)
    if out is None:
        out = torch.empty((H, S, d), device=o_parts.device, dtype=dtype)
    if lse is None:
        lse = torch.empty((H, S), device=o_parts.device, dtype=torch.float32)
    st = lib().gt_attn_merge(_ptr(o_parts), _ptr(lse_parts), P, _ptr(out), _ptr(lse), H, S, d,
                             GT_BF16 if out.dtype == torch.bfloat16 else GT_F32, _stream(stream))
    _check(st, "gt_attn_merge")
    return out, lse
