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

__all__ = ["gt_attn_fwd", "gt_attn_bwd", "gt_attn_bwd_phase", "gt_attn_ring_step",
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


def _dev_contig(*ts):
    for t in ts:
        if t is not None:
            _need(t.is_cuda and t.is_contiguous(), "tensors must be contiguous device tensors")


def gt_attn_fwd(q, k, v, spd, table, scale: float | None = None, out=None, lse=None,
                stream=None):
    """O, LSE of biased attention over all N nodes (C ABI gt_attn_fwd).
    q, k, v [H, N, d] bf16|fp32; spd [N, N] uint8; table [H, n_buckets] fp32."""
    H, N, d = q.shape
    _dev_contig(q, k, v, spd, table, out, lse)
    _need(spd.dtype == torch.uint8 and tuple(spd.shape) == (N, N), "spd must be uint8 [N, N]")
    _need(table.dtype == torch.float32 and table.dim() == 2 and table.shape[0] == H,
          "table must be fp32 [H, n_buckets]")
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


def gt_attn_bwd_phase(phase: int, q, k, v, spd, table, o, lse, d_o, scale: float | None = None,
                      workspace=None, grads=None, stream=None, spd_t=None):
    """One stage of the backward (C ABI gt_attn_bwd_phase): 0 prepare,
    1 dK/dV/dtable, 2 dQ; phase -1 runs gt_attn_bwd (all three)."""
    H, N, d = q.shape
    _dev_contig(q, k, v, spd, table, o, lse, d_o)
    if spd_t is not None:
        _dev_contig(spd_t)
        if tuple(spd_t.shape) != tuple(spd.shape) or spd_t.dtype != spd.dtype:
            raise ValueError("spd_t must have the shape and dtype of spd")
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    if grads is None:
        grads = (torch.empty_like(q), torch.empty_like(k), torch.empty_like(v),
                 torch.empty_like(table))
    dq, dk, dv, dtable = grads
    _dev_contig(dq, dk, dv, dtable)
    need = gt_attn_bwd_workspace_size(H, N, d, q.dtype)
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


def _batch_spd(spd, B, N):
    _need(spd.dtype == torch.uint8 and spd.dim() in (2, 3) and tuple(spd.shape[-2:]) == (N, N),
          "spd must be uint8 [B, N, N] or [N, N] (shared by the batch)")
    if spd.dim() == 2:
        return 0
    _need(spd.shape[0] == B, "spd must hold one [N, N] matrix per graph")
    return spd.stride(0) if B > 1 else 0


def gt_attn_fwd_batch(q, k, v, spd, table, scale: float | None = None, out=None, lse=None,
                      stream=None):
    """O, LSE of a batch of graphs (C ABI gt_attn_fwd_batch). q, k, v
    [B, H, N, d]; spd [B, N, N] uint8 (or [N, N] shared); table [H, nb]."""
    B, H, N, d = q.shape
    _dev_contig(q, k, v, spd, table, out, lse)
    stride = _batch_spd(spd, B, N)
    _need(table.dtype == torch.float32 and table.dim() == 2 and table.shape[0] == H,
          "table must be fp32 [H, n_buckets]")
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
    B, H, N, d = q.shape
    _dev_contig(q, k, v, spd, table, o, lse, d_o)
    stride = _batch_spd(spd, B, N)
    if spd_t is not None:
        _dev_contig(spd_t)
        _need(tuple(spd_t.shape) == tuple(spd.shape) and spd_t.dtype == spd.dtype and
              spd_t.stride() == spd.stride(), "spd_t must have the shape and layout of spd")
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    if grads is None:
        grads = (torch.empty_like(q), torch.empty_like(k), torch.empty_like(v),
                 torch.empty_like(table))
    dq, dk, dv, dtable = grads
    _dev_contig(dq, dk, dv, dtable)
    need = gt_attn_bwd_workspace_size(B * H, N, d, q.dtype)
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


def gt_attn_ring_step(q_shard, k_shard, v_shard, spd, row_off: int, col_off: int, table,
                      scale: float | None = None, out=None, lse=None, stream=None):
    """Partial (O_p fp32, LSE_p) of one context-parallel step (C ABI
    gt_attn_ring_step). spd: uint8 2-D tensor, element (r, c) = spd[r, c];
    its row stride is ld_spd."""
    H, Sq, d = q_shard.shape
    Sk = k_shard.shape[1] if k_shard is not None else 0
    _dev_contig(q_shard, k_shard, v_shard, table, out, lse)
    _need(spd is None or (spd.dtype == torch.uint8 and spd.dim() == 2 and spd.stride(1) == 1),
          "spd must be a uint8 2-D tensor with unit column stride")
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    if out is None:
        out = torch.empty((H, Sq, d), device=q_shard.device, dtype=torch.float32)
    if lse is None:
        lse = torch.empty((H, Sq), device=q_shard.device, dtype=torch.float32)
    ld = spd.stride(0) if spd is not None else 0
    st = lib().gt_attn_ring_step(_ptr(q_shard), Sq, _ptr(k_shard), _ptr(v_shard), Sk,
                                 _ptr(spd), ld, int(row_off), int(col_off), _ptr(table),
                                 table.shape[1], _ptr(out), _ptr(lse), H, d, _dt(q_shard),
                                 scale, _stream(stream))
    _check(st, "gt_attn_ring_step")
    return out, lse


def gt_attn_ring_step_acc(q_shard, k_shard, v_shard, spd, row_off: int, col_off: int, table,
                          state, scale: float | None = None, stream=None):
    """One context-parallel step merged in place into the running state
    (o_acc fp32 [H, Sq, d], lse_acc fp32 [H, Sq]) (C ABI
    gt_attn_ring_step_acc); returns the state. The first step's
    gt_attn_ring_step output is a valid starting state."""
    H, Sq, d = q_shard.shape
    Sk = k_shard.shape[1] if k_shard is not None else 0
    o_acc, lse_acc = state
    _dev_contig(q_shard, k_shard, v_shard, table, o_acc, lse_acc)
    _need(spd is None or (spd.dtype == torch.uint8 and spd.dim() == 2 and spd.stride(1) == 1),
          "spd must be a uint8 2-D tensor with unit column stride")
    _need(o_acc.dtype == torch.float32 and tuple(o_acc.shape) == (H, Sq, d),
          "o_acc must be fp32 [H, Sq, d]")
    _need(lse_acc.dtype == torch.float32 and tuple(lse_acc.shape) == (H, Sq),
          "lse_acc must be fp32 [H, Sq]")
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    ld = spd.stride(0) if spd is not None else 0
    st = lib().gt_attn_ring_step_acc(_ptr(q_shard), Sq, _ptr(k_shard), _ptr(v_shard), Sk,
                                     _ptr(spd), ld, int(row_off), int(col_off), _ptr(table),
                                     table.shape[1], _ptr(o_acc), _ptr(lse_acc), H, d,
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
    H, Sq, d = q_shard.shape
    Sk = k_blk.shape[1] if k_blk is not None else 0
    _dev_contig(q_shard, o_shard, lse_shard, d_o_shard, k_blk, v_blk, table)
    _need(spd is None or (spd.dtype == torch.uint8 and spd.dim() == 2 and spd.stride(1) == 1),
          "spd must be a uint8 2-D tensor with unit column stride")
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    dev = q_shard.device
    if acc is None:
        acc = (torch.zeros((H, Sq, d), device=dev, dtype=torch.float32),
               torch.zeros((H, Sk, d), device=dev, dtype=torch.float32),
               torch.zeros((H, Sk, d), device=dev, dtype=torch.float32),
               torch.zeros_like(table))
    dq, dk, dv, dtable = acc
    _dev_contig(dq, dk, dv, dtable)
    for t in acc:
        _need(t.dtype == torch.float32, "accumulators must be fp32")
    need = gt_attn_bwd_ring_workspace_size(H, Sq, Sk, d, q_shard.dtype)
    if workspace is None:
        workspace = torch.empty(max(need, 1), device=dev, dtype=torch.uint8)
    ld = spd.stride(0) if spd is not None else 0
    st = lib().gt_attn_bwd_ring_step(
        _ptr(q_shard), _ptr(o_shard), _ptr(lse_shard), _ptr(d_o_shard), Sq,
        _ptr(k_blk), _ptr(v_blk), Sk, _ptr(spd), ld, int(row_off), int(col_off),
        _ptr(table), table.shape[1], _ptr(dq), _ptr(dk), _ptr(dv), _ptr(dtable),
        _ptr(workspace), workspace.numel() * workspace.element_size(), H, d, _dt(q_shard),
        scale, _stream(stream))
    _check(st, "gt_attn_bwd_ring_step")
    return dq, dk, dv, dtable


def gt_attn_merge(o_parts, lse_parts, dtype=torch.bfloat16, out=None, lse=None, stream=None):
    """Combine partials [P, H, S, d] / [P, H, S] (C ABI gt_attn_merge)."""
    P, H, S, d = o_parts.shape
    _dev_contig(o_parts, lse_parts, out, lse)
    if out is None:
        out = torch.empty((H, S, d), device=o_parts.device, dtype=dtype)
    if lse is None:
        lse = torch.empty((H, S), device=o_parts.device, dtype=torch.float32)
    st = lib().gt_attn_merge(_ptr(o_parts), _ptr(lse_parts), P, _ptr(out), _ptr(lse), H, S, d,
                             GT_BF16 if out.dtype == torch.bfloat16 else GT_F32, _stream(stream))
    _check(st, "gt_attn_merge")
    return out, lse
