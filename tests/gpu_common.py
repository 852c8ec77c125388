"""Shared helpers of the GPU parity tests: device upload, error metrics,
and the tolerances every comparison uses.

Tolerances (bf16 numbers as required for this path; fp32 numbers derived
from fp32 rounding of sums over at most a few thousand terms):
  O, LSE        max-abs  <= 2e-2 (bf16),  1e-5 (fp32)
  dQ, dK, dV, dtable  relative L2 over the whole tensor <= 1e-2 (bf16), 1e-5 (fp32)
"""
from __future__ import annotations

import numpy as np
import torch

DEV = "cuda:0"
TOL = {
    "bf16": dict(o=2e-2, lse=2e-2, grad=1e-2),
    "f32": dict(o=1e-5, lse=1e-5, grad=1e-5),
}


def say(msg: str) -> None:
    print(f"[gpu-case] {msg}", flush=True)


def tdtype(name: str):
    return torch.bfloat16 if name == "bf16" else torch.float32


def to_dev(x: np.ndarray, dtype=torch.float32) -> torch.Tensor:
    t = torch.from_numpy(np.ascontiguousarray(x))
    if t.dtype != dtype:
        t = t.to(dtype)
    return t.to(DEV)


def to_np(t: torch.Tensor) -> np.ndarray:
    return t.detach().to(torch.float64).cpu().numpy()


def max_abs(a, b) -> float:
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    both_inf = np.isneginf(a) & np.isneginf(b)
    with np.errstate(invalid="ignore"):
        d = np.abs(np.where(both_inf, 0.0, a - b))
    return float(np.nan_to_num(d, nan=np.inf).max()) if d.size else 0.0


def rel_l2(a, b) -> float:
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    nb = np.linalg.norm(b)
    na = np.linalg.norm(a - b)
    if nb == 0.0:
        return float(na)
    return float(na / nb)


def check_fwd(tag, o_gpu, lse_gpu, o_ref, lse_ref, dt):
    eo, el = max_abs(o_gpu, o_ref), max_abs(lse_gpu, lse_ref)
    say(f"{tag}: O max-abs {eo:.3e}  LSE max-abs {el:.3e}")
    assert eo <= TOL[dt]["o"], (tag, "O", eo)
    assert el <= TOL[dt]["lse"], (tag, "LSE", el)
    assert np.array_equal(np.isneginf(lse_gpu), np.isneginf(lse_ref)), (tag, "-inf rows differ")


def check_grads(tag, got: dict, ref: dict, dt):
    for name in ("dq", "dk", "dv", "dtable"):
        if name not in got:
            continue
        e = rel_l2(got[name], ref[name])
        say(f"{tag}: {name} rel-L2 {e:.3e}")
        assert np.isfinite(got[name]).all(), (tag, name, "non-finite")
        assert e <= TOL[dt]["grad"], (tag, name, e)


def _oracle_head_job(args):
    """One head of the oracle on query rows R against all keys: O, LSE and
    the backward of rows R (runs in a worker process; two BLAS threads)."""
    q, k, v, do, spd_R, table, scale, R = args
    from threadpoolctl import threadpool_limits

    import oracle
    with threadpool_limits(2):
        o, l = oracle.block_attention(q[:, R], k, v, spd_R, table, scale)
        dq, dk, dv, dt = oracle.block_backward(q[:, R], k, v, spd_R, table, scale, do[:, R])
    return o, l, dq, dk, dv, dt


def oracle_by_head(q, k, v, do, spd_R, table, scale, R, workers=8):
    """The oracle on rows R, each head in its own worker process (spawned,
    numpy only: the workers never touch the GPU). Returns, per head,
    (O, LSE, dQ of rows R, dK, dV, dtable of a dO zero outside R)."""
    import multiprocessing

    H = q.shape[0]
    jobs = [(q[h:h + 1], k[h:h + 1], v[h:h + 1], do[h:h + 1], spd_R, table[h:h + 1], scale, R)
            for h in range(H)]
    with multiprocessing.get_context("spawn").Pool(min(workers, H)) as pool:
        return pool.map(_oracle_head_job, jobs)
