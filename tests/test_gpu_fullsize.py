"""GPU parity at the workloads' full sizes, through the same entry points and
launch configuration the benchmark times.

The oracle cannot materialise N x N at N = 131072, so the checks are:
  * sampled query rows R (seeded, both ends included): O, LSE and dQ of the
    dense run against the oracle on those rows (each row depends only on
    itself);
  * a second backward with dO zero outside R: then dK, dV and dtable depend
    only on rows R, and the oracle computes them exactly;
  * properties that hold at any size: sum_b dtable = 0, sum_j dK_j = 0,
    sum_j dV_j = sum_i dO_i, and the Q = 0 closed form of LSE from the row
    bucket counts of spd.
"""
import gc
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2609_34420_amd as gt
import synth
from gpu_common import DEV, TOL, check_fwd, check_grads, max_abs, rel_l2, say, to_np

pytestmark = pytest.mark.gpu


def _free():
    gc.collect()
    torch.cuda.empty_cache()


def _upload_spd(w, seed=0, rows=None):
    """Generate spd (all rows, or rows [r0, r1)) chunk by chunk straight into
    a device tensor."""
    r0, r1 = (0, w.N) if rows is None else rows
    n = r1 - r0
    spd = torch.empty((n, w.N), dtype=torch.uint8, device=DEV)
    chunk = min(n, 4096)
    host = torch.empty((chunk, w.N), dtype=torch.uint8, pin_memory=True)
    hv = host.numpy()
    for a in range(0, n, chunk):
        m = min(chunk, n - a)
        w.spd_block(r0 + a, m, seed=seed, out=hv[:m])
        spd[a:a + m].copy_(host[:m])
    torch.cuda.synchronize()
    return spd


def _bf16(x):
    return torch.from_numpy(x).to(torch.bfloat16).to(DEV)


def _sampled_parity(w, spd_dev, R, tag, layer=0, seed=0):
    """Dense fwd+bwd on the GPU, checked on rows R; then the row-masked bwd,
    checked in full. Returns the dense-run GPU results for further checks."""
    q, k, v = w.qkv(seed, layer=layer)
    do = w.d_out(seed, layer=layer)
    table = w.table(seed, layer=layer)
    scale = w.scale()
    Q, K, V, dO = _bf16(q), _bf16(k), _bf16(v), _bf16(do)
    T = torch.from_numpy(table).to(DEV)
    # as in the benchmark: a symmetric spd is its own transpose
    spd_t = spd_dev if (w.spd_symmetric and spd_dev.shape[0] == spd_dev.shape[1]) else None
    say(f"{tag}: dense fwd+bwd N={w.N} H={w.H} spd_t={'spd' if spd_t is not None else 'none'}")
    O, L = gt.gt_attn_fwd(Q, K, V, spd_dev, T, scale=scale)
    dq, dk, dv, dt = gt.gt_attn_bwd(Q, K, V, spd_dev, T, O, L, dO, scale=scale, spd_t=spd_t)
    torch.cuda.synchronize()
    spd_R = w.spd_rows(R, seed=seed)
    Rt = torch.from_numpy(R).to(DEV)
    o_ref, l_ref = oracle.block_attention(q[:, R], k, v, spd_R, table, scale)
    check_fwd(f"{tag} rows", to_np(O[:, Rt]), to_np(L[:, Rt]), o_ref, l_ref, "bf16")
    dq_ref, _, _, _ = oracle.block_backward(q[:, R], k, v, spd_R, table, scale, do[:, R])
    check_grads(f"{tag} rows", {"dq": to_np(dq[:, Rt])}, {"dq": dq_ref}, "bf16")

    say(f"{tag}: row-masked backward")
    mask = torch.zeros((1, w.N, 1), device=DEV, dtype=torch.bfloat16)
    mask[:, Rt] = 1
    dOm = (dO * mask).contiguous()
    _, dkm, dvm, dtm = gt.gt_attn_bwd(Q, K, V, spd_dev, T, O, L, dOm, scale=scale, spd_t=spd_t)
    torch.cuda.synchronize()
    _, dk_ref, dv_ref, dt_ref = oracle.block_backward(q[:, R], k, v, spd_R, table, scale, do[:, R])
    check_grads(f"{tag} masked", {"dk": to_np(dkm), "dv": to_np(dvm), "dtable": to_np(dtm)},
                {"dk": dk_ref, "dv": dv_ref, "dtable": dt_ref}, "bf16")
    return dict(Q=Q, K=K, V=V, dO=dO, T=T, O=O, L=L, dq=dq, dk=dk, dv=dv, dt=dt, do=do)


def _invariants(tag, r):
    """sum_b dtable = sum_ij dS_ij = sum_i (sum_j P_ij dP_ij - Dlt_i) is zero in
    exact arithmetic; in bf16 the residual per row is dO_i . (sum_j P_ij V_j -
    O_i) with O_i built from bf16-rounded P and stored in bf16, so it is
    bounded by 2^-7 sum_c |dO_ic| max_j |V_jc|. sum_j dK_j = scale sum_i
    (sum_j dS_ij) Q_i inherits the same relative residual; sum_j dV_j =
    sum_i dO_i holds to fp32 accumulation of bf16 products."""
    dt, dk, dv = to_np(r["dt"]), to_np(r["dk"]), to_np(r["dv"])
    V = r["V"].float() if "V" in r else None
    s_dk = np.linalg.norm(dk.sum(1)) / np.linalg.norm(dk)
    s_dv = rel_l2(dv.sum(1), r["do"].astype(np.float64).sum(1))
    msg = f"{tag}: invariants sum dK {s_dk:.2e}, sum dV vs sum dO {s_dv:.2e}"
    if V is not None:
        do_abs = np.abs(r["do"].astype(np.float64)).sum(1)             # [H, d]
        vmax = V.abs().amax(dim=1).double().cpu().numpy()            # [H, d]
        bound = 2.0 ** -7 * (do_abs * vmax).sum(1)                   # [H]
        resid = np.abs(dt.sum(1))
        msg += f", |sum dtable| / bound {np.max(resid / bound):.2e}"
        assert np.all(resid <= bound), (resid, bound)
    say(msg)
    assert s_dk <= 1e-2 and s_dv <= 1e-2


def test_ba16k_full_size():
    """N=16384, H=8, d=64 bf16, Barabasi-Albert m=4 spd (clip 30)."""
    w = synth.workload("ba16k")
    spd = _upload_spd(w)
    R = w.sample_rows(254)
    r = _sampled_parity(w, spd, R, "ba16k")
    _invariants("ba16k", r)
    del r, spd
    _free()


def test_sbm128k_full_size():
    """N=131072, H=8, d=64 bf16, clustered planted-partition spd (clip 62,
    unreachable 63; 17.2 GB in HBM)."""
    w = synth.workload("sbm128k")
    say("sbm128k: generating spd")
    spd = _upload_spd(w)
    R = w.sample_rows(62)
    r = _sampled_parity(w, spd, R, "sbm128k")
    _invariants("sbm128k", r)
    # Q = 0: LSE_i = ln sum_b cnt_i[b] exp(table[h, b]) (row bucket counts)
    say("sbm128k: Q = 0 closed form")
    Z = torch.zeros_like(r["Q"])
    _, L0 = gt.gt_attn_fwd(Z, r["K"], r["V"], spd, r["T"], scale=w.scale())
    torch.cuda.synchronize()
    Rt = torch.from_numpy(R).to(DEV)
    lse_cf = oracle.lse_bias_only(w.spd_rows(R), w.table(0))
    e = max_abs(to_np(L0[:, Rt]), lse_cf)
    say(f"sbm128k: Q=0 LSE max-abs {e:.2e}")
    assert e <= TOL["bf16"]["lse"]
    del r, spd, Z, L0
    _free()


def test_context_parallel_share_cp256k():
    """N=262144 in 8 shards of 32768; this device holds query shard 3 and only
    its spd rows [32768, 262144]. Ring steps visit KV blocks 3,2,1,0,7,6,5,4
    (block (rank - t) mod P), the partials are merged and compared with one
    unsharded step over all keys and with the oracle on sampled rows."""
    w = synth.workload("cp256k")
    P, S, rank = w.shards, w.S, w.shard
    r0 = rank * S
    say("cp256k: generating spd shard rows")
    spd_sh = _upload_spd(w, rows=(r0, r0 + S))
    q, k, v = w.qkv(0)
    table = w.table(0)
    scale = w.scale()
    Qs = _bf16(np.ascontiguousarray(q[:, r0:r0 + S]))
    K, V = _bf16(k), _bf16(v)
    T = torch.from_numpy(table).to(DEV)
    parts_o, parts_l = [], []
    for t in range(P):
        blk = (rank - t) % P
        c0 = blk * S
        say(f"cp256k: ring step {t} (KV block {blk})")
        o_p, l_p = gt.gt_attn_ring_step(Qs, K[:, c0:c0 + S].contiguous(), V[:, c0:c0 + S].contiguous(),
                                        spd_sh, 0, c0, T, scale=scale)
        parts_o.append(o_p)
        parts_l.append(l_p)
    O, L = gt.gt_attn_merge(torch.stack(parts_o), torch.stack(parts_l), dtype=torch.bfloat16)
    O_full, L_full = gt.gt_attn_ring_step(Qs, K, V, spd_sh, 0, 0, T, scale=scale)
    torch.cuda.synchronize()
    e_o = max_abs(to_np(O), to_np(O_full))
    e_l = max_abs(to_np(L), to_np(L_full))
    say(f"cp256k: merged vs unsharded step O {e_o:.2e} LSE {e_l:.2e}")
    assert e_o <= TOL["bf16"]["o"] and e_l <= 1e-4
    # the same ring with the in-place running merge (state started by step 0)
    state = (parts_o[0].clone(), parts_l[0].clone())
    for t in range(1, P):
        c0 = ((rank - t) % P) * S
        gt.gt_attn_ring_step_acc(Qs, K[:, c0:c0 + S].contiguous(), V[:, c0:c0 + S].contiguous(),
                                 spd_sh, 0, c0, T, state, scale=scale)
    torch.cuda.synchronize()
    e_o2 = max_abs(to_np(state[0]), to_np(O_full))
    e_l2 = max_abs(to_np(state[1]), to_np(L_full))
    say(f"cp256k: accumulated ring vs unsharded step O {e_o2:.2e} LSE {e_l2:.2e}")
    assert e_o2 <= TOL["bf16"]["o"] and e_l2 <= 1e-4
    R = w.sample_rows(62, lo=r0, hi=r0 + S)
    spd_R = w.spd_rows(R)
    o_ref, l_ref = oracle.block_attention(q[:, R], k, v, spd_R, table, scale)
    Rl = torch.from_numpy(R - r0).to(DEV)
    check_fwd("cp256k rows", to_np(O[:, Rl]), to_np(L[:, Rl]), o_ref, l_ref, "bf16")
    del parts_o, parts_l, spd_sh, K, V, Qs
    _free()


def test_deep_stack_deep32k():
    """12 layers of biased attention fwd+bwd, N=32768, H=16, d=64 bf16, 256
    Zipf(1.2) spd buckets shared by every layer, one table per layer. Layers 1
    and 12 are checked against the oracle on sampled rows (and row-masked);
    every layer is checked through the gradient invariants."""
    w = synth.workload("deep32k")
    say("deep32k: generating Zipf spd")
    spd = _upload_spd(w)
    R = w.sample_rows(30)
    gen = torch.Generator(device=DEV)
    for layer in range(w.layers):
        if layer in (0, w.layers - 1):
            r = _sampled_parity(w, spd, R, f"deep32k layer {layer + 1}", layer=layer)
            _invariants(f"deep32k layer {layer + 1}", r)
            del r
        else:
            gen.manual_seed(1000 + layer)
            shp = (w.H, w.N, w.d)
            Q = (torch.randn(shp, generator=gen, device=DEV) / 8).to(torch.bfloat16)
            K = (torch.randn(shp, generator=gen, device=DEV) / 8).to(torch.bfloat16)
            V = (torch.randn(shp, generator=gen, device=DEV) / 8).to(torch.bfloat16)
            dO = torch.randn(shp, generator=gen, device=DEV).to(torch.bfloat16)
            T = torch.randn((w.H, w.n_buckets), generator=gen, device=DEV) * 0.02
            say(f"deep32k layer {layer + 1}: fwd+bwd")
            O, L = gt.gt_attn_fwd(Q, K, V, spd, T)
            dq, dk, dv, dt = gt.gt_attn_bwd(Q, K, V, spd, T, O, L, dO)
            torch.cuda.synchronize()
            assert torch.isfinite(dq).all() and torch.isfinite(dt).all()
            _invariants(f"deep32k layer {layer + 1}", dict(dt=dt, dk=dk, dv=dv, do=to_np(dO), V=V))
    del spd
    _free()


def test_ring_step_spd_offset_beyond_4gib():
    """A ring step whose bias slice starts more than 2^32 bytes into spd
    (64-bit row offsets): spd [34000, 131072] uint8 (4.46 GB), rows
    33500.., columns 65536.."""
    rows, ld, nb = 34000, 131072, 40
    row_off, col_off, Sq, Sk, H, d = 33500, 65536, 300, 4096, 2, 64
    assert row_off * ld > 2 ** 32
    say("offset>4GiB: filling spd on the device")
    spd = torch.empty((rows, ld), dtype=torch.uint8, device=DEV)
    cols = torch.arange(ld, device=DEV, dtype=torch.int64)
    for r0 in range(0, rows, 2000):
        rr = torch.arange(r0, min(rows, r0 + 2000), device=DEV, dtype=torch.int64)[:, None]
        spd[r0:r0 + rr.shape[0]] = ((rr * 2654435761 + cols * 40503) >> 7) % (nb + 3)
    g = np.random.default_rng(77)
    q = synth.round_bf16(g.standard_normal((H, Sq, d)).astype(np.float32) / 8)
    k = synth.round_bf16(g.standard_normal((H, Sk, d)).astype(np.float32) / 8)
    v = synth.round_bf16(g.standard_normal((H, Sk, d)).astype(np.float32))
    table = (g.standard_normal((H, nb)) * 0.5).astype(np.float32)
    o, l = gt.gt_attn_ring_step(_bf16(q), _bf16(k), _bf16(v), spd, row_off, col_off,
                                torch.from_numpy(table).to(DEV), scale=0.125)
    torch.cuda.synchronize()
    r = np.arange(row_off, row_off + Sq, dtype=np.int64)[:, None]
    c = np.arange(ld, dtype=np.int64)[None, :]
    spd_host = (((r * 2654435761 + c * 40503) >> 7) % (nb + 3)).astype(np.uint8)
    o_ref, l_ref = oracle.ring_step(q, k, v, spd_host, 0, col_off, table, 0.125)
    check_fwd("offset>4GiB", to_np(o), to_np(l), o_ref, l_ref, "bf16")
    del spd
    _free()
