"""GPU parity at the workloads' full sizes, through the same entry points and
launch configuration the benchmark times.

The oracle cannot materialise N x N at N = 131072, so the checks are:
  * sampled query rows R, stratified so that every 256-row block (hence
    every forward and dQ workgroup's rows) holds sampled rows, plus both
    ends: O, LSE and dQ of the dense run against the oracle on those rows
    (each row depends only on itself);
  * a second backward with dO zero outside R: then dK, dV and dtable depend
    only on rows R, and the oracle computes them exactly;
  * properties that hold at any size: sum_b dtable = 0, sum_j dK_j = 0,
    sum_j dV_j = sum_i dO_i, and the Q = 0 closed form of LSE from the row
    bucket counts of spd.
At N = 16384 the oracle runs over every row. Each workload's GPU work runs
once (a module fixture that keeps host copies of what the checks need), and
so does the oracle, every head in its own worker process; one test per head
then compares. Every per-head comparison applies the whole-tensor parity
bars to that head's slice, which is stricter than to the tensor.
"""
import gc
import math
import time

import numpy as np
import pytest
import torch

import oracle
import paper_2609_34420_amd as gt
import synth
from gpu_common import DEV, TOL, check_fwd, check_grads, max_abs, oracle_by_head, say, to_np
from paper_2609_34420_amd import ring

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
    return torch.from_numpy(np.ascontiguousarray(x)).to(torch.bfloat16).to(DEV)


def _host(t):
    return t.detach().to(torch.float64).cpu().numpy()


def _invariants(tag, dt, dk, dv, do, V):
    """sum_b dtable = sum_ij dS_ij = sum_i (sum_j P_ij dP_ij - Dlt_i) is zero in
    exact arithmetic; in bf16 the residual per row is dO_i . (sum_j P_ij V_j -
    O_i) with O_i built from bf16-rounded P and stored in bf16, so it is
    bounded by 2^-7 sum_c |dO_ic| max_j |V_jc|. sum_j dK_j = scale sum_i
    (sum_j dS_ij) Q_i inherits the same relative residual; sum_j dV_j =
    sum_i dO_i holds to fp32 accumulation of bf16 products. Reductions run on
    the device, in fp64."""
    dk64, dv64, do64 = dk.double(), dv.double(), do.double()
    s_dk = (torch.linalg.vector_norm(dk64.sum(1)) / torch.linalg.vector_norm(dk64)).item()
    s_dv = (torch.linalg.vector_norm(dv64.sum(1) - do64.sum(1)) /
            torch.linalg.vector_norm(do64.sum(1))).item()
    bound = 2.0 ** -7 * (do64.abs().sum(1) * V.double().abs().amax(dim=1)).sum(1)      # [H]
    resid = dt.double().sum(1).abs()
    ratio = (resid / bound).max().item()
    say(f"{tag}: invariants sum dK {s_dk:.2e}, sum dV vs sum dO {s_dv:.2e}, "
        f"|sum dtable| / bound {ratio:.2e}")
    assert ratio <= 1.0
    assert s_dk <= 1e-2 and s_dv <= 1e-2


def _dense_and_masked(w, spd_dev, R, tag, layer=0, seed=0):
    """Dense fwd+bwd on the GPU and the backward with dO zero outside rows R.
    Returns host copies: O, LSE, dQ on rows R (dense run) and dK, dV, dtable
    of the masked run (of the dense run when R holds every row)."""
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
    Rt = torch.from_numpy(R).to(DEV)
    out = dict(R=R, q=q, k=k, v=v, do=do, table=table, scale=scale,
               O_R=_host(O[:, Rt]), L_R=_host(L[:, Rt]), dq_R=_host(dq[:, Rt]))
    _invariants(tag, dt, dk, dv, dO, V)
    if len(R) == w.N:
        out.update(dk_m=_host(dk), dv_m=_host(dv), dt_m=_host(dt), Q=Q, K=K, V=V, T=T)
        return out
    say(f"{tag}: row-masked backward ({len(R)} rows)")
    mask = torch.zeros((1, w.N, 1), device=DEV, dtype=torch.bfloat16)
    mask[:, Rt] = 1
    dOm = (dO * mask).contiguous()
    _, dkm, dvm, dtm = gt.gt_attn_bwd(Q, K, V, spd_dev, T, O, L, dOm, scale=scale, spd_t=spd_t)
    torch.cuda.synchronize()
    out.update(dk_m=_host(dkm), dv_m=_host(dvm), dt_m=_host(dtm))
    out.update(Q=Q, K=K, V=V, T=T)     # device tensors for further checks; dropped by the caller
    return out


def _oracle(r, spd_R):
    """The oracle over rows R for every head (worker processes)."""
    t0 = time.time()
    r["ref"] = oracle_by_head(r["q"], r["k"], r["v"], r["do"], spd_R, r["table"], r["scale"], r["R"])
    say(f"oracle on {len(r['R'])} rows x {r['q'].shape[0]} heads in {time.time() - t0:.1f}s")


def _check_head(tag, r, h):
    """Head h: O, LSE, dQ of the dense run on rows R and dK, dV, dtable of the
    row-masked run against the oracle."""
    hs = slice(h, h + 1)
    o_ref, l_ref, dq_ref, dk_ref, dv_ref, dt_ref = r["ref"][h]
    check_fwd(f"{tag} head {h} rows", r["O_R"][hs], r["L_R"][hs], o_ref, l_ref, "bf16")
    check_grads(f"{tag} head {h} rows", {"dq": r["dq_R"][hs]}, {"dq": dq_ref}, "bf16")
    check_grads(f"{tag} head {h} masked",
                {"dk": r["dk_m"][hs], "dv": r["dv_m"][hs], "dtable": r["dt_m"][hs]},
                {"dk": dk_ref, "dv": dv_ref, "dtable": dt_ref}, "bf16")


# ---------------------------------------------------------------------------
# N = 16384: the full oracle, every row
# ---------------------------------------------------------------------------
@pytest.fixture(scope="module")
def ba16k():
    """N=16384, H=8, d=64 bf16, Barabasi-Albert m=4 spd (clip 30)."""
    w = synth.workload("ba16k")
    spd = _upload_spd(w)
    R = np.arange(w.N, dtype=np.int64)
    r = _dense_and_masked(w, spd, R, "ba16k")
    for key in ("Q", "K", "V", "T"):
        r.pop(key)
    del spd
    _free()
    _oracle(r, w.spd_block(0, w.N))
    return r


@pytest.mark.parametrize("h", range(8))
def test_ba16k_full_oracle(ba16k, h):
    """Every row of head h against the oracle (with R = all rows the masked
    run is the dense backward)."""
    _check_head("ba16k", ba16k, h)


# ---------------------------------------------------------------------------
# Headline N = 131072: stratified rows
# ---------------------------------------------------------------------------
@pytest.fixture(scope="module")
def sbm128k():
    """N=131072, H=8, d=64 bf16, clustered planted-partition spd (clip 62,
    unreachable 63; 17.2 GB in HBM). R: 1024 rows, 2 in every 256-row block,
    plus rows 0 and N-1."""
    w = synth.workload("sbm128k")
    say("sbm128k: generating spd")
    spd = _upload_spd(w)
    R = w.stratified_rows(1024, block=256)
    assert len(R) >= 1024 and R[0] == 0 and R[-1] == w.N - 1
    assert np.unique(R // 256).size == w.N // 256
    r = _dense_and_masked(w, spd, R, "sbm128k")
    # Q = 0: LSE_i = ln sum_b cnt_i[b] exp(table[h, b]) (row bucket counts)
    Z = torch.zeros_like(r["Q"])
    _, L0 = gt.gt_attn_fwd(Z, r["K"], r["V"], spd, r["T"], scale=w.scale())
    torch.cuda.synchronize()
    r["L0_R"] = _host(L0[:, torch.from_numpy(R).to(DEV)])
    for key in ("Q", "K", "V", "T"):
        r.pop(key)
    del spd, Z, L0
    _free()
    r["spd_R"] = w.spd_rows(R)
    _oracle(r, r["spd_R"])
    return r


@pytest.mark.parametrize("h", range(8))
def test_sbm128k_rows(sbm128k, h):
    _check_head("sbm128k", sbm128k, h)


def test_sbm128k_bias_only_closed_form(sbm128k):
    lse_cf = oracle.lse_bias_only(sbm128k["spd_R"], sbm128k["table"])
    e = max_abs(sbm128k["L0_R"], lse_cf)
    say(f"sbm128k: Q=0 LSE max-abs {e:.2e} over {len(sbm128k['R'])} rows")
    assert e <= TOL["bf16"]["lse"]


# ---------------------------------------------------------------------------
# Context-parallel share: N = 262144 in 8 shards, this device holds shard 3
# ---------------------------------------------------------------------------
@pytest.fixture(scope="module")
def cp256k():
    """Query shard 3 of 8 (rows [98304, 131072)) and only its spd rows
    [32768, 262144] (8.6 GB). The forward ring visits KV blocks 3,2,1,0,7,6,5,4
    (block (rank - t) mod P); its partials are merged (and, separately, merged
    in place), and compared with one unsharded step over all keys. The
    backward ring then visits the same blocks with the merged (O, LSE), once
    with the dense dO and once with dO zero outside the sampled rows R (512
    rows, 4 in every 256-row block of the shard, plus its ends)."""
    w = synth.workload("cp256k")
    P, S, rank = w.shards, w.S, w.shard
    r0 = rank * S
    say("cp256k: generating spd shard rows")
    spd_sh = _upload_spd(w, rows=(r0, r0 + S))
    q, k, v = w.qkv(0)
    do = w.d_out(0)
    table = w.table(0)
    scale = w.scale()
    Qs = _bf16(q[:, r0:r0 + S])
    dOs = _bf16(do[:, r0:r0 + S])
    K, V = _bf16(k), _bf16(v)
    T = torch.from_numpy(table).to(DEV)
    bounds = [b * S for b in range(P + 1)]
    steps = ring.ring_steps(bounds, rank)
    assert [c0 // S for c0, _ in steps] == [3, 2, 1, 0, 7, 6, 5, 4]
    parts_o, parts_l = [], []
    for t, (c0, c1) in enumerate(steps):
        say(f"cp256k: forward ring step {t} (KV block {c0 // S})")
        o_p, l_p = gt.gt_attn_ring_step(Qs, K[:, c0:c1].contiguous(), V[:, c0:c1].contiguous(),
                                        spd_sh, 0, c0, T, scale=scale)
        parts_o.append(o_p)
        parts_l.append(l_p)
    O, L = gt.gt_attn_merge(torch.stack(parts_o), torch.stack(parts_l), dtype=torch.bfloat16)
    O_full, L_full = gt.gt_attn_ring_step(Qs, K, V, spd_sh, 0, 0, T, scale=scale)
    torch.cuda.synchronize()
    e_o = max_abs(_host(O), _host(O_full))
    e_l = max_abs(_host(L), _host(L_full))
    say(f"cp256k: merged vs unsharded step O {e_o:.2e} LSE {e_l:.2e}")
    assert e_o <= TOL["bf16"]["o"] and e_l <= 1e-4
    state = (parts_o[0].clone(), parts_l[0].clone())
    for c0, c1 in steps[1:]:
        gt.gt_attn_ring_step_acc(Qs, K[:, c0:c1].contiguous(), V[:, c0:c1].contiguous(),
                                 spd_sh, 0, c0, T, state, scale=scale)
    torch.cuda.synchronize()
    e_o2 = max_abs(_host(state[0]), _host(O_full))
    e_l2 = max_abs(_host(state[1]), _host(L_full))
    say(f"cp256k: accumulated ring vs unsharded step O {e_o2:.2e} LSE {e_l2:.2e}")
    assert e_o2 <= TOL["bf16"]["o"] and e_l2 <= 1e-4
    del parts_o, parts_l, O_full, L_full, state

    R = w.stratified_rows(512, block=256, lo=r0, hi=r0 + S)
    assert np.unique((R - r0) // 256).size == S // 256
    Rl = torch.from_numpy(R - r0).to(DEV)
    mask = torch.zeros((1, S, 1), device=DEV, dtype=torch.bfloat16)
    mask[:, Rl] = 1
    out = dict(R=R, q=q, k=k, v=v, do=do, table=table, scale=scale,
               O_R=_host(O[:, Rl]), L_R=_host(L[:, Rl]))
    for label, dO_use in (("dense", dOs), ("masked", (dOs * mask).contiguous())):
        dq = torch.zeros((w.H, S, w.d), device=DEV)
        dtab = torch.zeros_like(T)
        dks, dvs = [], []
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        ev[0].record()
        for c0, c1 in steps:
            dk_b = torch.zeros((w.H, c1 - c0, w.d), device=DEV)
            dv_b = torch.zeros_like(dk_b)
            gt.gt_attn_bwd_ring_step(Qs, O, L, dO_use, K[:, c0:c1].contiguous(),
                                     V[:, c0:c1].contiguous(), spd_sh, 0, c0, T, scale=scale,
                                     acc=(dq, dk_b, dv_b, dtab))
            dks.append(dk_b)
            dvs.append(dv_b)
        ev[1].record()
        torch.cuda.synchronize()
        say(f"cp256k: backward ring ({label} dO), 8 steps, {ev[0].elapsed_time(ev[1]):.1f} ms "
            f"(includes the per-block slicing)")
        order = np.argsort([c0 for c0, _ in steps])
        dk = torch.cat([dks[i] for i in order], dim=1)
        dv = torch.cat([dvs[i] for i in order], dim=1)
        if label == "dense":
            out["dq_R"] = _host(dq[:, Rl])
            assert torch.isfinite(dk).all() and torch.isfinite(dv).all()
        else:
            out.update(dk_m=_host(dk), dv_m=_host(dv), dt_m=_host(dtab))
        del dk, dv, dks, dvs, dq, dtab
    del spd_sh, K, V, Qs, dOs, O, L, T, mask
    _free()
    _oracle(out, w.spd_rows(R))
    return out


@pytest.mark.parametrize("h", range(8))
def test_context_parallel_share_cp256k(cp256k, h):
    """Forward (merged ring partials), dQ of the dense backward ring and dK,
    dV, dtable of the row-masked backward ring, head h, on the sampled rows
    of the shard against the unsharded oracle over all 262144 keys."""
    _check_head("cp256k", cp256k, h)


# ---------------------------------------------------------------------------
# Deep stack: 12 layers, N = 32768, H = 16, 256 Zipf buckets
# ---------------------------------------------------------------------------
@pytest.fixture(scope="module")
def deep32k():
    """12 layers of biased attention fwd+bwd, N=32768, H=16, d=64 bf16, 256
    Zipf(1.2) spd buckets shared by every layer, one table per layer. Layers
    1 and 12 keep host copies for the oracle (256 stratified rows plus the
    ends); every layer is checked through the gradient invariants."""
    w = synth.workload("deep32k")
    say("deep32k: generating Zipf spd")
    spd = _upload_spd(w)
    R = w.stratified_rows(256, block=256)
    gen = torch.Generator(device=DEV)
    kept = {}
    for layer in range(w.layers):
        if layer in (0, w.layers - 1):
            r = _dense_and_masked(w, spd, R, f"deep32k layer {layer + 1}", layer=layer)
            for key in ("Q", "K", "V", "T"):
                r.pop(key)
            kept[layer] = r
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
            _invariants(f"deep32k layer {layer + 1}", dt, dk, dv, dO, V)
            del Q, K, V, dO, T, O, L, dq, dk, dv, dt
    del spd
    _free()
    spd_R = w.spd_rows(R)
    for r in kept.values():
        _oracle(r, spd_R)
    return kept


@pytest.mark.parametrize("layer", [0, 11])
def test_deep_stack_deep32k(deep32k, layer):
    """Layers 1 and 12, every head, against the oracle on the sampled rows
    (dense and row-masked)."""
    r = deep32k[layer]
    for h in range(r["q"].shape[0]):
        _check_head(f"deep32k layer {layer + 1}", r, h)


# ---------------------------------------------------------------------------
# A bias slice past 4 GiB
# ---------------------------------------------------------------------------
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
