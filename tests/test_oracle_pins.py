"""Pins of the CPU oracle to things other than itself.

Each test checks the oracle against a library routine (torch SDPA, torch
autograd, torch.logsumexp), a closed form, an invariant of the mathematics,
central finite differences, or values worked out by hand (tests/golden).
The cases are chosen so that a dropped term, a wrong sign, a transposed
index or a swapped operand in the oracle fails at least one of them.
"""
import math
import re

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle

RNG = np.random.default_rng(1234)


def _rand_case(H=2, N=24, d=8, nb=6, seed=0, asym=True, out_of_range=False):
    g = np.random.default_rng(seed)
    q = g.standard_normal((H, N, d))
    k = g.standard_normal((H, N, d))
    v = g.standard_normal((H, N, d))
    do = g.standard_normal((H, N, d))
    table = 0.7 * g.standard_normal((H, nb))
    hi = nb + 3 if out_of_range else nb
    spd = g.integers(0, hi, size=(N, N)).astype(np.uint8)
    if not asym:
        spd = np.minimum(spd, spd.T)
    np.fill_diagonal(spd, 0)
    return q, k, v, do, table, spd


def _torch_bias(table, spd):
    """Bias via torch indexing into a zero-padded 256-entry table."""
    t = torch.as_tensor(table, dtype=torch.float64)
    H, nb = t.shape
    pad = torch.cat([t, torch.zeros(H, 256 - nb, dtype=torch.float64)], dim=1)
    idx = torch.as_tensor(spd.astype(np.int64))
    return pad[:, idx]  # [H, N, N]


# ---------------------------------------------------------------------------
# Forward pins
# ---------------------------------------------------------------------------

def test_zero_bias_is_plain_softmax_attention():
    """table == 0: biased attention reduces to softmax attention (SDPA)."""
    q, k, v, _, table, spd = _rand_case(seed=1)
    table = np.zeros_like(table)
    scale = 1 / math.sqrt(q.shape[2])
    O, L = oracle.forward(q, k, v, spd, table, scale)
    qt, kt, vt = (torch.as_tensor(x) for x in (q, k, v))
    ref = F.scaled_dot_product_attention(qt, kt, vt, scale=scale).numpy()
    np.testing.assert_allclose(O, ref, rtol=1e-12, atol=1e-12)
    lse_ref = torch.logsumexp(scale * qt @ kt.transpose(-1, -2), dim=-1).numpy()
    np.testing.assert_allclose(L, lse_ref, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("seed", [2, 3])
def test_biased_matches_sdpa_with_additive_mask(seed):
    """Arbitrary table/spd: SDPA with the bias passed as a float attn_mask,
    and torch.logsumexp for LSE."""
    q, k, v, _, table, spd = _rand_case(seed=seed, out_of_range=True)
    scale = 0.37
    O, L = oracle.forward(q, k, v, spd, table, scale)
    qt, kt, vt = (torch.as_tensor(x) for x in (q, k, v))
    B = _torch_bias(table, spd)
    ref = F.scaled_dot_product_attention(qt, kt, vt, attn_mask=B, scale=scale).numpy()
    np.testing.assert_allclose(O, ref, rtol=1e-12, atol=1e-12)
    lse_ref = torch.logsumexp(scale * qt @ kt.transpose(-1, -2) + B, dim=-1).numpy()
    np.testing.assert_allclose(L, lse_ref, rtol=1e-12, atol=1e-12)


def test_orientation_successor_graph():
    """spd[i, i+1] = 1 (a directed cycle), every other pair 2, diagonal 0;
    with a huge bias on bucket 1, row i attends to node i+1 only: O_i = V_{i+1}.
    A transposed index would give V_{i-1}."""
    N, d = 11, 3
    g = np.random.default_rng(5)
    spd = np.full((N, N), 2, dtype=np.uint8)
    np.fill_diagonal(spd, 0)
    spd[np.arange(N), (np.arange(N) + 1) % N] = 1
    table = np.array([[0.0, 60.0, 0.0]])
    q = g.standard_normal((1, N, d))
    k = g.standard_normal((1, N, d))
    v = g.standard_normal((1, N, d))
    O, L = oracle.forward(q, k, v, spd, table, 0.1)
    np.testing.assert_allclose(O[0], v[0][(np.arange(N) + 1) % N], atol=1e-20, rtol=1e-18)
    # LSE_i = S_{i,i+1} + ln(1 + sum_{j != i+1} exp(S_ij - S_{i,i+1})) ~= S_{i,i+1}
    s_next = 0.1 * np.einsum("nd,nd->n", q[0], k[0][(np.arange(N) + 1) % N]) + 60.0
    np.testing.assert_allclose(L[0], s_next, atol=1e-20, rtol=1e-15)


def test_shift_invariance_per_head_constant():
    """table[h, :] == c_h leaves O unchanged and shifts LSE by exactly c_h."""
    q, k, v, _, table, spd = _rand_case(seed=6)
    scale = 0.3
    O0, L0 = oracle.forward(q, k, v, spd, np.zeros_like(table), scale)
    c = np.array([1.75, -3.5])
    O1, L1 = oracle.forward(q, k, v, spd, np.repeat(c[:, None], table.shape[1], 1), scale)
    np.testing.assert_allclose(O1, O0, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(L1 - L0, np.broadcast_to(c[:, None], L0.shape), atol=1e-12)


def test_uniform_closed_form():
    """Q = 0 and table = 0: every score is 0, so O_i = mean_j V_j, LSE_i = ln N."""
    H, N, d = 3, 37, 5
    g = np.random.default_rng(7)
    k = g.standard_normal((H, N, d))
    v = g.standard_normal((H, N, d))
    spd = g.integers(0, 4, (N, N)).astype(np.uint8)
    O, L = oracle.forward(np.zeros((H, N, d)), k, v, spd, np.zeros((H, 4)), 0.5)
    np.testing.assert_allclose(O, np.broadcast_to(v.mean(axis=1, keepdims=True), O.shape), atol=1e-14)
    np.testing.assert_allclose(L, np.full((H, N), math.log(N)), atol=1e-14)


def test_bias_only_closed_form():
    """Q = 0: LSE_i = ln sum_b cnt_i[b] e^{table[b]} (row counts, so an i/j swap
    of an asymmetric spd fails), and O_i = sum_j e^{table[spd_ij]} V_j / e^{LSE_i}."""
    H, N, d, nb = 2, 29, 4, 7
    g = np.random.default_rng(8)
    spd = g.integers(0, nb + 2, (N, N)).astype(np.uint8)  # some out of range
    table = g.standard_normal((H, nb))
    k = g.standard_normal((H, N, d))
    v = g.standard_normal((H, N, d))
    O, L = oracle.forward(np.zeros((H, N, d)), k, v, spd, table, 1.0)
    lse_cf = oracle.lse_bias_only(spd, table)
    np.testing.assert_allclose(L, lse_cf, atol=1e-13)
    # independent: by explicit python sums
    for h in range(H):
        for i in (0, 13, N - 1):
            w = [math.exp(table[h, s]) if s < nb else 1.0 for s in spd[i]]
            tot = sum(w)
            assert abs(L[h, i] - math.log(tot)) < 1e-12
            oi = sum(wj * v[h, j] for j, wj in enumerate(w)) / tot
            np.testing.assert_allclose(O[h, i], oi, atol=1e-13)
    assert not np.allclose(oracle.lse_bias_only(spd.T, table), L)


def test_single_node():
    """N = 1: O = V, LSE = scale q.k + table[spd00]; dV = dO, dQ = dK = 0, dTable = 0."""
    g = np.random.default_rng(9)
    q, k, v, do = (g.standard_normal((2, 1, 6)) for _ in range(4))
    table = g.standard_normal((2, 5))
    spd = np.array([[3]], dtype=np.uint8)
    O, L = oracle.forward(q, k, v, spd, table, 0.25)
    np.testing.assert_allclose(O, v, atol=1e-15)
    np.testing.assert_allclose(L[:, 0], 0.25 * (q * k).sum(-1)[:, 0] + table[:, 3], atol=1e-15)
    dq, dk, dv, dt = oracle.backward(q, k, v, spd, table, 0.25, do)
    np.testing.assert_allclose(dv, do, atol=1e-15)
    assert np.abs(dq).max() < 1e-15 and np.abs(dk).max() < 1e-15 and np.abs(dt).max() < 1e-15


def test_permutation_equivariance():
    """Relabelling nodes by pi (rows of Q,K,V,dO and both axes of spd) permutes
    O, LSE, dQ, dK, dV the same way and leaves dTable unchanged."""
    q, k, v, do, table, spd = _rand_case(seed=10, N=20)
    pi = np.random.default_rng(11).permutation(20)
    s = 0.4
    O, L = oracle.forward(q, k, v, spd, table, s)
    g = oracle.backward(q, k, v, spd, table, s, do)
    sp = spd[pi][:, pi]
    Op, Lp = oracle.forward(q[:, pi], k[:, pi], v[:, pi], sp, table, s)
    gp = oracle.backward(q[:, pi], k[:, pi], v[:, pi], sp, table, s, do[:, pi])
    np.testing.assert_allclose(Op, O[:, pi], atol=1e-13)
    np.testing.assert_allclose(Lp, L[:, pi], atol=1e-13)
    for a, b in zip(gp[:3], g[:3]):
        np.testing.assert_allclose(a, b[:, pi], atol=1e-12)
    np.testing.assert_allclose(gp[3], g[3], atol=1e-12)


def test_out_of_range_bucket_is_zero_bias_no_grad():
    """spd >= n_buckets contributes bias 0 and no gradient: same result as a
    table explicitly extended with zeros whose gradient is discarded."""
    q, k, v, do, table, spd = _rand_case(seed=12, out_of_range=True, nb=5)
    assert (spd >= 5).any()
    ext = np.concatenate([table, np.zeros((table.shape[0], 251))], axis=1)
    s = 0.5
    O, L = oracle.forward(q, k, v, spd, table, s)
    Oe, Le = oracle.forward(q, k, v, spd, ext, s)
    np.testing.assert_allclose(O, Oe, atol=1e-14)
    np.testing.assert_allclose(L, Le, atol=1e-14)
    g = oracle.backward(q, k, v, spd, table, s, do)
    ge = oracle.backward(q, k, v, spd, ext, s, do)
    for a, b in zip(g[:3], ge[:3]):
        np.testing.assert_allclose(a, b, atol=1e-13)
    np.testing.assert_allclose(g[3], ge[3][:, :5], atol=1e-13)
    assert g[3].shape == (2, 5)


def test_fully_masked_row():
    """-inf table entries: a row whose every bucket is -inf gives O = 0,
    LSE = -inf, zero gradients and no NaN; other rows match SDPA on them."""
    H, N, d = 1, 9, 4
    g = np.random.default_rng(13)
    q, k, v, do = (g.standard_normal((H, N, d)) for _ in range(4))
    table = np.array([[-np.inf, -np.inf, 0.3, -0.2]])
    spd = g.integers(0, 4, (N, N)).astype(np.uint8)
    spd[0] = g.integers(0, 2, N)         # row 0 only hits -inf buckets
    spd[1, :] = 2                         # row 1 only bucket 2
    O, L = oracle.forward(q, k, v, spd, table, 0.5)
    assert np.isneginf(L[0, 0]) and np.all(O[0, 0] == 0)
    assert np.isfinite(L[0, 1:]).all() and np.isfinite(O).all()
    dq, dk, dv, dt = oracle.backward(q, k, v, spd, table, 0.5, do)
    for x in (dq, dk, dv, dt):
        assert np.isfinite(x).all()
    assert np.all(dq[0, 0] == 0)
    rows = np.arange(1, N)
    B = _torch_bias(table, spd)[:, 1:]
    ref = F.scaled_dot_product_attention(torch.as_tensor(q[:, rows]), torch.as_tensor(k),
                                         torch.as_tensor(v), attn_mask=B, scale=0.5).numpy()
    np.testing.assert_allclose(O[:, rows], ref, atol=1e-12)
    # the masked row contributes nothing: same grads as zeroing its dO
    do2 = do.copy()
    do2[:, 0] = 0
    g2 = oracle.backward(q, k, v, spd, table, 0.5, do2)
    for a, b in zip((dq, dk, dv, dt), g2):
        np.testing.assert_allclose(a, b, atol=1e-14)


# ---------------------------------------------------------------------------
# Backward pins
# ---------------------------------------------------------------------------

def _loss(q, k, v, spd, table, s, do):
    O, _ = oracle.forward(q, k, v, spd, table, s)
    return float((O * do).sum())


def test_gradients_match_central_differences():
    """Every gradient entry against (L(x+h) - L(x-h)) / 2h on N <= 32."""
    q, k, v, do, table, spd = _rand_case(H=2, N=12, d=4, nb=5, seed=14, out_of_range=True)
    s = 0.6
    grads = oracle.backward(q, k, v, spd, table, s, do)
    h = 1e-6
    for which, arr in enumerate((q, k, v, table)):
        fd = np.zeros_like(arr)
        for idx in np.ndindex(arr.shape):
            args = [q.copy(), k.copy(), v.copy(), table.copy()]
            args[which][idx] += h
            lp = _loss(args[0], args[1], args[2], spd, args[3], s, do)
            args[which][idx] -= 2 * h
            lm = _loss(args[0], args[1], args[2], spd, args[3], s, do)
            fd[idx] = (lp - lm) / (2 * h)
        err = np.linalg.norm(grads[which] - fd) / np.linalg.norm(fd)
        assert err < 1e-6, (which, err)


def test_gradients_match_torch_autograd():
    """torch fp64 autograd of softmax(s QK^T + table[spd]) V (the gather's
    backward is a scatter-add, which pins dTable), N = 200, ragged sizes."""
    q, k, v, do, table, spd = _rand_case(H=3, N=200, d=16, nb=9, seed=15, out_of_range=True)
    s = 0.25
    dq, dk, dv, dt = oracle.backward(q, k, v, spd, table, s, do)
    qt, kt, vt, tt = (torch.tensor(x, requires_grad=True) for x in (q, k, v, table))
    H, nb = table.shape
    pad = torch.cat([tt, torch.zeros(H, 256 - nb, dtype=torch.float64)], dim=1)
    B = pad[:, torch.as_tensor(spd.astype(np.int64))]
    O = torch.softmax(s * qt @ kt.transpose(-1, -2) + B, dim=-1) @ vt
    (O * torch.as_tensor(do)).sum().backward()
    for mine, ref in ((dq, qt.grad), (dk, kt.grad), (dv, vt.grad), (dt, tt.grad)):
        np.testing.assert_allclose(mine, ref.numpy(), rtol=1e-10, atol=1e-12)


def test_gradient_invariants():
    """sum_b dTable[h,b] = 0 (shift invariance), sum_j dK[h,j] = 0 (rows of dS
    sum to 0), sum_j dV[h,j] = sum_i dO[h,i] (rows of P sum to 1)."""
    q, k, v, do, table, spd = _rand_case(H=2, N=40, d=6, nb=8, seed=16)
    dq, dk, dv, dt = oracle.backward(q, k, v, spd, table, 0.3, do)
    np.testing.assert_allclose(dt.sum(axis=1), 0, atol=1e-12)
    np.testing.assert_allclose(dk.sum(axis=1), 0, atol=1e-12)
    np.testing.assert_allclose(dv.sum(axis=1), do.sum(axis=1), atol=1e-12)
    assert np.abs(dt).max() > 1e-3


def test_golden_hand_example(golden_dir):
    """Values worked out by hand for a 2-node graph (tests/golden/hand_n2.txt)."""
    vals = {}
    for line in (golden_dir / "hand_n2.txt").read_text().splitlines():
        if not line.strip() or line.startswith("#"):
            continue
        key, *toks = line.split()

        def ev(t):
            return eval(re.sub(r"ln(\d+(?:\.\d+)?)", r"math.log(\1)", t), {"math": math})
        vals[key] = np.array([ev(t) for t in toks], dtype=np.float64)
    q = vals["q"].reshape(1, 2, 1)
    k = vals["k"].reshape(1, 2, 1)
    v = vals["v"].reshape(1, 2, 1)
    do = vals["do"].reshape(1, 2, 1)
    table = vals["table"].reshape(1, 3)
    spd = vals["spd"].astype(np.uint8).reshape(2, 2)
    O, L = oracle.forward(q, k, v, spd, table, 1.0)
    np.testing.assert_allclose(O.ravel(), vals["o"], atol=1e-14)
    np.testing.assert_allclose(L.ravel(), vals["lse"], atol=1e-14)
    dq, dk, dv, dt = oracle.backward(q, k, v, spd, table, 1.0, do)
    np.testing.assert_allclose(dq.ravel(), vals["dq"], atol=1e-14)
    np.testing.assert_allclose(dk.ravel(), vals["dk"], atol=1e-14)
    np.testing.assert_allclose(dv.ravel(), vals["dv"], atol=1e-14)
    np.testing.assert_allclose(dt.ravel(), vals["dtable"], atol=1e-14)


# ---------------------------------------------------------------------------
# Ring step + merge pins
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("bounds", [[0, 50], [0, 13, 50], [0, 7, 31, 50],
                                    [0, 3, 9, 10, 22, 30, 33, 41, 50]])
def test_ring_merge_equals_unsharded(bounds):
    """Merged ring partials (each rank using only its spd row shard, KV blocks
    visited in ring order) equal the unsharded forward, for P = 1, 2, 3, 8
    with uneven shards."""
    q, k, v, _, table, spd = _rand_case(H=2, N=50, d=8, nb=6, seed=17, out_of_range=True)
    s = 0.35
    O, L = oracle.forward(q, k, v, spd, table, s)
    Or, Lr = oracle.ring_forward(q, k, v, spd, table, s, bounds)
    np.testing.assert_allclose(Or, O, atol=1e-12)
    np.testing.assert_allclose(Lr, L, atol=1e-12)


def test_merge_ignores_neg_inf_parts():
    """A part with LSE = -inf contributes nothing; all -inf gives O = 0, LSE = -inf;
    a single part is returned unchanged."""
    g = np.random.default_rng(18)
    o = g.standard_normal((3, 1, 4, 2))
    lse = g.standard_normal((3, 1, 4))
    lse[1, 0, :2] = -np.inf
    lse[:, 0, 3] = -np.inf
    O, L = oracle.merge(o, lse)
    O2, L2 = oracle.merge(o[[0, 2]], lse[[0, 2]])
    np.testing.assert_allclose(O[0, :2], O2[0, :2], atol=1e-15)
    np.testing.assert_allclose(L[0, :2], L2[0, :2], atol=1e-15)
    assert np.isneginf(L[0, 3]) and np.all(O[0, 3] == 0)
    O1, L1 = oracle.merge(o[:1], lse[:1])
    np.testing.assert_allclose(O1[:, :3], o[0][:, :3], atol=1e-15)
    np.testing.assert_allclose(L1, lse[0], atol=1e-15)
    assert np.all(O1[0, 3] == 0)
    # closed form for two parts with equal LSE: plain average, LSE + ln 2
    Oe, Le = oracle.merge(o[:2, :, 2:3], np.zeros((2, 1, 1)))
    np.testing.assert_allclose(Oe, o[:2, :, 2:3].mean(0), atol=1e-15)
    np.testing.assert_allclose(Le, math.log(2), atol=1e-15)


def test_ring_step_offsets_select_the_right_slice():
    """ring_step reads spd[row_off + i, col_off + j]: with a bias that is large
    only at one global column per row, the partial picks that key."""
    N = 16
    g = np.random.default_rng(19)
    q, k, v = (g.standard_normal((1, N, 3)) for _ in range(3))
    spd = np.zeros((N, N), dtype=np.uint8)
    target = (np.arange(N) * 5 + 3) % N
    spd[np.arange(N), target] = 1
    table = np.array([[0.0, 80.0]])
    for row_off, col_off, Sq, Sk in [(4, 8, 4, 8), (0, 0, 16, 16), (9, 2, 5, 14)]:
        o, l = oracle.ring_step(q[:, row_off:row_off + Sq], k[:, col_off:col_off + Sk],
                                v[:, col_off:col_off + Sk], spd, row_off, col_off, table, 0.1)
        for i in range(Sq):
            t = target[row_off + i]
            if col_off <= t < col_off + Sk:
                np.testing.assert_allclose(o[0, i], v[0, t], atol=1e-25, rtol=1e-20)


def test_row_sampled_backward_equals_masked_full_backward():
    """The full-size GPU checks rely on two facts, checked here on the full
    oracle: dQ of a query row depends only on that row, and with dO zero
    outside rows R the full dK, dV, dtable equal the backward of rows R."""
    q, k, v, do, table, spd = _rand_case(H=2, N=60, d=8, nb=7, seed=21, out_of_range=True)
    R = np.array([0, 5, 17, 33, 59])
    s = 0.4
    dq, _, _, _ = oracle.backward(q, k, v, spd, table, s, do)
    dq_r, dk_r, dv_r, dt_r = oracle.block_backward(q[:, R], k, v, spd[R], table, s, do[:, R])
    np.testing.assert_allclose(dq_r, dq[:, R], atol=1e-12)
    dom = np.zeros_like(do)
    dom[:, R] = do[:, R]
    _, dk_m, dv_m, dt_m = oracle.backward(q, k, v, spd, table, s, dom)
    np.testing.assert_allclose(dk_r, dk_m, atol=1e-12)
    np.testing.assert_allclose(dv_r, dv_m, atol=1e-12)
    np.testing.assert_allclose(dt_r, dt_m, atol=1e-12)
    O, L = oracle.forward(q, k, v, spd, table, s)
    O_r, L_r = oracle.block_attention(q[:, R], k, v, spd[R], table, s)
    np.testing.assert_allclose(O_r, O[:, R], atol=1e-12)
    np.testing.assert_allclose(L_r, L[:, R], atol=1e-12)


# ---------------------------------------------------------------------------
# Backward ring step pins
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("bounds", [[0, 50], [0, 13, 50], [0, 7, 31, 50],
                                    [0, 3, 9, 10, 22, 30, 33, 41, 50]])
def test_ring_backward_equals_unsharded(bounds):
    """Every rank visiting every KV block with the merged LSE and Dlt, dQ
    accumulated locally and dK/dV/dTable accumulated per block, reproduces
    the unsharded backward (itself pinned by autograd and finite
    differences), for P = 1, 2, 3, 8 with uneven shards and out-of-range
    buckets."""
    q, k, v, do, table, spd = _rand_case(H=2, N=50, d=8, nb=6, seed=21, out_of_range=True)
    s = 0.35
    ref = oracle.backward(q, k, v, spd, table, s, do)
    got = oracle.ring_backward(q, k, v, spd, table, s, do, bounds)
    for a, b in zip(got, ref):
        np.testing.assert_allclose(a, b, atol=1e-11)


def test_ring_backward_step_single_block_is_block_backward():
    """One step covering every key (row_off = col_off = 0) with the block's
    own LSE is exactly block_backward for those query rows."""
    q, k, v, do, table, spd = _rand_case(H=2, N=30, d=6, nb=5, seed=22)
    s = 0.5
    R = np.arange(4, 19)
    O, L = oracle.forward(q, k, v, spd, table, s)
    got = oracle.ring_backward_step(q[:, R], O[:, R], L[:, R], do[:, R], k, v, spd[R], 0, 0,
                                    table, s)
    ref = oracle.block_backward(q[:, R], k, v, spd[R], table, s, do[:, R])
    for a, b in zip(got, ref):
        np.testing.assert_allclose(a, b, atol=1e-12)


def test_ring_backward_step_masked_rows_and_offsets():
    """A query row whose merged LSE is -inf gets no gradient; the spd slice
    is taken at (row_off, col_off) of a larger matrix (an i/j or offset
    mistake changes the bucket sums)."""
    q, k, v, do, table, spd = _rand_case(H=1, N=24, d=4, nb=7, seed=23)
    s = 0.7
    O, L = oracle.forward(q, k, v, spd, table, s)
    rows, cols = np.arange(5, 14), np.arange(10, 22)
    Lm = L[:, rows].copy()
    Lm[0, 2] = -np.inf
    dq, dk, dv, dt = oracle.ring_backward_step(q[:, rows], O[:, rows], Lm, do[:, rows], k[:, cols],
                                               v[:, cols], spd, 5, 10, table, s)
    assert np.all(dq[0, 2] == 0)
    # direct evaluation of the bucket sums of dS on the selected slice
    Sg = s * q[0, rows] @ k[0, cols].T + np.where(spd[np.ix_(rows, cols)] < 7,
                                                  table[0][np.minimum(spd[np.ix_(rows, cols)], 6)], 0.0)
    P = np.exp(Sg - np.where(np.isfinite(Lm[0]), Lm[0], 0.0)[:, None])
    P[2] = 0.0
    dS = P * (do[0, rows] @ v[0, cols].T - (do[0, rows] * O[0, rows]).sum(1)[:, None])
    b = spd[np.ix_(rows, cols)]
    ref = np.array([dS[b == j].sum() for j in range(7)])
    np.testing.assert_allclose(dt[0], ref, atol=1e-12)


# ---------------------------------------------------------------------------
# Super nodes (regular nodes partitioned, super nodes replicated)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("bounds,n_super", [([0, 40], 7), ([0, 11, 40], 7), ([0, 5, 19, 40], 1),
                                            ([0, 3, 9, 10, 22, 30, 33, 37, 40], 10),
                                            ([0, 13, 40], 0)])
def test_ring_super_equals_unsharded(bounds, n_super):
    """Each rank's shard = its regular rows plus every super-node row; the
    ring visits the P regular KV blocks and the super-node block once. The
    merged result equals the unsharded forward over all N = N' + N_s nodes,
    and every rank computes the same super-node rows."""
    N = 40 + n_super
    q, k, v, _, table, spd = _rand_case(H=2, N=N, d=8, nb=6, seed=31, out_of_range=True)
    s = 0.35
    O, L = oracle.forward(q, k, v, spd, table, s)
    Or, Lr, sup = oracle.ring_forward_super(q, k, v, spd, table, s, bounds, n_super)
    np.testing.assert_allclose(Or, O, atol=1e-12)
    np.testing.assert_allclose(Lr, L, atol=1e-12)
    for o_s, l_s in sup:
        np.testing.assert_allclose(o_s, O[:, 40:], atol=1e-12)
        np.testing.assert_allclose(l_s, L[:, 40:], atol=1e-12)
    if n_super == 0:
        O0, L0 = oracle.ring_forward(q, k, v, spd, table, s, bounds)
        np.testing.assert_allclose(Or, O0, atol=1e-14)


def test_super_nodes_in_every_block_are_counted_per_block():
    """Putting the super-node columns into every KV block (each block =
    regular columns plus the super columns) counts each super node P times:
    every row's total weight on the super nodes is multiplied by P, so for
    P = 3 the merged LSE of every row sits between the unsharded LSE and
    the unsharded LSE + ln 3, strictly above it, and differs from the
    count-once ring. With P = 1 the two coincide."""
    n_reg, n_super = 30, 5
    N = n_reg + n_super
    q, k, v, _, table, spd = _rand_case(H=2, N=N, d=8, nb=6, seed=32)
    s = 0.35
    O, L = oracle.forward(q, k, v, spd, table, s)
    for bounds in ([0, 30], [0, 9, 20, 30]):
        P = len(bounds) - 1
        for r in range(P):
            rows = oracle.super_shard_rows(bounds, N, n_super, r)
            parts_o, parts_l = [], []
            for t in range(P):
                c0, c1 = bounds[(r - t) % P], bounds[(r - t) % P + 1]
                cols = np.concatenate([np.arange(c0, c1), np.arange(n_reg, N)])
                o_p, l_p = oracle.block_attention(q[:, rows], k[:, cols], v[:, cols],
                                                  spd[np.ix_(rows, cols)], table, s)
                parts_o.append(o_p)
                parts_l.append(l_p)
            On, Ln = oracle.merge(np.stack(parts_o), np.stack(parts_l))
            if P == 1:
                np.testing.assert_allclose(Ln, L[:, rows], atol=1e-12)
                np.testing.assert_allclose(On, O[:, rows], atol=1e-12)
            else:
                assert np.all(Ln > L[:, rows] + 1e-9)
                assert np.all(Ln < L[:, rows] + math.log(P) + 1e-9)
                assert np.abs(On - O[:, rows]).max() > 1e-3


@pytest.mark.parametrize("bounds,n_super", [([0, 40], 6), ([0, 11, 40], 6),
                                            ([0, 3, 9, 22, 30, 40], 9)])
def test_ring_backward_super_equals_unsharded(bounds, n_super):
    """Backward with super nodes: rank 0 carries the super rows' dO, the other
    ranks pass zero for them; dQ per rank, dK/dV/dTable per block (super
    block included) add up to the unsharded backward."""
    N = 40 + n_super
    q, k, v, do, table, spd = _rand_case(H=2, N=N, d=8, nb=6, seed=33, out_of_range=True)
    s = 0.35
    ref = oracle.backward(q, k, v, spd, table, s, do)
    got = oracle.ring_backward_super(q, k, v, spd, table, s, do, bounds, n_super)
    for a, b in zip(got, ref):
        np.testing.assert_allclose(a, b, atol=1e-11)
