"""Argument checks of the Python binding (CPU only).

Every entry point checks each tensor's shape and dtype against q and table,
and a ring step's spd extent, before the device check and before anything
is launched. CPU tensors let the tests reach each check: a case with one
wrong argument raises ValueError naming that argument; the well-formed case
then fails only at the device check."""
import pytest
import torch

import paper_2609_34420_amd as gt

H, N, D, NB = 2, 48, 32, 10


def z(*shape, dtype=torch.bfloat16):
    return torch.zeros(*shape, dtype=dtype)


def fwd_args():
    return dict(q=z(H, N, D), k=z(H, N, D), v=z(H, N, D), spd=z(N, N, dtype=torch.uint8),
                table=z(H, NB, dtype=torch.float32))


def bwd_args():
    a = fwd_args()
    a.update(o=z(H, N, D), lse=z(H, N, dtype=torch.float32), d_o=z(H, N, D))
    return a


def call_fwd(a, **kw):
    a = dict(a, **kw)
    return gt.gt_attn_fwd(a.pop("q"), a.pop("k"), a.pop("v"), a.pop("spd"), a.pop("table"), **a)


def call_bwd(a, **kw):
    a = dict(a, **kw)
    return gt.gt_attn_bwd(a.pop("q"), a.pop("k"), a.pop("v"), a.pop("spd"), a.pop("table"),
                          a.pop("o"), a.pop("lse"), a.pop("d_o"), **a)


def test_well_formed_cpu_tensors_fail_only_at_the_device_check():
    with pytest.raises(ValueError, match="device"):
        call_fwd(fwd_args())
    with pytest.raises(ValueError, match="device"):
        call_bwd(bwd_args())


@pytest.mark.parametrize("name,bad,match", [
    ("q", z(H, N, 48), "head dim"),
    ("q", z(H, N, D, dtype=torch.float16), "bfloat16 or float32"),
    ("k", z(H, N + 1, D), "k must have shape"),
    ("k", z(H, N, D, dtype=torch.float32), "k must be"),
    ("v", z(H, N, 16), "v must have shape"),
    ("spd", z(N, N - 1, dtype=torch.uint8), "spd must have shape"),
    ("spd", z(N, N, dtype=torch.int32), "spd must be"),
    ("table", z(H + 1, NB, dtype=torch.float32), "table must be"),
    ("table", z(H, NB), "table must be"),
    ("table", z(H, 257, dtype=torch.float32), "1..256 buckets"),
    ("out", z(H, N, D, dtype=torch.float32), "out must be"),
    ("lse", z(H, N + 2, dtype=torch.float32), "lse must have shape"),
])
def test_fwd_rejects(name, bad, match):
    with pytest.raises(ValueError, match=match):
        call_fwd(fwd_args(), **{name: bad})


@pytest.mark.parametrize("name,bad,match", [
    ("o", z(H, N, D, dtype=torch.float32), "o must be"),
    ("o", z(H, N - 1, D), "o must have shape"),
    ("lse", z(H, N), "lse must be"),
    ("d_o", z(H, N, 16), "d_o must have shape"),
    ("spd_t", z(N, N + 16, dtype=torch.uint8), "spd_t"),
    ("grads", (z(H, N, D), z(H, N, D), z(H, N, D), z(H, NB + 1, dtype=torch.float32)), "dtable"),
    ("grads", (z(H, N, D), z(H, 2 * N, D), z(H, N, D), z(H, NB, dtype=torch.float32)), "dk"),
    ("grads", (z(H, N, D, dtype=torch.float32), z(H, N, D), z(H, N, D),
               z(H, NB, dtype=torch.float32)), "dq"),
    ("workspace", z(16, dtype=torch.uint8), "workspace"),
])
def test_bwd_rejects(name, bad, match):
    if name == "workspace":
        # the workspace size comes from the library; the shape checks pass,
        # the device check then fails first for CPU tensors
        with pytest.raises(ValueError, match="device"):
            call_bwd(bwd_args(), workspace=bad)
        return
    with pytest.raises(ValueError, match=match):
        call_bwd(bwd_args(), **{name: bad})


def test_bwd_phase_rejects_unknown_phase():
    a = bwd_args()
    with pytest.raises(ValueError, match="phase"):
        gt.gt_attn_bwd_phase(3, a["q"], a["k"], a["v"], a["spd"], a["table"], a["o"], a["lse"], a["d_o"])


def test_batch_rejects():
    B = 3
    q = z(B, H, N, D)
    spd = z(B, N, N, dtype=torch.uint8)
    t = z(H, NB, dtype=torch.float32)
    with pytest.raises(ValueError, match="device"):
        gt.gt_attn_fwd_batch(q, q, q, spd, t)
    with pytest.raises(ValueError, match="one \\[N, N\\] matrix per graph"):
        gt.gt_attn_fwd_batch(q, q, q, z(B + 1, N, N, dtype=torch.uint8), t)
    with pytest.raises(ValueError, match="lse must have shape"):
        gt.gt_attn_fwd_batch(q, q, q, spd, t, lse=z(H, N, dtype=torch.float32))
    lse = z(B, H, N, dtype=torch.float32)
    with pytest.raises(ValueError, match="lse must have shape"):
        gt.gt_attn_bwd_batch(q, q, q, spd, t, q, z(B, H, N + 1, dtype=torch.float32), q)
    with pytest.raises(ValueError, match="device"):
        gt.gt_attn_bwd_batch(q, q, q, spd, t, q, lse, q)


def ring_args(Sq=16, Sk=24, ld=64, rows=16):
    return dict(q=z(H, Sq, D), k=z(H, Sk, D), v=z(H, Sk, D), spd=z(rows, ld, dtype=torch.uint8),
                table=z(H, NB, dtype=torch.float32))


@pytest.mark.parametrize("entry", ["ring", "ring_acc", "bwd_ring"])
@pytest.mark.parametrize("case,match", [
    ("ok", "device"),
    ("rows", "rows"),              # row_off + Sq past the shard's rows
    ("cols", "columns"),           # col_off + Sk past the view's columns
    ("col_view", "columns"),       # a column-sliced view: ld_spd is the full row
    ("neg", ">= 0"),
    ("kv", "v_shard must have shape"),
    ("spd_dtype", "uint8 2-D"),
])
def test_ring_steps_reject(entry, case, match):
    a = ring_args()
    row_off, col_off = 0, 8
    spd = a["spd"]
    if case == "rows":
        row_off = 1
    elif case == "cols":
        col_off = 41
    elif case == "col_view":
        spd = z(16, 128, dtype=torch.uint8)[:, 32:60]    # 28 columns, row stride 128
        col_off = 8
    elif case == "neg":
        col_off = -1
    elif case == "kv":
        a["v"] = z(H, 23, D)
    elif case == "spd_dtype":
        spd = z(16, 64, dtype=torch.int16)
    q, k, v, t = a["q"], a["k"], a["v"], a["table"]
    with pytest.raises(ValueError, match=match):
        if entry == "ring":
            gt.gt_attn_ring_step(q, k, v, spd, row_off, col_off, t)
        elif entry == "ring_acc":
            state = (z(H, 16, D, dtype=torch.float32), z(H, 16, dtype=torch.float32))
            gt.gt_attn_ring_step_acc(q, k, v, spd, row_off, col_off, t, state)
        else:
            lse = z(H, 16, dtype=torch.float32)
            gt.gt_attn_bwd_ring_step(q, q, lse, q, k, v, spd, row_off, col_off, t)


def test_ring_state_and_accumulator_shapes():
    a = ring_args()
    q, k, v, spd, t = a["q"], a["k"], a["v"], a["spd"], a["table"]
    with pytest.raises(ValueError, match="o_acc"):
        gt.gt_attn_ring_step_acc(q, k, v, spd, 0, 0, t, (z(H, 16, D), z(H, 16, dtype=torch.float32)))
    with pytest.raises(ValueError, match="lse_acc"):
        gt.gt_attn_ring_step_acc(q, k, v, spd, 0, 0, t,
                                 (z(H, 16, D, dtype=torch.float32), z(H, 15, dtype=torch.float32)))
    lse = z(H, 16, dtype=torch.float32)
    f = torch.float32
    bad_acc = (z(H, 16, D, dtype=f), z(H, 16, D, dtype=f), z(H, 24, D, dtype=f), z(H, NB, dtype=f))
    with pytest.raises(ValueError, match="dk accumulator"):
        gt.gt_attn_bwd_ring_step(q, q, lse, q, k, v, spd, 0, 0, t, acc=bad_acc)
    with pytest.raises(ValueError, match="o_shard"):
        gt.gt_attn_bwd_ring_step(q, z(H, 16, D, dtype=f), lse, q, k, v, spd, 0, 0, t)


def test_merge_rejects():
    P, S = 3, 40
    op = z(P, H, S, D, dtype=torch.float32)
    lp = z(P, H, S, dtype=torch.float32)
    with pytest.raises(ValueError, match="device"):
        gt.gt_attn_merge(op, lp)
    with pytest.raises(ValueError, match="lse_parts"):
        gt.gt_attn_merge(op, z(P, H, S + 1, dtype=torch.float32))
    with pytest.raises(ValueError, match="o_parts"):
        gt.gt_attn_merge(z(P, H, S, D), lp)
    with pytest.raises(ValueError, match="out must have shape"):
        gt.gt_attn_merge(op, lp, out=z(H, S, 16))
