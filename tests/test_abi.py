"""C ABI of libgtattn.so on the host: exported symbols and the validation
paths, which return before anything is launched (no GPU needed)."""
import ctypes
import re
from pathlib import Path

import pytest

import paper_2609_34420_amd as gt

ROOT = Path(__file__).resolve().parents[1]
HEADER = ROOT / "include" / "gt_attn.h"

OK, INVALID, UNSUPPORTED, WORKSPACE, LAUNCH = 0, 1, 2, 3, 4
F32, BF16 = 0, 1
FAKE = 0x10000      # aligned non-null stand-in; validation fails before any use
MIS = 0x10008       # 8-byte aligned only


def declared_symbols():
    text = HEADER.read_text()
    return sorted(set(re.findall(r"\b(gt_[a-z_0-9]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    L = gt.lib()
    syms = declared_symbols()
    assert {"gt_attn_fwd", "gt_attn_bwd", "gt_attn_ring_step", "gt_attn_ring_step_acc", "gt_attn_merge",
            "gt_attn_bwd_ring_step", "gt_attn_bwd_ring_workspace_size",
            "gt_attn_bwd_workspace_size", "gt_status_string"} <= set(syms)
    for s in syms:
        assert hasattr(L, s), s
        assert ctypes.cast(getattr(L, s), ctypes.c_void_p).value


def test_status_strings_and_version():
    for code, name in [(OK, "GT_OK"), (INVALID, "GT_ERR_INVALID"), (UNSUPPORTED, "GT_ERR_UNSUPPORTED"),
                       (WORKSPACE, "GT_ERR_WORKSPACE"), (LAUNCH, "GT_ERR_LAUNCH")]:
        assert gt.gt_status_string(code).startswith(name)
    assert "unknown" in gt.gt_status_string(99)
    assert gt.gt_attn_version() >= 100


def _fwd(**kw):
    a = dict(q=FAKE, k=FAKE, v=FAKE, spd=FAKE, table=FAKE, nb=22, o=FAKE, lse=FAKE,
             H=4, N=512, d=32, dt=F32, scale=0.125)
    a.update(kw)
    return gt.lib().gt_attn_fwd(a["q"], a["k"], a["v"], a["spd"], a["table"], a["nb"], a["o"],
                                a["lse"], a["H"], a["N"], a["d"], a["dt"], a["scale"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(q=None), INVALID), (dict(k=None), INVALID), (dict(v=None), INVALID),
    (dict(spd=None), INVALID), (dict(table=None), INVALID), (dict(o=None), INVALID),
    (dict(lse=None), INVALID), (dict(H=0), INVALID), (dict(N=0), INVALID), (dict(N=-5), INVALID),
    (dict(nb=0), INVALID), (dict(nb=257), INVALID), (dict(scale=0.0), INVALID),
    (dict(scale=-1.0), INVALID), (dict(scale=float("inf")), INVALID),
    (dict(scale=float("nan")), INVALID), (dict(d=48), UNSUPPORTED), (dict(d=128), UNSUPPORTED),
    (dict(dt=7), UNSUPPORTED), (dict(q=MIS), INVALID), (dict(o=MIS), INVALID),
])
def test_fwd_validation(kw, code):
    assert _fwd(**kw) == code


def _fwd_batch(**kw):
    a = dict(q=FAKE, k=FAKE, v=FAKE, spd=FAKE, bs=512 * 512, table=FAKE, nb=22, o=FAKE, lse=FAKE,
             B=3, H=4, N=512, d=32, dt=F32, scale=0.125)
    a.update(kw)
    return gt.lib().gt_attn_fwd_batch(a["q"], a["k"], a["v"], a["spd"], a["bs"], a["table"],
                                      a["nb"], a["o"], a["lse"], a["B"], a["H"], a["N"], a["d"],
                                      a["dt"], a["scale"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(B=0), INVALID), (dict(B=-2), INVALID), (dict(bs=-1), INVALID), (dict(H=0), INVALID),
    (dict(N=0), INVALID), (dict(q=None), INVALID), (dict(spd=None), INVALID),
    (dict(lse=None), INVALID), (dict(nb=257), INVALID), (dict(scale=float("nan")), INVALID),
    (dict(d=48), UNSUPPORTED), (dict(dt=7), UNSUPPORTED), (dict(o=MIS), INVALID),
    (dict(B=70000, H=70000), INVALID),            # B * H past 2^31
])
def test_fwd_batch_validation(kw, code):
    assert _fwd_batch(**kw) == code


def _bwd_batch(**kw):
    B, H, N, d = 3, 2, 100, 64
    need = gt.lib().gt_attn_bwd_workspace_size(B * H, N, d, BF16)
    a = dict(q=FAKE, k=FAKE, v=FAKE, spd=FAKE, spd_t=None, bs=N * N, table=FAKE, nb=8, o=FAKE,
             lse=FAKE, do=FAKE, dq=FAKE, dk=FAKE, dv=FAKE, dt=FAKE, ws=FAKE, wsb=need, B=B, H=H,
             N=N, d=d, dtype=BF16, scale=0.125)
    a.update(kw)
    return gt.lib().gt_attn_bwd_batch(a["q"], a["k"], a["v"], a["spd"], a["spd_t"], a["bs"],
                                      a["table"], a["nb"], a["o"], a["lse"], a["do"], a["dq"],
                                      a["dk"], a["dv"], a["dt"], a["ws"], a["wsb"], a["B"], a["H"],
                                      a["N"], a["d"], a["dtype"], a["scale"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(B=0), INVALID), (dict(bs=-16), INVALID), (dict(dt=None), INVALID),
    (dict(do=None), INVALID), (dict(ws=None), WORKSPACE),
    (dict(wsb=gt.lib().gt_attn_bwd_workspace_size(2, 100, 64, BF16)), WORKSPACE),  # sized for one graph
    (dict(d=24), UNSUPPORTED), (dict(dq=MIS), INVALID),
])
def test_bwd_batch_validation(kw, code):
    assert _bwd_batch(**kw) == code


def _ring(entry="gt_attn_ring_step", **kw):
    a = dict(q=FAKE, Sq=100, k=FAKE, v=FAKE, Sk=64, spd=FAKE, ld=4096, ro=0, co=128, table=FAKE,
             nb=32, o=FAKE, lse=FAKE, H=8, d=64, dt=BF16, scale=0.125)
    a.update(kw)
    return getattr(gt.lib(), entry)(a["q"], a["Sq"], a["k"], a["v"], a["Sk"], a["spd"], a["ld"],
                                    a["ro"], a["co"], a["table"], a["nb"], a["o"], a["lse"],
                                    a["H"], a["d"], a["dt"], a["scale"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(Sq=0), INVALID), (dict(Sk=-1), INVALID), (dict(ro=-1), INVALID), (dict(co=-1), INVALID),
    (dict(ld=191), INVALID),                      # ld < col_off + Sk
    (dict(ld=1 << 25), UNSUPPORTED),
    (dict(k=None), INVALID), (dict(v=None), INVALID), (dict(spd=None), INVALID),
    (dict(q=None), INVALID), (dict(o=None), INVALID), (dict(lse=None), INVALID),
    (dict(table=None), INVALID), (dict(nb=300), INVALID), (dict(d=24), UNSUPPORTED),
    (dict(scale=0.0), INVALID), (dict(k=MIS), INVALID),
])
@pytest.mark.parametrize("entry", ["gt_attn_ring_step", "gt_attn_ring_step_acc"])
def test_ring_step_validation(entry, kw, code):
    assert _ring(entry, **kw) == code


def _bwd(**kw):
    H, N, d = 2, 100, 64
    need = gt.lib().gt_attn_bwd_workspace_size(H, N, d, BF16)
    a = dict(q=FAKE, k=FAKE, v=FAKE, spd=FAKE, spd_t=None, table=FAKE, nb=8, o=FAKE, lse=FAKE, do=FAKE,
             dq=FAKE, dk=FAKE, dv=FAKE, dt=FAKE, ws=FAKE, wsb=need, H=H, N=N, d=d, dtype=BF16,
             scale=0.125)
    a.update(kw)
    return gt.lib().gt_attn_bwd(a["q"], a["k"], a["v"], a["spd"], a["spd_t"], a["table"], a["nb"], a["o"],
                                a["lse"], a["do"], a["dq"], a["dk"], a["dv"], a["dt"], a["ws"],
                                a["wsb"], a["H"], a["N"], a["d"], a["dtype"], a["scale"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(ws=None), WORKSPACE), (dict(wsb=0), WORKSPACE), (dict(ws=FAKE + 16), WORKSPACE),
    (dict(do=None), INVALID), (dict(dq=None), INVALID), (dict(dk=None), INVALID),
    (dict(dv=None), INVALID), (dict(dt=None), INVALID), (dict(o=None), INVALID),
    (dict(lse=None), INVALID), (dict(d=96), UNSUPPORTED), (dict(N=0), INVALID),
    (dict(dq=MIS), INVALID), (dict(scale=float("nan")), INVALID),
])
def test_bwd_validation(kw, code):
    assert _bwd(**kw) == code


def test_bwd_workspace_size():
    L = gt.lib()
    # two fp32 [H, N] arrays and fp32 [H, ceil(N/256), 4], each padded to 256 bytes
    assert L.gt_attn_bwd_workspace_size(8, 131072, 64, BF16) == 2 * 8 * 131072 * 4 + 8 * 512 * 4 * 4
    assert L.gt_attn_bwd_workspace_size(1, 7, 32, F32) == 3 * 256
    assert L.gt_attn_bwd_workspace_size(0, 7, 32, F32) == 0


def _bwd_ring(**kw):
    H, Sq, Sk, d = 4, 100, 64, 64
    need = gt.lib().gt_attn_bwd_ring_workspace_size(H, Sq, Sk, d, BF16)
    a = dict(q=FAKE, o=FAKE, lse=FAKE, do=FAKE, Sq=Sq, k=FAKE, v=FAKE, Sk=Sk, spd=FAKE, ld=4096,
             ro=0, co=128, table=FAKE, nb=32, dq=FAKE, dk=FAKE, dv=FAKE, dt=FAKE, ws=FAKE, wsb=need,
             H=H, d=d, dtype=BF16, scale=0.125)
    a.update(kw)
    return gt.lib().gt_attn_bwd_ring_step(
        a["q"], a["o"], a["lse"], a["do"], a["Sq"], a["k"], a["v"], a["Sk"], a["spd"], a["ld"],
        a["ro"], a["co"], a["table"], a["nb"], a["dq"], a["dk"], a["dv"], a["dt"], a["ws"], a["wsb"],
        a["H"], a["d"], a["dtype"], a["scale"], None)


@pytest.mark.parametrize("kw,code", [
    (dict(Sq=0), INVALID), (dict(Sk=-1), INVALID), (dict(ro=-1), INVALID), (dict(co=-1), INVALID),
    (dict(ld=191), INVALID),                      # ld < col_off + Sk
    (dict(ld=(1 << 25) + 16), UNSUPPORTED), (dict(ld=1 << 25), UNSUPPORTED),
    (dict(q=None), INVALID), (dict(o=None), INVALID), (dict(lse=None), INVALID),
    (dict(do=None), INVALID), (dict(table=None), INVALID), (dict(dq=None), INVALID),
    (dict(dt=None), INVALID), (dict(k=None), INVALID), (dict(v=None), INVALID),
    (dict(spd=None), INVALID), (dict(dk=None), INVALID), (dict(dv=None), INVALID),
    (dict(nb=0), INVALID), (dict(nb=257), INVALID), (dict(scale=float("inf")), INVALID),
    (dict(d=24), UNSUPPORTED), (dict(dtype=3), UNSUPPORTED),
    (dict(q=MIS), INVALID), (dict(do=MIS), INVALID), (dict(dq=MIS), INVALID), (dict(dk=MIS), INVALID),
    (dict(ws=None), WORKSPACE), (dict(wsb=0), WORKSPACE), (dict(ws=FAKE + 16), WORKSPACE),
])
def test_bwd_ring_step_validation(kw, code):
    assert _bwd_ring(**kw) == code


def test_bwd_ring_step_empty_block_touches_nothing():
    """Sk = 0 is valid and launches nothing: the key-side pointers may be NULL
    (the call returns before any HIP call, so it runs without a device)."""
    assert _bwd_ring(Sk=0, k=None, v=None, spd=None, dk=None, dv=None) == OK


def test_bwd_ring_workspace_size():
    L = gt.lib()
    # two fp32 [H, Sq] arrays and fp32 [H, ceil(max(Sq, Sk)/256), 4], each padded to 256 bytes
    assert L.gt_attn_bwd_ring_workspace_size(8, 16384, 16384, 64, BF16) == \
        2 * 8 * 16384 * 4 + 8 * 64 * 4 * 4
    assert L.gt_attn_bwd_ring_workspace_size(2, 100, 1000, 64, BF16) == 2 * 1024 + 256
    assert L.gt_attn_bwd_ring_workspace_size(2, 1000, 0, 32, F32) == 2 * 8192 + 256
    assert L.gt_attn_bwd_ring_workspace_size(1, 0, 5, 32, F32) == 0
    assert L.gt_attn_bwd_ring_workspace_size(1, 4, -1, 32, F32) == 0


@pytest.mark.parametrize("kw,code", [
    (dict(P=0), INVALID), (dict(H=0), INVALID), (dict(S=0), INVALID), (dict(op=None), INVALID),
    (dict(lp=None), INVALID), (dict(o=None), INVALID), (dict(l=None), INVALID),
    (dict(d=12), UNSUPPORTED), (dict(dt=5), UNSUPPORTED), (dict(op=MIS), INVALID),
])
def test_merge_validation(kw, code):
    a = dict(op=FAKE, lp=FAKE, P=8, o=FAKE, l=FAKE, H=8, S=1000, d=64, dt=BF16)
    a.update(kw)
    assert gt.lib().gt_attn_merge(a["op"], a["lp"], a["P"], a["o"], a["l"], a["H"], a["S"],
                                  a["d"], a["dt"], None) == code


def test_binding_raises_without_device():
    """The Python binding has no CPU path: CPU tensors are rejected."""
    import torch
    q = torch.zeros(1, 4, 32)
    with pytest.raises(ValueError):
        gt.gt_attn_fwd(q, q, q, torch.zeros(4, 4, dtype=torch.uint8), torch.zeros(1, 3))
