"""The allocation-free backward (C ABI gt_attn_bwd_noalloc) against the
backward with a caller workspace (gt_attn_bwd), through the C ABI, on two
calls in a row, the second with a smaller input (the library's scratch keeps
the first call's contents), plus the size limit."""
import math

import numpy as np
import pytest
import torch

import paper_2609_34420_amd as gt
import synth
from gpu_common import DEV, rel_l2, say, to_np

pytestmark = pytest.mark.gpu

GT_BF16, GT_F32, GT_ERR_WORKSPACE = 1, 0, 3


def _case(H, N, d, nb, dtype, seed):
    g = np.random.default_rng(seed)
    td = torch.bfloat16 if dtype == "bf16" else torch.float32

    def t(x):
        x = synth.round_bf16(x) if dtype == "bf16" else x
        return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(td).to(DEV)

    q = t(g.standard_normal((H, N, d)) / math.sqrt(d))
    k = t(g.standard_normal((H, N, d)) / math.sqrt(d))
    v = t(g.standard_normal((H, N, d)))
    do = t(g.standard_normal((H, N, d)))
    spd = torch.from_numpy(g.integers(0, nb + 1, size=(N, N), dtype=np.uint8)).to(DEV)
    table = torch.from_numpy((g.standard_normal((H, nb)) * 0.3).astype(np.float32)).to(DEV)
    return q, k, v, do, spd, table


def _noalloc_c_abi(q, k, v, spd, table, o, lse, do, grads, scale):
    """gt_attn_bwd_noalloc called through the C ABI with raw pointers."""
    H, N, d = q.shape
    dq, dk, dv, dt = grads
    st = gt.lib().gt_attn_bwd_noalloc(
        q.data_ptr(), k.data_ptr(), v.data_ptr(), spd.data_ptr(), None, table.data_ptr(),
        table.shape[1], o.data_ptr(), lse.data_ptr(), do.data_ptr(), dq.data_ptr(), dk.data_ptr(),
        dv.data_ptr(), dt.data_ptr(), H, N, d, GT_BF16 if q.dtype == torch.bfloat16 else GT_F32,
        scale, torch.cuda.current_stream().cuda_stream)
    return st


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_noalloc_matches_workspace_backward(dtype):
    # the first call is the larger one; the second, smaller, reuses the scratch
    for H, N, d, nb in ((4, 700, 64, 30), (2, 300, 32, 12)):
        say(f"no-alloc backward {dtype} H={H} N={N} d={d}")
        q, k, v, do, spd, table = _case(H, N, d, nb, dtype, seed=N)
        scale = 1.0 / math.sqrt(d)
        o, lse = gt.gt_attn_fwd(q, k, v, spd, table, scale=scale)
        ref = gt.gt_attn_bwd(q, k, v, spd, table, o, lse, do, scale=scale)
        got = (torch.full_like(q, float("nan")), torch.full_like(k, float("nan")),
               torch.full_like(v, float("nan")), torch.full_like(table, float("nan")))
        assert _noalloc_c_abi(q, k, v, spd, table, o, lse, do, got, scale) == 0
        torch.cuda.synchronize()
        for name, a, b in zip(("dq", "dk", "dv"), got[:3], ref[:3]):
            assert torch.equal(a, b), (dtype, N, name)
        e = rel_l2(to_np(got[3]), to_np(ref[3]))
        say(f"no-alloc backward {dtype} N={N}: dq/dk/dv identical, dtable rel-L2 {e:.2e}")
        assert e <= 1e-5
        # the Python binding of the same entry point
        again = tuple(torch.empty_like(x) for x in got)
        gt.gt_attn_bwd_noalloc(q, k, v, spd, table, o, lse, do, again, scale=scale)
        torch.cuda.synchronize()
        for a, b in zip(again[:3], ref[:3]):
            assert torch.equal(a, b)


def test_noalloc_rejects_sizes_past_the_scratch():
    cap = gt.gt_attn_bwd_noalloc_max_bytes()
    assert cap == 16 << 20
    H, N = 8, 1 << 19          # workspace 32 MiB > 16 MiB
    assert gt.gt_attn_bwd_workspace_size(H, N, 64, torch.bfloat16) > cap
    fake = 0x10000
    st = gt.lib().gt_attn_bwd_noalloc(fake, fake, fake, fake, None, fake, 8, fake, fake, fake,
                                      fake, fake, fake, fake, H, N, 64, GT_BF16, 0.125, None)
    assert st == GT_ERR_WORKSPACE
