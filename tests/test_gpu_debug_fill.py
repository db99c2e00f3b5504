"""The NaN-fill debug flag (MRA_DEBUG_NANFILL=1): every computing entry point
first fills its outputs and the part of the workspace it uses with quiet NaN
(index outputs with the same bits). Every result must come out bit-identical
to a run without the flag, which shows that each output element is written by
the call and that no kernel reads a workspace or output value before the
call wrote it."""
import numpy as np
import pytest
import torch

from paper_2207_10284_amd import inputs
from tests.parity import dev

pytestmark = pytest.mark.gpu


def _both(monkeypatch, fn):
    """fn() without and with the flag; returns the two result tuples."""
    monkeypatch.delenv("MRA_DEBUG_NANFILL", raising=False)
    a = fn()
    torch.cuda.synchronize()
    monkeypatch.setenv("MRA_DEBUG_NANFILL", "1")
    b = fn()
    torch.cuda.synchronize()
    monkeypatch.delenv("MRA_DEBUG_NANFILL", raising=False)
    return a, b


def _same(a, b):
    for x, y in zip(a, b):
        assert torch.equal(x, y)
        if x.is_floating_point():
            assert torch.isfinite(x.float()).all()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("d", [32, 64, 128])
def test_forwards_write_every_output(gpu, monkeypatch, dtype, d):
    B, H, n, m = 2, 3, 320, 3
    q, k, v = (dev(a, dtype) for a in inputs.random_qkv(4100 + d, B, H, n, d, dtype, scale=1.3))
    nb = n // 32

    def run():
        idx = torch.empty(B, H, nb, m, dtype=torch.int32, device="cuda")
        lse = torch.empty(B, H, n, dtype=torch.float32, device="cuda")
        out = gpu.attention_forward(q, k, v, m, idx_out=idx, lse_out=lse)
        sidx = torch.empty_like(idx)
        slse = torch.empty_like(lse)
        sout = gpu.sparse_attention_forward(q, k, v, m, idx_out=sidx, lse_out=slse)
        nidx = torch.empty_like(idx)
        nout = gpu.attention_forward_noalloc(q, k, v, m, idx_out=nidx)
        gidx = torch.empty(B, H, nb, nb, dtype=torch.int32, device="cuda")
        gout = gpu.attention_forward_global(q, k, v, 11, True, idx_out=gidx)
        i1 = torch.empty(B, H, n // 64, 2, dtype=torch.int32, device="cuda")
        i2 = torch.empty(B, H, nb, m, dtype=torch.int32, device="cuda")
        mout = gpu.attention_forward_multilevel(q, k, v, 64, 2, m, idx1_out=i1, idx2_out=i2)
        l0 = torch.empty(B, H, 1, 1, dtype=torch.int32, device="cuda")
        l1 = torch.empty(B, H, 2, 1, dtype=torch.int32, device="cuda")
        l2 = torch.empty(B, H, nb, m, dtype=torch.int32, device="cuda")
        lout = gpu.attention_forward_levels(q, k, v, (320, 160, 32), (1, 1, m), idx_outs=[l0, l1, l2])
        return out, idx, lse, sout, sidx, slse, nout, nidx, gout, gidx, mout, i1, i2, lout, l0, l1, l2

    a, b = _both(monkeypatch, run)
    _same(a, b)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_steps_write_every_output(gpu, monkeypatch, dtype):
    q, k, v = (dev(a, dtype) for a in inputs.random_qkv(4200, 2, 2, 384, 64, dtype, scale=1.1))

    def run():
        qp, kp, vp = gpu.pool(q, k, v)
        S = gpu.coarse_scores(qp, kp)
        idx = gpu.select(S, 4)
        gidx = gpu.select_global(S, 30, True)
        cm, cs, cv = gpu.coarse_term(S, idx, vp)
        lse = torch.empty(2, 2, 384, dtype=torch.float32, device="cuda")
        out = gpu.block_sddmm_spmm(q, k, v, idx, cm, cs, cv, lse_out=lse)
        sout = gpu.block_sddmm_spmm(q, k, v, idx)
        return qp, kp, vp, S, idx, gidx, cm, cs, cv, out, lse, sout

    a, b = _both(monkeypatch, run)
    _same(a, b)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("d", [32, 64, 128])
def test_backward_writes_every_gradient(gpu, monkeypatch, dtype, d):
    B, H, n, m = 1, 2, 256, 3
    q, k, v = (dev(a, dtype) for a in inputs.random_qkv(4300 + d, B, H, n, d, dtype, scale=1.0))
    g = dev(np.random.Generator(np.random.PCG64(4301)).standard_normal((B, H, n, d)), dtype)
    idx = torch.empty(B, H, n // 32, m, dtype=torch.int32, device="cuda")
    lse = torch.empty(B, H, n, dtype=torch.float32, device="cuda")
    out = gpu.attention_forward(q, k, v, m, idx_out=idx, lse_out=lse)

    def run():
        return gpu.attention_backward(q, k, v, out, g, lse, idx)

    a, b = _both(monkeypatch, run)
    _same(a, b)
    # given the block means, the backward reads them and not its workspace's
    # (NaN-filled) copy
    pooled = gpu.pool(q, k, v)

    def run_pooled():
        return gpu.attention_backward(q, k, v, out, g, lse, idx, pooled=pooled)

    c, e = _both(monkeypatch, run_pooled)
    _same(c, e)
    _same(a, c)
