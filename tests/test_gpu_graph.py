"""The forward (with a caller's workspace and the entry point that allocates
nothing) and the backward captured into HIP graphs: every replay, with eager
work and synchronisations between replays, is bit-identical to the eager
calls. Covers the round-by-round launch of the tile pass (a head whose K and
V exceed an XCD's L2) and the any-depth forward. No call records a memset:
every buffer the kernels clear is cleared by a kernel."""
import ctypes

import numpy as np
import pytest
import torch

from paper_2207_10284_amd import inputs
from tests.parity import dev

pytestmark = pytest.mark.gpu


def _replay_and_compare(g, outs, refs, eager_between):
    for rep in range(3):
        for t in outs:
            t.zero_()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for t, r in zip(outs, refs):
            assert torch.equal(t, r), f"replay {rep} differs"
        eager_between()
        torch.cuda.synchronize()


@pytest.mark.parametrize("dtype,B,H,n,d,m", [("bf16", 2, 3, 2048, 64, 8), ("f32", 1, 2, 1024, 32, 5),
                                             ("bf16", 1, 2, 16384, 128, 16)])
def test_forward_in_a_graph(gpu, dtype, B, H, n, d, m):
    print("graph forward", dtype, B, H, n, d, m, flush=True)
    q, k, v = (dev(a, dtype) for a in inputs.random_qkv(1700 + n + d, B, H, n, d, dtype, scale=1.2))
    q2, k2, v2 = (dev(a, dtype) for a in inputs.random_qkv(1701 + n, B, H, n, d, dtype, scale=0.7))
    nb = n // 32
    ws = torch.empty(gpu.forward_workspace_bytes(B, H, n, d, m, q.dtype), dtype=torch.uint8, device="cuda")
    out = torch.empty_like(q)
    idx = torch.empty(B, H, nb, m, dtype=torch.int32, device="cuda")
    lse = torch.empty(B, H, n, dtype=torch.float32, device="cuda")
    ref = gpu.attention_forward(q, k, v, m, idx_out=idx, lse_out=lse, workspace=ws).clone()
    ref_idx, ref_lse = idx.clone(), lse.clone()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        gpu.attention_forward(q, k, v, m, out=out, idx_out=idx, lse_out=lse, workspace=ws)   # warm-up
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    with torch.cuda.graph(g):
        gpu.attention_forward(q, k, v, m, out=out, idx_out=idx, lse_out=lse, workspace=ws)
    # eager work between replays: another forward on other inputs, same workspace
    other = lambda: gpu.attention_forward(q2, k2, v2, m, workspace=ws)
    _replay_and_compare(g, [out, idx, lse], [ref, ref_idx, ref_lse], other)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_noalloc_forward_in_a_graph(gpu, dtype):
    B, H, n, d, m = 2, 2, 2048, 64, 8
    print("graph noalloc", dtype, flush=True)
    lib = gpu.load()
    q, k, v = (dev(a, dtype) for a in inputs.random_qkv(1710, B, H, n, d, dtype, scale=1.2))
    q2 = dev(inputs.random_qkv(1711, 1, 1, 1024, d, dtype, scale=1.0)[0], dtype)
    out = torch.empty_like(q)
    idx = torch.empty(B, H, n // 32, m, dtype=torch.int32, device="cuda")
    lse = torch.empty(B, H, n, dtype=torch.float32, device="cuda")
    code = 1 if dtype == "bf16" else 0

    def call(stream, qq=q, kk=k, vv=v, o=out, i=idx, l=lse):
        Bq, Hq, nq, dq = qq.shape
        st = lib.mra_attention_forward_noalloc(qq.data_ptr(), kk.data_ptr(), vv.data_ptr(), o.data_ptr(),
                                               i.data_ptr(), l.data_ptr(), Bq, Hq, nq, dq, 32, m if i is idx else 4,
                                               code, ctypes.c_void_p(stream.cuda_stream))
        assert st == 0, lib.mra_status_str(st).decode()

    call(torch.cuda.current_stream())
    torch.cuda.synchronize()
    ref, ref_idx, ref_lse = out.clone(), idx.clone(), lse.clone()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call(torch.cuda.current_stream())
    o2 = torch.empty_like(q2)
    i2 = torch.empty(1, 1, 32, 4, dtype=torch.int32, device="cuda")
    l2 = torch.empty(1, 1, 1024, dtype=torch.float32, device="cuda")
    # eager work between replays: a smaller call that reuses the static scratch
    other = lambda: call(torch.cuda.current_stream(), q2, q2, q2, o2, i2, l2)
    _replay_and_compare(g, [out, idx, lse], [ref, ref_idx, ref_lse], other)


def test_levels_and_backward_in_a_graph(gpu):
    B, H, n, d, m = 1, 3, 2048, 64, 8
    print("graph levels + backward", flush=True)
    q, k, v = (dev(a, "bf16") for a in inputs.random_qkv(1720, B, H, n, d, "bf16", scale=1.2))
    gz = dev(np.random.Generator(np.random.PCG64(1721)).standard_normal((B, H, n, d)), "bf16")
    scales, budgets = (512, 128, 32), (2, 6, m)
    lws = torch.empty(gpu.forward_levels_workspace_bytes(B, H, n, d, scales, budgets, q.dtype),
                      dtype=torch.uint8, device="cuda")
    bws = torch.empty(gpu.backward_workspace_bytes(B, H, n, d, q.dtype), dtype=torch.uint8, device="cuda")
    lout = torch.empty_like(q)
    idx = torch.empty(B, H, n // 32, m, dtype=torch.int32, device="cuda")
    lse = torch.empty(B, H, n, dtype=torch.float32, device="cuda")
    out = gpu.attention_forward(q, k, v, m, idx_out=idx, lse_out=lse)
    dq, dk, dv = (torch.empty_like(q) for _ in range(3))

    def work():
        gpu.attention_forward_levels(q, k, v, scales, budgets, out=lout, workspace=lws)
        gpu.attention_backward(q, k, v, out, gz, lse, idx, dq=dq, dk=dk, dv=dv, workspace=bws)

    work()
    torch.cuda.synchronize()
    refs = [lout.clone(), dq.clone(), dk.clone(), dv.clone()]
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        work()
    _replay_and_compare(g, [lout, dq, dk, dv], refs, lambda: gpu.attention_forward(k, q, v, m))


@pytest.mark.parametrize("dtype,d", [("bf16", 64), ("f32", 32)])
def test_training_step_in_a_graph(gpu, dtype, d):
    """A training step of the layer as one graph: the forward with log
    normalisers, then the backward given the forward's block means (views of
    the forward's workspace); every replay matches the eager step bit for
    bit."""
    B, H, n, m = 2, 2, 1024, 6
    print("graph training step", dtype, d, flush=True)
    q, k, v = (dev(a, dtype) for a in inputs.random_qkv(1730 + d, B, H, n, d, dtype, scale=1.1))
    gz = dev(np.random.Generator(np.random.PCG64(1731)).standard_normal((B, H, n, d)), dtype)
    ws = torch.empty(gpu.forward_workspace_bytes(B, H, n, d, m, q.dtype), dtype=torch.uint8, device="cuda")
    bws = torch.empty(gpu.backward_workspace_bytes(B, H, n, d, q.dtype), dtype=torch.uint8, device="cuda")
    pooled = gpu.forward_pooled_rows(ws, B, H, n, d)
    out = torch.empty_like(q)
    idx = torch.empty(B, H, n // 32, m, dtype=torch.int32, device="cuda")
    lse = torch.empty(B, H, n, dtype=torch.float32, device="cuda")
    dq, dk, dv = (torch.empty_like(q) for _ in range(3))

    def work():
        gpu.attention_forward(q, k, v, m, out=out, idx_out=idx, workspace=ws, lse_out=lse)
        gpu.attention_backward(q, k, v, out, gz, lse, idx, dq=dq, dk=dk, dv=dv, workspace=bws, pooled=pooled)

    work()
    torch.cuda.synchronize()
    refs = [t.clone() for t in (out, lse, dq, dk, dv)]
    plain = gpu.attention_backward(q, k, v, out, gz, lse, idx)
    for a, b in zip(plain, refs[2:]):
        assert torch.equal(a, b)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        work()
    _replay_and_compare(g, [out, lse, dq, dk, dv], refs, lambda: gpu.attention_forward(k, q, v, m))
