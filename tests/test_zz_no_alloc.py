"""The entry point that allocates nothing (mra_attention_forward_noalloc),
called through the C ABI, against mra_attention_forward with a caller's
workspace: the same kernels, so selection, output and log normalisers must be
bit-identical, on two calls in a row (the second on a smaller input, so the
static scratch holds the first call's intermediates when it starts), and the
output within the forward's bar of the float64 oracle."""
import ctypes

import numpy as np
import pytest
import torch

from oracle import mra_oracle as O
from paper_2207_10284_amd import inputs
from tests.parity import TOL, check_selection, dev, host, row_rel_err

pytestmark = pytest.mark.gpu


def _noalloc(lib, tq, tk, tv, budget):
    """Direct C-ABI call; returns (status, out, idx, lse)."""
    B, H, n, d = tq.shape
    out = torch.empty_like(tq)
    idx = torch.empty(B, H, n // 32, budget, dtype=torch.int32, device=tq.device)
    lse = torch.empty(B, H, n, dtype=torch.float32, device=tq.device)
    code = 1 if tq.dtype == torch.bfloat16 else 0
    stream = torch.cuda.current_stream(tq.device).cuda_stream
    st = lib.mra_attention_forward_noalloc(tq.data_ptr(), tk.data_ptr(), tv.data_ptr(), out.data_ptr(),
                                           idx.data_ptr(), lse.data_ptr(), B, H, n, d, 32, budget, code,
                                           ctypes.c_void_p(stream))
    return st, out, idx, lse


def _with_workspace(gpu, tq, tk, tv, budget):
    B, H, n, d = tq.shape
    idx = torch.empty(B, H, n // 32, budget, dtype=torch.int32, device=tq.device)
    lse = torch.empty(B, H, n, dtype=torch.float32, device=tq.device)
    out = gpu.attention_forward(tq, tk, tv, budget, idx_out=idx, lse_out=lse)
    return out, idx, lse


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_noalloc_matches_forward_twice(gpu, dtype):
    lib = gpu.load()
    cases = [(2, 3, 4096, 64, 16, 41), (1, 2, 1024, 32, 5, 42)]       # second call smaller
    for B, H, n, d, m, seed in cases:
        print("noalloc", dtype, B, H, n, d, m, flush=True)
        q, k, v = inputs.random_qkv(seed, B, H, n, d, dtype, scale=1.2)
        tq, tk, tv = dev(q, dtype), dev(k, dtype), dev(v, dtype)
        st, out, idx, lse = _noalloc(lib, tq, tk, tv, m)
        assert st == 0, lib.mra_status_str(st).decode()
        ref_out, ref_idx, ref_lse = _with_workspace(gpu, tq, tk, tv, m)
        torch.cuda.synchronize()
        assert torch.equal(idx, ref_idx)
        assert torch.equal(out, ref_out)
        assert torch.equal(lse, ref_lse)
        gi = host(idx).astype(np.int64)
        for b in range(B):
            for h in range(H):
                S = O.coarse_logits(O.block_mean(q[b, h], 32), O.block_mean(k[b, h], 32))
                check_selection(gi[b, h], S, m)
        Z, _ = O.mra_batched(q, k, v, 32, m, idx=gi)
        assert row_rel_err(host(out), Z) <= TOL[dtype]


def test_noalloc_rejects_too_large(gpu):
    lib = gpu.load()
    t = torch.zeros(1, 1, 64, 64, device="cuda", dtype=torch.bfloat16)
    # 128 heads of 32k tokens at d = 128 need ~285 MB of workspace: rejected
    # before anything is enqueued (the pointers are never read)
    st = lib.mra_attention_forward_noalloc(t.data_ptr(), t.data_ptr(), t.data_ptr(), t.data_ptr(), None, None,
                                           1, 128, 32768, 128, 32, 32, 1, None)
    assert st == 6
