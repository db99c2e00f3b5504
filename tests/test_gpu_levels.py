"""GPU parity of MRA with any number of resolutions R = {s_0 > ... > 32, 1}
(Sec. 4.2 Alg. 1 refined level by level with a budget per block-row at every
level; Sec. 4.3 Alg. 2 over the resulting set) through the C ABI, against the
float64 oracle on the same seeded inputs. Selections: level 0 against the
oracle's scores of the scale-s_0 means, every later level against its scores
restricted to the candidates the GPU's previous level leaves, all exact except
near-ties (band 1e-6). Outputs: 1e-5 (float32 inputs) / 2e-2 (bfloat16 inputs)
max row-normwise relative error, the oracle evaluated under the GPU's
selections."""
import numpy as np
import pytest
import torch

from oracle import mra_oracle as O
from paper_2207_10284_amd import inputs
from tests.parity import TOL, check_selection, dev, err_stats, host, record, row_rel_err

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)


def _check_selections(idx, q, k, scales, budgets):
    """idx: one head's selections per level. Returns the rows (all levels)
    that differ from the oracle's by near-ties."""
    differ = 0
    for l, (s, m) in enumerate(zip(scales, budgets)):
        S = O.coarse_logits(O.block_mean(q, s), O.block_mean(k, s))
        if l > 0:
            p = scales[l - 1] // s
            masked = np.full_like(S, -np.inf)
            for x in range(S.shape[0]):
                cand = [int(Y) * p + t for Y in idx[l - 1][x // p] for t in range(p)]
                masked[x, cand] = S[x, cand]
            S = masked
        differ += check_selection(idx[l], S, m)
    return differ


def _run(gpu, q, k, v, scales, budgets, dtype, lse=False):
    B, H, n, d = q.shape
    outs = [torch.empty(B, H, n // s, m, dtype=torch.int32, device="cuda") for s, m in zip(scales, budgets)]
    lse_t = torch.empty(B, H, n, dtype=torch.float32, device="cuda") if lse else None
    out = gpu.attention_forward_levels(dev(q, dtype), dev(k, dtype), dev(v, dtype), scales, budgets,
                                       idx_outs=outs, lse_out=lse_t)
    torch.cuda.synchronize()
    idx = [host(t).astype(np.int64) for t in outs]
    return (out, idx, lse_t) if lse else (out, idx)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("d", [32, 64, 128])
@pytest.mark.parametrize("B,H,n,scales,budgets", [
    (1, 1, 128, (128, 64, 32), (1, 2, 3)),
    (2, 3, 512, (256, 64, 32), (1, 3, 4)),
    (1, 2, 1024, (512, 128, 64, 32), (2, 5, 7, 9)),
    (1, 1, 1024, (256, 128, 32), (0, 0, 0)),
    (1, 2, 1152, (384, 96, 32), (2, 5, 11)),
    (2, 1, 2048, (1024, 256, 128, 64, 32), (1, 3, 5, 8, 12)),
    (1, 1, 2048, (512, 128, 32), (4, 16, 64)),
])
def test_levels_small(gpu, dtype, d, B, H, n, scales, budgets):
    _say("levels", dtype, d, B, H, n, scales, budgets)
    q, k, v = inputs.random_qkv(1500 + d + n + sum(budgets), B, H, n, d, dtype, scale=1.2)
    out, idx = _run(gpu, q, k, v, scales, budgets, dtype)
    Z = np.empty(q.shape)
    for b in range(B):
        for h in range(H):
            ih = [i[b, h] for i in idx]
            _check_selections(ih, q[b, h], k[b, h], scales, budgets)
            Z[b, h], _ = O.mra_levels_factored(q[b, h], k[b, h], v[b, h], scales, budgets, idx=ih)
    err = row_rel_err(host(out), Z)
    assert err <= TOL[dtype], err


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_levels_one_scale_is_the_two_level_forward(gpu, dtype):
    """R = {32, 1}: bit-identical to mra_attention_forward (output, selection,
    log normalisers)."""
    q, k, v = (dev(a, dtype) for a in inputs.random_qkv(1601, 2, 3, 1024, 64, dtype, scale=1.2))
    i1 = torch.empty(2, 3, 32, 7, dtype=torch.int32, device="cuda")
    l1 = torch.empty(2, 3, 1024, dtype=torch.float32, device="cuda")
    a = gpu.attention_forward_levels(q, k, v, (32,), (7,), idx_outs=[i1], lse_out=l1)
    i2 = torch.empty_like(i1)
    l2 = torch.empty_like(l1)
    b = gpu.attention_forward(q, k, v, 7, idx_out=i2, lse_out=l2)
    torch.cuda.synchronize()
    assert torch.equal(a, b) and torch.equal(i1, i2) and torch.equal(l1, l2)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_levels_transparent_middle_level(gpu, dtype):
    """A middle level that keeps every candidate changes nothing: the finest
    selection and the output equal those without it, bit for bit (its blocks
    enter the coarse term with weight zero)."""
    q, k, v = inputs.random_qkv(1602, 1, 2, 2048, 64, dtype, scale=1.2)
    a, ia = _run(gpu, q, k, v, (512, 128, 32), (2, 8, 11), dtype)
    b, ib = _run(gpu, q, k, v, (512, 32), (2, 11), dtype)
    assert np.array_equal(ia[0], ib[0]) and np.array_equal(ia[2], ib[1])
    assert torch.equal(a, b)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_levels_full_budgets_exact(gpu, dtype):
    """Every block kept at every level: exact softmax attention."""
    q, k, v = inputs.random_qkv(1603, 1, 2, 512, 64, dtype, scale=1.0)
    out, idx = _run(gpu, q, k, v, (256, 64, 32), (2, 8, 16), dtype)
    assert (idx[2] == np.arange(16)).all()
    ref = np.stack([np.stack([O.exact_attention(q[0, h], k[0, h], v[0, h]) for h in range(2)])])
    assert row_rel_err(host(out), ref) <= TOL[dtype]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_levels_repeat_smaller_call_and_lse(gpu, dtype):
    """Two calls in a row, the second on a smaller input with other scales,
    give the results of fresh calls; the log normalisers are those of the
    oracle's output rows."""
    q, k, v = inputs.random_qkv(1604, 2, 2, 1024, 64, dtype, scale=1.0)
    a, _ = _run(gpu, q, k, v, (256, 64, 32), (2, 5, 6), dtype)
    a2, _ = _run(gpu, q, k, v, (256, 64, 32), (2, 5, 6), dtype)
    assert torch.equal(a, a2)
    qs, ks, vs = q[:1, :1, :512], k[:1, :1, :512], v[:1, :1, :512]
    b, idx, lse = _run(gpu, qs, ks, vs, (128, 64, 32), (2, 3, 4), dtype, lse=True)
    ih = [i[0, 0] for i in idx]
    Z, _ = O.mra_levels_factored(qs[0, 0], ks[0, 0], vs[0, 0], (128, 64, 32), (2, 3, 4), idx=ih)
    assert row_rel_err(host(b)[0, 0], Z) <= TOL[dtype]
    # ln of the row sum of A^: from the dense slab of each finest block-row
    want = np.concatenate([np.log(np.exp(O.levels_logits_slab(qs[0, 0], ks[0, 0], (128, 64, 32), ih, x)).sum(axis=1))
                           for x in range(16)])
    assert np.abs(host(lse)[0, 0] - want).max() <= (1e-5 if dtype == "f32" else 2e-2)


@pytest.mark.parametrize("name", list(inputs.WORKLOADS))
def test_levels_workload_full_size(gpu, name):
    """Each workload at its real shape with four resolutions; every block-row
    of every head checked against the oracle under the GPU's selections, which
    are checked against the oracle's scores at every level."""
    w = inputs.WORKLOADS[name]
    scales, budgets = inputs.LEVELS[name]
    _say("levels workload", name, scales, budgets)
    q, k, v = inputs.make_qkv(w)
    out, idx = _run(gpu, q, k, v, scales, budgets, w.dtype)
    out_h = host(out)
    del out
    Zall = np.empty(out_h.shape)
    differ = 0
    for b in range(w.B):
        for h in range(w.H):
            qh, kh, vh = q[b, h].astype(np.float64), k[b, h].astype(np.float64), v[b, h].astype(np.float64)
            ih = [i[b, h] for i in idx]
            differ += _check_selections(ih, qh, kh, scales, budgets)
            Zall[b, h], _ = O.mra_levels_factored(qh, kh, vh, scales, budgets, idx=ih)
    st = err_stats(out_h, Zall)
    record(f"four resolutions R = {{{', '.join(map(str, scales))}, 1}}, budgets {'/'.join(map(str, budgets))}",
           name, w.dtype, w.B * w.H, w.B * w.H * w.nb, st, TOL[w.dtype], differ, note="tie rows at all levels")
    _say("  levels", name, "worst", st["row"])
    assert st["row"] <= TOL[w.dtype]
