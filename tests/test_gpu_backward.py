"""GPU parity of the gradient pass (mra_attention_backward: dQ, dK, dV with the
selection held fixed) and of the forward's per-query log normalisers, through
the C ABI, against the float64 oracle on the same seeded inputs:
``O.mra_grads`` (torch float64 autograd of the factored form) and
``O.mra_lse``, both evaluated under the GPU's own selection.

Metrics, per head and tensor:
* row error against the term magnitudes: max over rows i of
  ||err_i||_inf / ||M_i||_inf, where M = O.mra_grad_terms(..., absolute=True)
  sums the magnitudes of the terms each gradient element is a sum of. A
  gradient row is a sum of many signed terms (the logit gradients
  p (G.v - delta) of a row sum to zero), so its own magnitude can be far below
  its terms' and relative to itself it carries the rounding of the terms
  magnified by that ratio; against M the first-order rounding bound is the
  number of roundings times the unit roundoff. bfloat16 inputs: the
  probabilities and logit gradients are rounded to bfloat16 (u = 2^-8) before
  the matrix-core products (a logit gradient from an already rounded
  probability: two roundings) and the result once more: at most 3 u = 1.2e-2
  to first order, bar 1.5e-2. float32 inputs: float32 logits, products and
  sums: bar 1e-4;
* max|err| / max|ref| over the whole tensor (<= 2e-5 float32, 2e-2 bfloat16).
Log normalisers: |err| <= 1e-5 (float32) or 4e-3 (bfloat16: rounded weights
change the row sum by at most u = 2^-8 relative) times max(1, |L|)."""
import numpy as np
import pytest
import torch

from oracle import mra_oracle as O
from paper_2207_10284_amd import inputs
from tests.parity import dev, host, record

pytestmark = pytest.mark.gpu

GRAD_TOL = {"f32": 2e-5, "bf16": 2e-2}        # max|err| / max|ref|
GRAD_ROW_TOL = {"f32": 1e-4, "bf16": 1.5e-2}  # row error / term magnitudes
LSE_TOL = {"f32": 1e-5, "bf16": 4e-3}


def _say(*a):
    print(*a, flush=True)


def _case(index, B, H, n, d, dtype, budget, kind="ar1"):
    """Seeded inputs of one test case (the workload recipe at a small shape)
    and an output gradient G ~ N(0, 1), all exact in the compute dtype."""
    w = inputs.Workload(f"grad-{index}", 100 + index, B=B, H=H, n=n, d=d, dtype=dtype, budget=budget,
                        kind=kind, rho=0.9, s2=1.0)
    q, k, v = inputs.make_qkv(w)
    g = np.random.Generator(np.random.PCG64(w.seed + 7)).standard_normal(q.shape)
    g = inputs.round_to_bf16(g) if dtype == "bf16" else g.astype(np.float32)
    return q, k, v, g


def _rel(a, ref):
    return float(np.abs(a - ref).max() / max(np.abs(ref).max(), 1e-30))


def _rowerr(a, ref, mag):
    """max over rows (tokens) of ||a_i - ref_i||_inf / ||mag_i||_inf."""
    return float((np.abs(a - ref).max(axis=-1) / np.maximum(np.abs(mag).max(axis=-1), 1e-300)).max())


def _fro(a, ref):
    return float(np.sqrt(((a - ref) ** 2).sum()) / max(np.sqrt((ref ** 2).sum()), 1e-300))


def _forward(gpu, variant, tq, tk, tv, budget, prior=False):
    B, H, n, d = tq.shape
    nb = n // 32
    lse = torch.empty(B, H, n, dtype=torch.float32, device="cuda")
    if variant == "global":
        idx = torch.empty(B, H, nb, nb, dtype=torch.int32, device="cuda")
        out = gpu.attention_forward_global(tq, tk, tv, budget, prior, idx_out=idx, lse_out=lse)
    else:
        idx = torch.empty(B, H, nb, budget, dtype=torch.int32, device="cuda")
        fwd = gpu.attention_forward if variant == "mra2" else gpu.sparse_attention_forward
        out = fwd(tq, tk, tv, budget, idx_out=idx, lse_out=lse)
    return out, idx, lse


def _check(gpu, variant, q, k, v, g, budget, dtype, prior=False, heads=None):
    """Forward (with log normalisers) and backward on the GPU; the sampled
    heads (all by default) against the oracle. Returns the worst errors."""
    tq, tk, tv, tg = dev(q, dtype), dev(k, dtype), dev(v, dtype), dev(g, dtype)
    out, idx, lse = _forward(gpu, variant, tq, tk, tv, budget, prior)
    coarse = variant != "mra2s"
    dq, dk, dv = gpu.attention_backward(tq, tk, tv, out, tg, lse, idx, coarse=coarse)
    torch.cuda.synchronize()
    gi = host(idx).astype(np.int64)
    L = host(lse)
    grads = [host(t) for t in (dq, dk, dv)]
    B, H = q.shape[:2]
    heads = [(b, h) for b in range(B) for h in range(H)] if heads is None else heads
    worst = {"lse": 0.0, "dq": 0.0, "dk": 0.0, "dv": 0.0, "dq_row": 0.0, "dk_row": 0.0, "dv_row": 0.0,
             "dq_fro": 0.0, "dk_fro": 0.0, "dv_fro": 0.0}
    for b, h in heads:
        qh, kh, vh, gh = (a[b, h].astype(np.float64) for a in (q, k, v, g))
        Lref = O.mra_lse(qh, kh, 32, gi[b, h], coarse)
        worst["lse"] = max(worst["lse"], float((np.abs(L[b, h] - Lref) / np.maximum(1.0, np.abs(Lref))).max()))
        ref = O.mra_grads(qh, kh, vh, gh, 32, gi[b, h], coarse)
        mags = O.mra_grad_terms(qh, kh, vh, gh, 32, gi[b, h], coarse, absolute=True)
        for name, got, want, mag in zip(("dq", "dk", "dv"), grads, ref, mags):
            worst[name] = max(worst[name], _rel(got[b, h], want))
            worst[name + "_row"] = max(worst[name + "_row"], _rowerr(got[b, h], want, mag))
            worst[name + "_fro"] = max(worst[name + "_fro"], _fro(got[b, h], want))
    _say(" ", variant, q.shape, dtype, budget, {k_: f"{e:.2e}" for k_, e in worst.items()})
    assert worst["lse"] <= LSE_TOL[dtype], worst
    for name in ("dq", "dk", "dv"):
        assert worst[name] <= GRAD_TOL[dtype], (name, worst)
        assert worst[name + "_row"] <= GRAD_ROW_TOL[dtype], (name, worst)
    return worst


def _record_grads(label, w, heads, worst):
    for name in ("dq", "dk", "dv"):
        record(f"backward {name} ({label})", w.name, w.dtype, len(heads), len(heads) * w.nb,
               {"row": worst[name + "_row"], "global": worst[name], "fro": worst[name + "_fro"]},
               GRAD_ROW_TOL[w.dtype], "-", note="row error / term magnitudes; whole heads")


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("d", [32, 64, 128])
@pytest.mark.parametrize("n,budget", [(256, 0), (256, 3), (256, 8), (96, 1)])
def test_backward_mra2(gpu, n, budget, d, dtype):
    """Per-row budget: no refined block (all coarse), a few, all of them
    (exact attention), and a three-block sequence."""
    _say("mra2 backward", n, budget, d, dtype)
    q, k, v, g = _case(d + n + budget, 2, 2, n, d, dtype, budget)
    _check(gpu, "mra2", q, k, v, g, budget, dtype)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_backward_mra2_many_blocks(gpu, dtype):
    """66 blocks per side: the coarse passes span two 64-block chunks with a
    ragged tail, and the column lists two ballot steps."""
    _say("mra2 backward 66 blocks", dtype)
    q, k, v, g = _case(7, 1, 2, 66 * 32, 64, dtype, 5, kind="hub")
    _check(gpu, "mra2", q, k, v, g, 5, dtype)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("d", [32, 64, 128])
@pytest.mark.parametrize("n,budget", [(256, 1), (256, 3), (256, 8)])
def test_backward_mra2s(gpu, n, budget, d, dtype):
    """MRA-2-s: softmax over the refined blocks only (no coarse part)."""
    _say("mra2s backward", n, budget, d, dtype)
    q, k, v, g = _case(500 + d + n + budget, 2, 2, n, d, dtype, budget)
    _check(gpu, "mra2s", q, k, v, g, budget, dtype)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("budget,prior", [(0, False), (5, False), (12, True), (64, False)])
def test_backward_global(gpu, budget, prior, dtype):
    """Head-wide budget: rows refine different numbers of blocks (some none),
    selection rows padded with -1."""
    _say("global backward", budget, prior, dtype)
    q, k, v, g = _case(900 + budget, 1, 3, 256, 64, dtype, budget)
    _check(gpu, "global", q, k, v, g, budget, dtype, prior)


def test_autograd_function_matches_entry_points(gpu):
    """ops.mra_attention (torch.autograd.Function over the two entry points)
    gives the forward's output and the backward entry point's gradients, bit
    for bit."""
    q, k, v, g = _case(31, 1, 2, 256, 64, "bf16", 3)
    tq, tk, tv, tg = dev(q, "bf16"), dev(k, "bf16"), dev(v, "bf16"), dev(g, "bf16")
    for variant in ("mra2", "mra2s", "global"):
        budget = 20 if variant == "global" else 3
        aq, ak, av = (t.clone().requires_grad_(True) for t in (tq, tk, tv))
        z = gpu.mra_attention(aq, ak, av, budget, variant, prior_diagonal=True)
        z.backward(tg)
        out, idx, lse = _forward(gpu, variant, tq, tk, tv, budget, True)
        dq, dk, dv = gpu.attention_backward(tq, tk, tv, out, tg, lse, idx, coarse=variant != "mra2s")
        assert torch.equal(z.detach(), out)
        for a, b_ in ((aq.grad, dq), (ak.grad, dk), (av.grad, dv)):
            assert torch.equal(a, b_), variant


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("d", [32, 64, 128])
@pytest.mark.parametrize("variant", ["mra2", "global", "mra2s"])
def test_backward_with_forward_pooled_rows(gpu, variant, d, dtype):
    """The forward's block means, read from its workspace
    (mra_forward_pooled_rows), are mra_pool's bits, and the backward that
    takes them (mra_attention_backward_pooled) gives the plain backward's
    gradients bit for bit (MRA-2-s does not read them)."""
    q, k, v, g = _case(51, 2, 3, 320, d, dtype, 4)
    tq, tk, tv, tg = dev(q, dtype), dev(k, dtype), dev(v, dtype), dev(g, dtype)
    B, H, n, _ = tq.shape
    nb = n // 32
    lse = torch.empty(B, H, n, dtype=torch.float32, device="cuda")
    if variant == "global":
        idx = torch.empty(B, H, nb, nb, dtype=torch.int32, device="cuda")
        ws = torch.empty(gpu.forward_global_workspace_bytes(B, H, n, d, tq.dtype), dtype=torch.uint8, device="cuda")
        out = gpu.attention_forward_global(tq, tk, tv, 17, True, idx_out=idx, workspace=ws, lse_out=lse)
        pooled = gpu.forward_pooled_rows(ws, B, H, n, d)
    else:
        idx = torch.empty(B, H, nb, 4, dtype=torch.int32, device="cuda")
        ws = torch.empty(gpu.forward_workspace_bytes(B, H, n, d, 4, tq.dtype), dtype=torch.uint8, device="cuda")
        fwd = gpu.attention_forward if variant == "mra2" else gpu.sparse_attention_forward
        out = fwd(tq, tk, tv, 4, idx_out=idx, workspace=ws, lse_out=lse)
        pooled = gpu.forward_pooled_rows(ws, B, H, n, d) if variant == "mra2" else gpu.pool(tq, tk, tv)
    torch.cuda.synchronize()
    for got, want in zip(pooled, gpu.pool(tq, tk, tv)):
        assert torch.equal(got, want)
    coarse = variant != "mra2s"
    plain = gpu.attention_backward(tq, tk, tv, out, tg, lse, idx, coarse=coarse)
    given = gpu.attention_backward(tq, tk, tv, out, tg, lse, idx, coarse=coarse, pooled=pooled)
    torch.cuda.synchronize()
    for a, b_ in zip(plain, given):
        assert torch.isfinite(a.float()).all()
        assert torch.equal(a, b_)


def test_backward_is_deterministic(gpu):
    """Two calls give identical bits (no atomics in any sum)."""
    q, k, v, g = _case(41, 2, 2, 512, 64, "bf16", 4)
    tq, tk, tv, tg = dev(q, "bf16"), dev(k, "bf16"), dev(v, "bf16"), dev(g, "bf16")
    out, idx, lse = _forward(gpu, "mra2", tq, tk, tv, 4)
    r1 = gpu.attention_backward(tq, tk, tv, out, tg, lse, idx)
    r2 = gpu.attention_backward(tq, tk, tv, out, tg, lse, idx)
    for a, b_ in zip(r1, r2):
        assert torch.equal(a, b_)


def test_backward_empty_and_errors(gpu):
    e = torch.zeros(0, 2, 64, 64, device="cuda", dtype=torch.bfloat16)
    lse = torch.zeros(0, 2, 64, device="cuda")
    idx = torch.zeros(0, 2, 2, 1, device="cuda", dtype=torch.int32)
    dq, dk, dv = gpu.attention_backward(e, e, e, e, e, lse, idx)
    assert dq.shape == e.shape
    t = torch.zeros(1, 1, 64, 64, device="cuda")
    bad = torch.zeros(1, 1, 2, 3, device="cuda", dtype=torch.int32)    # width 3 > nb = 2
    with pytest.raises(gpu.MraError):
        gpu.attention_backward(t, t, t, t, t, torch.zeros(1, 1, 64, device="cuda"), bad)


@pytest.mark.parametrize("name", [n for n in inputs.WORKLOADS if inputs.WORKLOADS[n].n <= 4096])
def test_backward_workload_full_size(gpu, name):
    """Each workload up to 4096 tokens at its real shape (forward and backward
    of every head on the GPU); two sampled heads checked in full against the
    oracle."""
    w = inputs.WORKLOADS[name]
    _say("backward workload", name)
    q, k, v = inputs.make_qkv(w)
    g = np.random.Generator(np.random.PCG64(w.seed + 7)).standard_normal(q.shape)
    g = inputs.round_to_bf16(g) if w.dtype == "bf16" else g.astype(np.float32)
    heads = sorted({(0, 0), (w.B - 1, w.H - 1)})
    worst = _check(gpu, "mra2", q, k, v, g, w.budget, w.dtype, heads=heads)
    _record_grads("MRA-2", w, heads, worst)


def test_backward_long_sequence_full_head(gpu):
    """The 32768-token workload at its real shape (forward and backward of
    all 16 heads on the GPU): dQ, dK, dV and the log normalisers of one whole
    head against the oracle (Sec. 4.3 Alg. 2 differentiated through
    eq. actual_approx_mat_form with the selection held fixed), and finite
    gradients everywhere."""
    w = inputs.WORKLOADS["long-32768"]
    _say("backward workload", w.name)
    q, k, v = inputs.make_qkv(w)
    g = np.random.Generator(np.random.PCG64(w.seed + 7)).standard_normal(q.shape)
    g = inputs.round_to_bf16(g)
    tq, tk, tv, tg = dev(q, w.dtype), dev(k, w.dtype), dev(v, w.dtype), dev(g, w.dtype)
    out, idx, lse = _forward(gpu, "mra2", tq, tk, tv, w.budget)
    dq, dk, dv = gpu.attention_backward(tq, tk, tv, out, tg, lse, idx)
    torch.cuda.synchronize()
    for t in (dq, dk, dv):
        assert torch.isfinite(t).all()
    b, h = w.B - 1, w.H - 1
    gi = host(idx[b, h]).astype(np.int64)
    qh, kh, vh, gh = (a[b, h].astype(np.float64) for a in (q, k, v, g))
    Lref = O.mra_lse(qh, kh, 32, gi)
    lerr = float((np.abs(host(lse[b, h]) - Lref) / np.maximum(1.0, np.abs(Lref))).max())
    ref = O.mra_grads(qh, kh, vh, gh, 32, gi)
    mags = O.mra_grad_terms(qh, kh, vh, gh, 32, gi, absolute=True)
    worst = {"lse": lerr}
    for name, got, want, mag in zip(("dq", "dk", "dv"), (dq, dk, dv), ref, mags):
        gh_ = host(got[b, h])
        worst[name], worst[name + "_row"], worst[name + "_fro"] = \
            _rel(gh_, want), _rowerr(gh_, want, mag), _fro(gh_, want)
    _say("  long-32768", {k_: f"{e:.2e}" for k_, e in worst.items()})
    _record_grads("MRA-2", w, [(b, h)], worst)
    assert lerr <= LSE_TOL[w.dtype]
    for name in ("dq", "dk", "dv"):
        assert worst[name] <= GRAD_TOL[w.dtype], (name, worst)
        assert worst[name + "_row"] <= GRAD_ROW_TOL[w.dtype], (name, worst)
