"""Seeded input generators: determinism, shapes, rounding and distributions."""
import numpy as np
import pytest
import torch

from paper_2207_10284_amd import inputs


def test_round_to_bf16_matches_torch_from_float32():
    # torch's float32 -> bfloat16 conversion rounds to nearest even; on inputs
    # that are already float32 there is no double rounding, so both must agree.
    r = np.random.Generator(np.random.PCG64(0))
    x32 = (r.standard_normal(200000) * np.exp(r.uniform(-20, 20, 200000))).astype(np.float32)
    ours = inputs.round_to_bf16(x32.astype(np.float64))
    ref = torch.from_numpy(x32).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(ours, ref)


def test_round_to_bf16_ties_and_no_double_rounding():
    one = 1.0
    ulp = 2.0 ** -7                      # bf16 spacing just above 1
    assert inputs.round_to_bf16(np.array([one + ulp / 2]))[0] == one           # tie -> even
    assert inputs.round_to_bf16(np.array([one + 3 * ulp / 2]))[0] == one + 2 * ulp
    # slightly above the tie in float64, but rounds to the tie in float32:
    x = one + ulp / 2 + 2.0 ** -40
    assert inputs.round_to_bf16(np.array([x]))[0] == one + ulp


def test_bf16_bits_roundtrip():
    v = inputs.round_to_bf16(np.array([1.0, -2.5, 3.140625]))
    bits = inputs.bf16_bits(v)
    back = (bits.astype(np.uint32) << 16).view(np.float32)
    assert np.array_equal(back, v)
    with pytest.raises(ValueError):
        inputs.bf16_bits(np.array([1.0 + 2.0 ** -20], dtype=np.float32))


@pytest.mark.parametrize("name", list(inputs.WORKLOADS))
def test_shapes_dtypes_determinism(name):
    w = inputs.WORKLOADS[name]
    q, k, v = inputs.make_qkv(w, B=1, H=min(w.H, 2), n=min(w.n, 1024))
    q2, _, _ = inputs.make_qkv(w, B=1, H=min(w.H, 2), n=min(w.n, 1024))
    assert q.shape == (1, min(w.H, 2), min(w.n, 1024), w.d) and q.dtype == np.float32
    assert np.array_equal(q, q2)
    if w.dtype == "bf16":
        for a in (q, k, v):
            inputs.bf16_bits(a)
    assert not np.array_equal(q, k)


def test_ar1_statistics():
    w = inputs.WORKLOADS["base-4096"]
    q, k, v = inputs.make_qkv(w, B=2, H=2)
    x = q.astype(np.float64)
    var = x.var()
    assert abs(var - 1.0 / (1 - w.rho ** 2)) / (1.0 / (1 - w.rho ** 2)) < 0.1
    lag1 = (x[:, :, 1:] * x[:, :, :-1]).mean() / var
    assert abs(lag1 - w.rho) < 0.02
    assert abs(v.astype(np.float64).var() - 1.0) < 0.02


def test_hub_positions():
    w = inputs.WORKLOADS["small-4096"]
    meta = {}
    q, k, v = inputs.make_qkv(w, B=2, H=2, meta=meta)
    n_hub = round(0.05 * w.n)
    assert len(meta["hubs"]) == 2
    for b, (u, pos) in enumerate(meta["hubs"]):
        assert abs(np.linalg.norm(u) - 4.0) < 1e-12 and len(set(pos.tolist())) == n_hub
        uh = u / 4.0
        proj = k[b].astype(np.float64) @ uh            # [H, n]
        rest = np.setdiff1d(np.arange(w.n), pos)
        for h in range(2):                             # the shift is shared by both heads
            assert abs(proj[h, pos].mean() - 4.0) < 0.3
            assert abs(proj[h, rest].mean()) < 0.1
        assert abs((q[b].astype(np.float64) @ uh)[:, pos].mean()) < 0.3
