"""Helpers shared by the GPU parity tests: upload, error metrics and the
tie-aware selection check. Holds no arithmetic of the method."""
import numpy as np
import torch

from oracle import mra_oracle as O

TOL = {"f32": 1e-5, "bf16": 2e-2}          # max row-normwise relative error
TIE_BAND = 1e-6                            # relative band around the m-th score


def dev(a, dtype="f32"):
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()
    return t.to(torch.bfloat16) if dtype == "bf16" else t


def host(t):
    return t.detach().float().cpu().numpy().astype(np.float64)


def row_rel_err(Z, Zref):
    """max over rows of ||Z_i - Zref_i||_inf / ||Zref_i||_inf (rows = last axis)."""
    num = np.abs(Z - Zref).max(axis=-1)
    den = np.maximum(np.abs(Zref).max(axis=-1), 1e-30)
    return float((num / den).max()) if num.size else 0.0


def check_selection(gpu_idx, S_ref, m, band=TIE_BAND):
    """GPU selection for rows of S_ref ([rows, nb], float64). Equal to the
    oracle's, except that rows may differ in elements whose reference score is
    within `band` (relative to the row's scale) of the m-th largest score.
    Also checks every GPU row is strictly ascending, in range, of length m.
    Returns the number of rows that differ."""
    gpu_idx = np.asarray(gpu_idx)
    ref = O.select_blocks(S_ref, m)
    nb = S_ref.shape[1]
    differ = 0
    for x in range(S_ref.shape[0]):
        g = gpu_idx[x]
        assert len(g) == m
        if m:
            assert (np.diff(g) > 0).all() and g[0] >= 0 and g[-1] < nb, g
        if np.array_equal(g, ref[x]):
            continue
        differ += 1
        srt = np.sort(S_ref[x])[::-1]
        tau = srt[m - 1]
        fin = S_ref[x][np.isfinite(S_ref[x])]       # -inf marks blocks outside a candidate set
        scale = max(abs(tau), np.abs(fin).max())
        for y in set(g.tolist()) ^ set(ref[x].tolist()):
            assert abs(S_ref[x, y] - tau) <= band * scale, (x, y, S_ref[x, y], tau)
    return differ


def check_selection_global(gpu_idx, S_ref, budget, prior_diagonal, band=TIE_BAND):
    """GPU head-wide selection ([nb, nb] rows padded with -1) for one head with
    float64 scores S_ref: rows strictly ascending and padded; priors present;
    equal to the oracle's set except blocks whose score lies within `band`
    (relative to the head's scale) of the budget-th largest non-prior score.
    Returns the number of blocks that differ."""
    gpu_idx = np.asarray(gpu_idx)
    nb = S_ref.shape[0]
    got = set()
    for x in range(nb):
        row = gpu_idx[x]
        k = int((row >= 0).sum())
        assert (row[k:] == -1).all() and (row[:k] >= 0).all() and (row[:k] < nb).all(), row
        assert (np.diff(row[:k]) > 0).all(), row
        got |= {x * nb + int(y) for y in row[:k]}
    ref_idx = O.select_global(S_ref, budget, prior_diagonal)
    want = {x * nb + int(y) for x in range(nb) for y in ref_idx[x] if y >= 0}
    if prior_diagonal:
        assert {x * nb + x for x in range(nb)} <= got
    assert len(got) == len(want)
    diff = got ^ want
    if diff:
        free = np.array([S_ref.ravel()[f] for f in range(nb * nb) if not (prior_diagonal and f // nb == f % nb)])
        tau = np.sort(free)[::-1][budget - 1]
        scale = max(abs(tau), np.abs(S_ref).max())
        for f in diff:
            assert abs(S_ref.ravel()[f] - tau) <= band * scale, (f, S_ref.ravel()[f], tau)
    return len(diff)


def err_stats(Z, Zref):
    """Error measures of an output against the oracle's (rows = last axis):
    the max row-normwise relative error (the bar), the largest elementwise
    error over the largest reference magnitude, and the relative Frobenius
    error."""
    Z = np.asarray(Z, dtype=np.float64)
    Zref = np.asarray(Zref, dtype=np.float64)
    diff = np.abs(Z - Zref)
    fro = float(np.sqrt((diff ** 2).sum()) / max(np.sqrt((Zref ** 2).sum()), 1e-300)) if Z.size else 0.0
    glob = float(diff.max() / max(np.abs(Zref).max(), 1e-300)) if Z.size else 0.0
    return {"row": row_rel_err(Z, Zref), "global": glob, "fro": fro}


# Parity results of the full-size tests, one dict per (variant, workload);
# conftest.py writes them as a table at the end of the session when the
# environment variable MRA_PARITY_LOG names a file.
RECORDS = []


def record(variant, workload, dtype, heads, rows, stats, tol, tie_rows, note=""):
    RECORDS.append({"variant": variant, "workload": workload, "dtype": dtype, "heads": heads, "rows": rows,
                    "row_err": stats["row"], "global_err": stats["global"], "fro_err": stats["fro"],
                    "tol": tol, "tie_rows": tie_rows, "note": note})
