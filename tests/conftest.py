import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")


def pytest_sessionfinish(session, exitstatus):
    """With MRA_PARITY_LOG set, write the full-size parity results the GPU
    tests collected (tests/parity.py RECORDS) to that file as a table."""
    path = os.environ.get("MRA_PARITY_LOG")
    if not path:
        return
    from tests import parity
    if not parity.RECORDS:
        return
    lines = ["# Full-size parity against the float64 oracle", "",
             "Command (one MI355X): `MRA_PARITY_LOG=gpurun_out/parity.md python -u -m pytest tests -m gpu -x -q "
             "--timeout 400 --timeout-method thread`", "",
             "Every block-row of every head of each workload is checked (selection against the oracle's float64 "
             "scores, exact except near-ties within 1e-6 of the m-th score; output against the oracle evaluated "
             "under the GPU's selection). Row-normwise error = max over rows of ||Z_i - Zref_i||_inf / "
             "||Zref_i||_inf. Gradient rows: error over the magnitude of the terms summed into the row (see "
             "tests/test_gpu_backward.py).", "",
             "| variant | workload | dtype | heads | block-rows checked | max row-normwise rel. err | "
             "max abs err / max abs ref | rel. Frobenius err | bar | rows with tie swaps | note |",
             "|---|---|---|---|---|---|---|---|---|---|---|"]
    for r in parity.RECORDS:
        lines.append(f"| {r['variant']} | {r['workload']} | {r['dtype']} | {r['heads']} | {r['rows']} | "
                     f"{r['row_err']:.3e} | {r['global_err']:.3e} | {r['fro_err']:.3e} | {r['tol']:g} | "
                     f"{r['tie_rows']} | {r['note']} |")
    d = os.path.dirname(path)
    if d:
        os.makedirs(d, exist_ok=True)
    with open(path, "w") as f:
        f.write("\n".join(lines) + "\n")


@pytest.fixture(scope="session")
def gpu():
    """The HIP library bound to cuda:0. GPU tests fail (not skip) without a GPU,
    so a run on a box whose GPU is missing cannot pass silently."""
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU test run without a visible GPU")
    from paper_2207_10284_amd import ops
    ops.load()          # raises if the HIP library is not built
    return ops
