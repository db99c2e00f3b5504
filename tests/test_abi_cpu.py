"""The C ABI without a GPU: the library loads, exports every function that
include/mra.h declares, and rejects invalid arguments on the host before any
HIP call (each call here either fails validation or is an empty problem, so
nothing is ever enqueued)."""
import ctypes
import os
import re

import pytest

from paper_2207_10284_amd import ops

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mra.h")

OK, INVALID, UNSUPPORTED, MISALIGNED, WORKSPACE, HIP, SCRATCH = range(7)
A = 1 << 20            # a fake, 16-byte aligned address: never dereferenced
MIS = A + 4            # misaligned


@pytest.fixture(scope="module")
def lib():
    return ops.load()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mra_[a-z_0-9]+)\s*\(", text)))


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert len(names) == 22, names
    for name in names:
        assert hasattr(lib, name), name
    assert set(names) == set(ops.SIGNATURES)


def test_exports_no_other_c_symbols():
    """Every unmangled function the library exports is an entry point of
    include/mra.h (helpers have internal linkage or live in a namespace)."""
    import shutil
    import subprocess
    if shutil.which("nm") is None:
        pytest.skip("nm not available")
    out = subprocess.run(["nm", "-D", "--defined-only", ops.LIB_PATH], capture_output=True, text=True,
                         check=True).stdout
    funcs = {line.split()[-1] for line in out.splitlines() if len(line.split()) == 3 and line.split()[1] == "T"}
    plain = {f for f in funcs if not f.startswith("_Z")}
    assert plain == set(declared_functions()), sorted(plain ^ set(declared_functions()))


def test_status_strings(lib):
    for code, name in ops.STATUS.items():
        assert lib.mra_status_str(code).decode().startswith(name)
    assert lib.mra_last_hip_error() == 0


def fwd(lib, q=A, k=A, v=A, out=A, idx=None, ws=A, wsb=1 << 40, B=1, H=1, n=64, d=64, block=32,
        budget=1, dtype=1, lse=None):
    return lib.mra_attention_forward(q, k, v, out, idx, lse, ws, wsb, B, H, n, d, block, budget, dtype, None)


def test_forward_validation(lib):
    assert fwd(lib, block=16) == UNSUPPORTED
    assert fwd(lib, block=0) == INVALID
    assert fwd(lib, d=48) == UNSUPPORTED
    assert fwd(lib, d=0) == INVALID
    assert fwd(lib, d=256) == UNSUPPORTED
    assert fwd(lib, n=48) == INVALID           # not a multiple of the block
    assert fwd(lib, n=65536 + 32) == UNSUPPORTED
    assert fwd(lib, B=-1) == INVALID
    assert fwd(lib, H=-3) == INVALID
    assert fwd(lib, budget=-1) == INVALID
    assert fwd(lib, budget=3) == INVALID       # nb = 2
    assert fwd(lib, dtype=7) == UNSUPPORTED
    assert fwd(lib, q=None) == INVALID
    assert fwd(lib, out=None) == INVALID
    assert fwd(lib, ws=None) == INVALID
    assert fwd(lib, v=MIS) == MISALIGNED
    assert fwd(lib, idx=MIS) == MISALIGNED
    assert fwd(lib, lse=MIS) == MISALIGNED
    need = lib.mra_forward_workspace_bytes(1, 1, 64, 64, 32, 1, 1)
    assert fwd(lib, wsb=need - 1) == WORKSPACE
    # empty problems succeed without touching any pointer
    assert fwd(lib, B=0, q=None, k=None, v=None, out=None, ws=None) == OK
    assert fwd(lib, n=0, budget=0, q=None, out=None, ws=None) == OK
    assert fwd(lib, n=0, budget=1) == INVALID  # nb = 0
    assert lib.mra_last_hip_error() == 0


def test_noalloc_forward_validation(lib):
    """The entry point without a workspace: every check of mra_attention_forward
    except the workspace's, then the static scratch's limit, all before any
    HIP call."""
    f = lambda q=A, k=A, v=A, out=A, idx=None, lse=None, B=1, H=1, n=64, d=64, block=32, budget=1, dtype=1: \
        lib.mra_attention_forward_noalloc(q, k, v, out, idx, lse, B, H, n, d, block, budget, dtype, None)
    assert f(block=16) == UNSUPPORTED
    assert f(d=48) == UNSUPPORTED
    assert f(n=48) == INVALID
    assert f(budget=3) == INVALID
    assert f(dtype=7) == UNSUPPORTED
    assert f(q=None) == INVALID
    assert f(out=MIS) == MISALIGNED
    assert f(idx=MIS) == MISALIGNED
    assert f(lse=MIS) == MISALIGNED
    assert f(B=0, q=None, k=None, v=None, out=None) == OK
    limit = 64 << 20
    # the largest benchmark workload fits; 128 heads of 32k tokens at d = 128 do not
    assert lib.mra_forward_workspace_bytes(1, 16, 32768, 128, 32, 32, 1) <= limit
    assert lib.mra_forward_workspace_bytes(1, 128, 32768, 128, 32, 32, 1) > limit
    assert f(B=1, H=128, n=32768, d=128, budget=32) == SCRATCH
    assert f(B=1, H=128, n=32768, d=128, budget=32, q=None) == INVALID   # argument checks come first
    assert lib.mra_last_hip_error() == 0


def sfwd(lib, q=A, k=A, v=A, out=A, idx=None, ws=A, wsb=1 << 40, B=1, H=1, n=64, d=64, block=32,
         budget=1, dtype=1, lse=None):
    return lib.mra_sparse_attention_forward(q, k, v, out, idx, lse, ws, wsb, B, H, n, d, block, budget,
                                            dtype, None)


def test_sparse_forward_validation(lib):
    """MRA-2-s: the forward's checks, and at least one selected block per row."""
    assert sfwd(lib, budget=0) == INVALID
    assert sfwd(lib, budget=-1) == INVALID
    assert sfwd(lib, budget=3) == INVALID      # nb = 2
    assert sfwd(lib, block=16) == UNSUPPORTED
    assert sfwd(lib, d=48) == UNSUPPORTED
    assert sfwd(lib, q=None) == INVALID
    assert sfwd(lib, k=MIS) == MISALIGNED
    assert sfwd(lib, lse=MIS) == MISALIGNED
    need = lib.mra_forward_workspace_bytes(1, 1, 64, 64, 32, 1, 1)
    assert sfwd(lib, wsb=need - 1) == WORKSPACE
    assert sfwd(lib, B=0, q=None, k=None, v=None, out=None, ws=None) == OK
    assert sfwd(lib, B=0, budget=0) == INVALID  # nb = 2: a block must be selected
    assert sfwd(lib, n=0, budget=0, q=None, out=None, ws=None) == OK
    assert lib.mra_last_hip_error() == 0


def test_workspace_bytes(lib):
    f = lib.mra_forward_workspace_bytes
    assert f(1, 1, 64, 48, 32, 1, 1) == 0
    assert f(1, 1, 64, 64, 32, 3, 1) == 0
    assert f(1, 1, 64, 64, 16, 1, 1) == 0
    assert f(1, 1, 64, 64, 32, 1, 9) == 0
    al = lambda x: (x + 255) // 256 * 256
    B, H, n, d, m = 8, 12, 4096, 64, 16
    bh, nb = B * H, n // 32
    for dd in (32, 64, 128):
        for dt, e in ((0, 4), (1, 2)):
            # packed K/V copy only where the tile pass cannot read raw rows (float32, d = 128)
            packed = al(2 * bh * n * dd * e) if dt == 0 and dd == 128 else 0
            want = 3 * al(bh * nb * dd * 4) + packed + al(bh * nb * m * 4) \
                + 2 * al(bh * nb * 4) + al(bh * nb * dd * 4)
            assert f(B, H, n, dd, 32, m, dt) == want, (dd, dt)


def test_global_workspace_bytes(lib):
    f = lib.mra_forward_global_workspace_bytes
    assert f(1, 1, 64, 48, 32, 1) == 0
    assert f(1, 1, 64, 64, 16, 1) == 0
    assert f(1, 1, 64, 64, 32, 9) == 0
    al = lambda x: (x + 255) // 256 * 256
    B, H, n, d = 8, 12, 4096, 64
    bh, nb = B * H, n // 32
    for dt in (0, 1):
        want = lib.mra_forward_workspace_bytes(B, H, n, d, 32, nb, dt) + al(bh * nb * nb * 4)
        assert f(B, H, n, d, 32, dt) == want


def test_global_selection_validation(lib):
    """Head-wide budget: 0 <= budget <= nb*nb (minus the nb diagonal priors),
    prior flag 0 or 1; the forward checks like mra_attention_forward."""
    sg = lambda scores=A, idx=A, B=1, H=1, n=128, budget=1, prior=0: \
        lib.mra_select_global(scores, idx, B, H, n, 32, budget, prior, None)
    assert sg(budget=-1) == INVALID
    assert sg(budget=17) == INVALID            # nb = 4
    assert sg(budget=13, prior=1) == INVALID   # 16 - 4 diagonal priors
    assert sg(prior=2) == INVALID
    assert sg(scores=None) == INVALID
    assert sg(idx=MIS) == MISALIGNED
    assert sg(n=48) == INVALID
    assert sg(B=0, scores=None, idx=None) == OK
    fg = lambda q=A, out=A, ws=A, wsb=1 << 40, n=128, d=64, budget=1, prior=0, dtype=1, lse=None: \
        lib.mra_attention_forward_global(q, A, A, out, None, lse, ws, wsb, 1, 1, n, d, 32, budget, prior, dtype,
                                         None)
    assert fg(budget=17) == INVALID
    assert fg(prior=-1) == INVALID
    assert fg(d=48) == UNSUPPORTED
    assert fg(q=None) == INVALID
    assert fg(ws=MIS) == MISALIGNED
    assert fg(lse=MIS) == MISALIGNED
    need = lib.mra_forward_global_workspace_bytes(1, 1, 128, 64, 32, 1)
    assert fg(wsb=need - 1) == WORKSPACE
    assert fg(n=0, budget=0, q=None, out=None, ws=None) == OK
    assert lib.mra_last_hip_error() == 0


def test_step_validation(lib):
    # pool: pairs must be given together, at least one pair
    p = lib.mra_pool
    assert p(A, None, None, None, None, None, 1, 1, 64, 64, 32, 1, None) == INVALID
    assert p(None, None, None, None, None, None, 1, 1, 64, 64, 32, 1, None) == INVALID
    assert p(A, None, None, MIS, None, None, 1, 1, 64, 64, 32, 1, None) == MISALIGNED
    assert p(A, A, A, A, A, A, 1, 1, 64, 64, 32, 5, None) == UNSUPPORTED
    assert p(A, A, None, A, None, None, 1, 1, 64, 64, 32, 1, None) == INVALID        # k without kp
    assert p(A, A, A, A, A, MIS, 1, 1, 64, 64, 32, 1, None) == MISALIGNED
    assert p(None, None, None, None, None, None, 0, 1, 64, 64, 32, 1, None) == INVALID
    # coarse scores
    assert lib.mra_coarse_scores(A, A, None, 1, 1, 64, 64, 32, None) == INVALID
    assert lib.mra_coarse_scores(A, A, A, 1, 1, 64, 100, 32, None) == UNSUPPORTED
    # select: budget range, pointers only needed for budget > 0
    assert lib.mra_select(A, A, 1, 1, 64, 32, 3, None) == INVALID
    assert lib.mra_select(None, None, 1, 1, 64, 32, 0, None) == OK
    assert lib.mra_select(A, None, 1, 1, 64, 32, 1, None) == INVALID
    # coarse term
    assert lib.mra_coarse_term(A, None, A, A, A, A, 1, 1, 64, 64, 32, 1, None) == INVALID
    assert lib.mra_coarse_term(A, A, A, A, A, MIS, 1, 1, 64, 64, 32, 1, None) == MISALIGNED
    # tile pass: coarse term all-or-nothing; sparse-only needs budget >= 1
    t = lambda q, k, v, idx, cm, cs, cv, out, B, H, n, d, blk, m, dt, lse=None: \
        lib.mra_block_sddmm_spmm(q, k, v, idx, cm, cs, cv, out, lse, B, H, n, d, blk, m, dt, None)
    assert t(A, A, A, A, A, None, A, A, 1, 1, 64, 64, 32, 1, 1) == INVALID
    assert t(A, A, A, None, None, None, None, A, 1, 1, 64, 64, 32, 0, 1) == INVALID
    assert t(A, A, A, A, A, A, A, A, 1, 1, 64, 64, 32, 3, 1) == INVALID
    assert t(A, A, A, A, A, A, A, MIS, 1, 1, 64, 64, 32, 1, 1) == MISALIGNED
    assert t(A, A, A, A, A, A, A, A, 1, 1, 64, 64, 32, 1, 1, lse=MIS) == MISALIGNED
    assert t(A, A, A, A, A, A, A, A, 1, 1, 64, 64, 32, 1, 2) == UNSUPPORTED
    assert t(A, A, None, A, A, A, A, A, 1, 1, 64, 64, 32, 1, 1) == INVALID   # no v
    assert t(A, None, A, A, A, A, A, A, 1, 1, 64, 64, 32, 1, 1) == INVALID   # no k
    assert t(A, MIS, A, A, A, A, A, A, 1, 1, 64, 64, 32, 1, 1) == MISALIGNED
    assert t(None, None, None, None, A, A, A, None, 0, 1, 64, 64, 32, 1, 1) == OK


def bwd(lib, q=A, k=A, v=A, out=A, dout=A, lse=A, idx=A, dq=A, dk=A, dv=A, ws=A, wsb=1 << 40,
        B=1, H=1, n=64, d=64, block=32, width=1, coarse=1, dtype=1):
    return lib.mra_attention_backward(q, k, v, out, dout, lse, idx, dq, dk, dv, ws, wsb,
                                      B, H, n, d, block, width, coarse, dtype, None)


def test_backward_validation(lib):
    assert bwd(lib, block=16) == UNSUPPORTED
    assert bwd(lib, d=48) == UNSUPPORTED
    assert bwd(lib, n=48) == INVALID
    assert bwd(lib, dtype=3) == UNSUPPORTED
    assert bwd(lib, width=-1) == INVALID
    assert bwd(lib, width=3) == INVALID       # nb = 2
    assert bwd(lib, coarse=2) == INVALID
    for name in ("q", "k", "v", "out", "dout", "lse", "dq", "dk", "dv", "ws"):
        assert bwd(lib, **{name: None}) == INVALID, name
        assert bwd(lib, **{name: MIS}) == MISALIGNED, name
    assert bwd(lib, idx=None) == INVALID      # width > 0 needs the selection
    assert bwd(lib, idx=MIS) == MISALIGNED
    need = lib.mra_backward_workspace_bytes(1, 1, 64, 64, 32, 1)
    assert bwd(lib, wsb=need - 1) == WORKSPACE
    assert bwd(lib, B=0, q=None, k=None, v=None, out=None, dout=None, lse=None, idx=None, dq=None,
               dk=None, dv=None, ws=None) == OK
    assert lib.mra_last_hip_error() == 0


def bwdp(lib, qp=A, kp=A, vp=A, ws=A, wsb=1 << 40, B=1, n=64, d=64, width=1, coarse=1, dtype=1, q=A):
    return lib.mra_attention_backward_pooled(q, A, A, A, A, A, A, qp, kp, vp, A, A, A, ws, wsb, B, 1, n, d, 32,
                                             width, coarse, dtype, None)


def test_backward_pooled_validation(lib):
    """The pooled-input backward takes the plain backward's checks plus its
    three block-mean pointers, required (and 16-byte aligned) for any
    non-empty problem, also with coarse = 0."""
    assert bwdp(lib, q=None) == INVALID
    assert bwdp(lib, d=48) == UNSUPPORTED
    assert bwdp(lib, coarse=2) == INVALID
    for name in ("qp", "kp", "vp"):
        assert bwdp(lib, **{name: None}) == INVALID, name
        assert bwdp(lib, **{name: MIS}) == MISALIGNED, name
        assert bwdp(lib, coarse=0, **{name: None}) == INVALID, name
    need = lib.mra_backward_workspace_bytes(1, 1, 64, 64, 32, 1)
    assert bwdp(lib, wsb=need - 1) == WORKSPACE
    assert bwdp(lib, B=0, q=None, qp=None, kp=None, vp=None, ws=None) == OK
    assert lib.mra_last_hip_error() == 0


def test_forward_pooled_rows(lib):
    """Host arithmetic only: Q~, K~, V~ lead the forward's workspace, each
    B*H*nb*d float32 rounded up to 256 bytes, whatever the budget or dtype;
    checked against the offsets the workspace sizes imply."""
    outs = [ctypes.c_void_p() for _ in range(3)]
    refs = [ctypes.byref(o) for o in outs]
    for B, H, n, d in ((1, 1, 64, 64), (2, 3, 96, 32), (1, 5, 4096, 128)):
        assert lib.mra_forward_pooled_rows(A, B, H, n, d, 32, *refs) == OK
        pooled = -(-B * H * (n // 32) * d * 4 // 256) * 256
        assert [o.value - A for o in outs] == [0, pooled, 2 * pooled]
        # the pooled rows fit every forward workspace of these sizes
        for budget in (0, n // 32):
            assert lib.mra_forward_workspace_bytes(B, H, n, d, 32, budget, 1) >= 3 * pooled
        assert lib.mra_forward_global_workspace_bytes(B, H, n, d, 32, 0) >= 3 * pooled
    assert lib.mra_forward_pooled_rows(None, 1, 1, 64, 64, 32, *refs) == INVALID
    assert lib.mra_forward_pooled_rows(MIS, 1, 1, 64, 64, 32, *refs) == MISALIGNED
    assert lib.mra_forward_pooled_rows(A, 1, 1, 64, 48, 32, *refs) == UNSUPPORTED
    assert lib.mra_forward_pooled_rows(A, 1, 1, 48, 64, 32, *refs) == INVALID
    assert lib.mra_forward_pooled_rows(A, 1, 1, 64, 64, 32, None, refs[1], refs[2]) == INVALID
    assert lib.mra_forward_pooled_rows(None, 0, 1, 64, 64, 32, *refs) == OK
    assert [o.value for o in outs] == [None, None, None]


def mfwd(lib, q=A, out=A, ws=A, wsb=1 << 40, n=256, d=64, cb=64, m1=1, m2=1, dtype=1, i1=None, i2=None, lse=None):
    return lib.mra_attention_forward_multilevel(q, A, A, out, i1, i2, lse, ws, wsb, 1, 1, n, d, 32, cb, m1, m2,
                                                dtype, None)


def test_multilevel_validation(lib):
    """R = {s0, 32, 1}: s0 a multiple of 32 above 32 dividing n; budgets
    0 <= m1 <= n/s0, 0 <= m2 <= m1 * s0/32."""
    assert mfwd(lib, cb=32) == UNSUPPORTED
    assert mfwd(lib, cb=48) == UNSUPPORTED
    assert mfwd(lib, cb=0) == UNSUPPORTED
    assert mfwd(lib, cb=96) == INVALID        # 256 % 96
    assert mfwd(lib, m1=5) == INVALID         # n/s0 = 4
    assert mfwd(lib, m1=-1) == INVALID
    assert mfwd(lib, m1=1, m2=3) == INVALID   # 1 * 64/32 = 2 candidates
    assert mfwd(lib, m1=0, m2=1) == INVALID
    assert mfwd(lib, d=48) == UNSUPPORTED
    assert mfwd(lib, q=None) == INVALID
    assert mfwd(lib, i1=MIS) == MISALIGNED
    assert mfwd(lib, i2=MIS) == MISALIGNED
    assert mfwd(lib, lse=MIS) == MISALIGNED
    need = lib.mra_forward_multilevel_workspace_bytes(1, 1, 256, 64, 32, 64, 1, 1, 1)
    assert need > 0
    assert mfwd(lib, wsb=need - 1) == WORKSPACE
    assert mfwd(lib, n=0, m1=0, m2=0, q=None, out=None, ws=None) == OK
    assert lib.mra_forward_multilevel_workspace_bytes(1, 1, 256, 64, 32, 96, 1, 1, 1) == 0
    al = lambda x: (x + 255) // 256 * 256
    B, H, n, d, s0, m1, m2 = 8, 12, 4096, 64, 128, 8, 16
    bh, nb, nb0 = B * H, n // 32, n // s0
    want = lib.mra_forward_workspace_bytes(B, H, n, d, 32, m2, 1) + 3 * al(bh * nb0 * d * 4) \
        + al(bh * nb0 * nb0 * 4) + al(bh * nb0 * m1 * 4) + al(bh * nb * nb * 4)
    assert lib.mra_forward_multilevel_workspace_bytes(B, H, n, d, 32, s0, m1, m2, 1) == want
    assert lib.mra_last_hip_error() == 0


def lfwd(lib, scales=(256, 64, 32), budgets=(2, 3, 4), levels=None, q=A, out=A, ws=A, wsb=1 << 40, n=1024,
         d=64, dtype=1, outs=None, lse=None):
    L = len(scales) if levels is None else levels
    sc = (ctypes.c_int * max(len(scales), 1))(*scales)
    bu = (ctypes.c_int * max(len(budgets), 1))(*budgets)
    po = None if outs is None else ctypes.cast((ctypes.c_void_p * len(outs))(*outs), ctypes.c_void_p)
    return lib.mra_attention_forward_levels(q, A, A, out, po, lse, ws, wsb, 1, 1, n, d, 32, L,
                                            ctypes.cast(sc, ctypes.c_void_p), ctypes.cast(bu, ctypes.c_void_p),
                                            dtype, None)


def lws(lib, scales, budgets, n=1024, d=64, B=1, H=1):
    sc = (ctypes.c_int * len(scales))(*scales)
    bu = (ctypes.c_int * len(budgets))(*budgets)
    return lib.mra_forward_levels_workspace_bytes(B, H, n, d, 32, len(scales), ctypes.cast(sc, ctypes.c_void_p),
                                                  ctypes.cast(bu, ctypes.c_void_p), 1)


def test_levels_validation(lib):
    """R = {s_0 > ... > s_{L-1} = 32, 1}: each scale a larger multiple of the
    next dividing n, the last 32, at most 8 levels; budgets within the
    candidates of the parent level."""
    assert lfwd(lib, scales=(256, 64, 48)) == UNSUPPORTED       # last scale not 32
    assert lfwd(lib, scales=(64, 256, 32)) == UNSUPPORTED       # not decreasing
    assert lfwd(lib, scales=(256, 96, 32)) == UNSUPPORTED       # 96 does not divide 256
    assert lfwd(lib, scales=(192, 96, 32), n=1024) == INVALID   # 1024 % 192
    assert lfwd(lib, levels=0) == INVALID
    assert lfwd(lib, scales=(8192, 4096, 2048, 1024, 512, 256, 128, 64, 32), budgets=(1,) * 9,
                n=8192) == UNSUPPORTED                           # nine levels
    assert lfwd(lib, budgets=(5, 3, 4)) == INVALID              # n/s0 = 4
    assert lfwd(lib, budgets=(2, 9, 4)) == INVALID              # 2 * 256/64 = 8 candidates
    assert lfwd(lib, budgets=(2, 3, 7)) == INVALID              # 3 * 64/32 = 6 candidates
    assert lfwd(lib, budgets=(2, -1, 0)) == INVALID
    assert lfwd(lib, d=48) == UNSUPPORTED
    assert lfwd(lib, q=None) == INVALID
    assert lfwd(lib, outs=[None, MIS, None]) == MISALIGNED
    assert lfwd(lib, lse=MIS) == MISALIGNED
    need = lws(lib, (256, 64, 32), (2, 3, 4))
    assert need > 0
    assert lfwd(lib, wsb=need - 1) == WORKSPACE
    assert lfwd(lib, n=0, budgets=(0, 0, 0), q=None, out=None, ws=None) == OK
    assert lws(lib, (256, 96, 32), (2, 3, 4)) == 0
    # one level is the two-level forward, two levels the three-resolution one
    assert lws(lib, (32,), (16,), n=4096, B=8, H=12) == lib.mra_forward_workspace_bytes(8, 12, 4096, 64, 32, 16, 1)
    assert lws(lib, (128, 32), (8, 16), n=4096, B=8, H=12) == \
        lib.mra_forward_multilevel_workspace_bytes(8, 12, 4096, 64, 32, 128, 8, 16, 1)
    al = lambda x: (x + 255) // 256 * 256
    B, H, n, d = 8, 12, 4096, 64
    bh, nb = B * H, n // 32
    want = lib.mra_forward_workspace_bytes(B, H, n, d, 32, 16, 1) + al(bh * nb * nb * 4)
    for s, m in ((512, 2), (128, 5)):
        nbl = n // s
        want += 3 * al(bh * nbl * d * 4) + al(bh * nbl * nbl * 4) + al(bh * nbl * m * 4)
    assert lws(lib, (512, 128, 32), (2, 5, 16), n=n, B=B, H=H) == want
    assert lib.mra_last_hip_error() == 0


def test_backward_workspace_bytes(lib):
    f = lib.mra_backward_workspace_bytes
    assert f(1, 1, 64, 48, 32, 1) == 0
    assert f(1, 1, 64, 64, 16, 1) == 0
    assert f(1, 1, 64, 64, 32, 9) == 0
    al = lambda x: (x + 255) // 256 * 256
    B, H, n, d = 8, 12, 4096, 64
    bh, nb = B * H, n // 32
    for dt, e in ((0, 4), (1, 2)):
        raw = dt == 1                                 # bf16 reads raw tiles
        copies = 0 if raw else 7
        bias = al(bh * n * 16) if raw else 0          # per query, the column pass's bias operand
        want = 7 * al(bh * nb * d * 4) + copies * al(bh * n * d * e) + al(bh * nb * 64 * 4) + bias \
            + al(bh * nb * (nb // 32) * 4) + 2 * al(bh * nb * nb * 4)
        assert f(B, H, n, d, 32, dt) == want
    # bf16 with d = 128 reads raw tiles too; float32 keeps its rearranged copies
    want = 7 * al(bh * nb * 128 * 4) + al(bh * nb * 64 * 4) + al(bh * n * 16) \
        + al(bh * nb * (nb // 32) * 4) + 2 * al(bh * nb * nb * 4)
    assert f(B, H, n, 128, 32, 1) == want
    want = 7 * al(bh * nb * 128 * 4) + 7 * al(bh * n * 128 * 4) + al(bh * nb * 64 * 4) \
        + al(bh * nb * (nb // 32) * 4) + 2 * al(bh * nb * nb * 4)
    assert f(B, H, n, 128, 32, 0) == want


def test_binding_fails_loudly_without_library(tmp_path, monkeypatch):
    monkeypatch.setattr(ops, "_lib", None)
    with pytest.raises(RuntimeError, match="not built"):
        ops.load(str(tmp_path / "missing.so"))
