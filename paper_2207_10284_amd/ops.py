"""Thin Python binding of libmra (C ABI in include/mra.h).

Argument marshalling only: every function checks tensor placement, dtype and
shape, allocates outputs with torch (device memory is plumbing here), and
calls the library on the current torch stream. All arithmetic runs in the HIP
kernels. There is no fallback: if the library is not built, ``load`` raises.

Shapes: q, k, v are [B, H, n, d] tensors on a ROCm device, float32 or
bfloat16, contiguous; n is a multiple of 32 and d is 32, 64 or 128.
"""
from __future__ import annotations

import ctypes
import os

import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libmra.so")
BLOCK = 32

MRA_F32, MRA_BF16 = 0, 1
STATUS = {0: "MRA_OK", 1: "MRA_ERR_INVALID_ARG", 2: "MRA_ERR_UNSUPPORTED",
          3: "MRA_ERR_MISALIGNED", 4: "MRA_ERR_WORKSPACE", 5: "MRA_ERR_HIP", 6: "MRA_ERR_SCRATCH"}

# name -> (restype, argtypes); mirrors include/mra.h
_P, _I, _Z = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
SIGNATURES = {
    "mra_pool": (_I, [_P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _P]),
    "mra_coarse_scores": (_I, [_P, _P, _P, _I, _I, _I, _I, _I, _P]),
    "mra_select": (_I, [_P, _P, _I, _I, _I, _I, _I, _P]),
    "mra_coarse_term": (_I, [_P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _P]),
    "mra_block_sddmm_spmm": (_I, [_P, _P, _P, _P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _I, _P]),
    "mra_forward_workspace_bytes": (_Z, [_I, _I, _I, _I, _I, _I, _I]),
    "mra_attention_forward": (_I, [_P, _P, _P, _P, _P, _P, _P, _Z, _I, _I, _I, _I, _I, _I, _I, _P]),
    "mra_sparse_attention_forward": (_I, [_P, _P, _P, _P, _P, _P, _P, _Z, _I, _I, _I, _I, _I, _I, _I, _P]),
    "mra_attention_forward_noalloc": (_I, [_P, _P, _P, _P, _P, _P, _I, _I, _I, _I, _I, _I, _I, _P]),
    "mra_select_global": (_I, [_P, _P, _I, _I, _I, _I, _I, _I, _P]),
    "mra_forward_global_workspace_bytes": (_Z, [_I, _I, _I, _I, _I, _I]),
    "mra_attention_forward_global": (_I, [_P, _P, _P, _P, _P, _P, _P, _Z, _I, _I, _I, _I, _I, _I, _I, _I, _P]),
    "mra_forward_multilevel_workspace_bytes": (_Z, [_I, _I, _I, _I, _I, _I, _I, _I, _I]),
    "mra_attention_forward_multilevel": (_I, [_P, _P, _P, _P, _P, _P, _P, _P, _Z, _I, _I, _I, _I, _I, _I,
                                              _I, _I, _I, _P]),
    "mra_forward_levels_workspace_bytes": (_Z, [_I, _I, _I, _I, _I, _I, _P, _P, _I]),
    "mra_attention_forward_levels": (_I, [_P, _P, _P, _P, _P, _P, _P, _Z, _I, _I, _I, _I, _I, _I,
                                          _P, _P, _I, _P]),
    "mra_backward_workspace_bytes": (_Z, [_I, _I, _I, _I, _I, _I]),
    "mra_attention_backward": (_I, [_P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _Z,
                                    _I, _I, _I, _I, _I, _I, _I, _I, _P]),
    "mra_attention_backward_pooled": (_I, [_P] * 14 + [_Z] + [_I] * 8 + [_P]),
    "mra_forward_pooled_rows": (_I, [_P, _I, _I, _I, _I, _I, _P, _P, _P]),
    "mra_status_str": (ctypes.c_char_p, [_I]),
    "mra_last_hip_error": (_I, []),
}

_lib = None


class MraError(RuntimeError):
    def __init__(self, fn: str, status: int, lib):
        msg = lib.mra_status_str(status).decode()
        if status == 5:
            msg += f" (hipError_t {lib.mra_last_hip_error()})"
        super().__init__(f"{fn}: {msg}")
        self.status = status


def load(path: str = LIB_PATH):
    """Open libmra.so once and declare its signatures. Raises if it is missing."""
    global _lib
    if _lib is None:
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is not built; run `python -m paper_2207_10284_amd.build` "
                               "(hipcc, gfx950) first")
        lib = ctypes.CDLL(path)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(lib, name)
            fn.restype, fn.argtypes = res, args
        _lib = lib
    return _lib


def _call(name: str, *args):
    lib = load()
    st = getattr(lib, name)(*args)
    if st != 0:
        raise MraError(name, st, lib)


def _ptr(t):
    return None if t is None else t.data_ptr()


def _stream(device):
    return torch.cuda.current_stream(device).cuda_stream


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return MRA_F32
    if t.dtype == torch.bfloat16:
        return MRA_BF16
    raise TypeError(f"unsupported dtype {t.dtype}; expected float32 or bfloat16")


def _check_qkv(*ts):
    ref = next(t for t in ts if t is not None)
    for t in ts:
        if t is None:
            continue
        if not t.is_cuda:
            raise ValueError("tensors must be on a ROCm device")
        if t.dim() != 4 or t.shape != ref.shape or t.dtype != ref.dtype or t.device != ref.device:
            raise ValueError("q, k, v must share shape [B, H, n, d], dtype and device")
        if not t.is_contiguous():
            raise ValueError("q, k, v must be contiguous")
    return ref


def _check_f32(t, shape, name):
    if t.dtype != torch.float32 or tuple(t.shape) != tuple(shape) or not t.is_contiguous() or not t.is_cuda:
        raise ValueError(f"{name} must be a contiguous float32 device tensor of shape {tuple(shape)}")


def pool(q, k=None, v=None):
    """Block means (Sec. 4.1/4.3): returns (qp, kp, vp), float32 [B, H, n/32, d]
    (None for a tensor not given)."""
    ref = _check_qkv(q, k, v)
    B, H, n, d = ref.shape
    outs = [None if t is None else torch.empty(B, H, n // BLOCK, d, device=ref.device, dtype=torch.float32)
            for t in (q, k, v)]
    _call("mra_pool", _ptr(q), _ptr(k), _ptr(v), *(_ptr(o) for o in outs),
          B, H, n, d, BLOCK, _dtype_code(ref), _stream(ref.device))
    return tuple(outs)


def coarse_scores(qp, kp):
    """Coarse logits S~ = Q~ K~^T / sqrt(d): float32 [B, H, nb, nb]."""
    B, H, nb, d = qp.shape
    _check_f32(qp, (B, H, nb, d), "qp")
    _check_f32(kp, (B, H, nb, d), "kp")
    S = torch.empty(B, H, nb, nb, device=qp.device, dtype=torch.float32)
    _call("mra_coarse_scores", _ptr(qp), _ptr(kp), _ptr(S), B, H, nb * BLOCK, d, BLOCK, _stream(qp.device))
    return S


def select(scores, budget: int):
    """Per block-row top-`budget` column blocks, ascending: int32 [B, H, nb, budget]."""
    B, H, nb, _ = scores.shape
    _check_f32(scores, (B, H, nb, nb), "scores")
    idx = torch.empty(B, H, nb, budget, device=scores.device, dtype=torch.int32)
    _call("mra_select", _ptr(scores), _ptr(idx), B, H, nb * BLOCK, BLOCK, budget, _stream(scores.device))
    return idx


def select_global(scores, budget: int, prior_diagonal: bool = False):
    """Head-wide selection of Alg. 1: the `budget` best blocks of each head
    (plus the diagonal blocks with ``prior_diagonal``); int32 [B, H, nb, nb],
    each row ascending, padded with -1."""
    B, H, nb, _ = scores.shape
    _check_f32(scores, (B, H, nb, nb), "scores")
    idx = torch.empty(B, H, nb, nb, device=scores.device, dtype=torch.int32)
    _call("mra_select_global", _ptr(scores), _ptr(idx), B, H, nb * BLOCK, BLOCK, budget,
          int(bool(prior_diagonal)), _stream(scores.device))
    return idx


def _check_idx(idx, B, H, nb, budget, device):
    if idx.dtype != torch.int32 or tuple(idx.shape) != (B, H, nb, budget) or not idx.is_contiguous() \
            or idx.device != device:
        raise ValueError(f"idx must be a contiguous int32 tensor of shape {(B, H, nb, budget)}")


def coarse_term(scores, idx, vp):
    """Low-resolution term of the unselected blocks: (cmax, csum, cvec)."""
    B, H, nb, d = vp.shape
    budget = idx.shape[-1]
    _check_f32(scores, (B, H, nb, nb), "scores")
    _check_f32(vp, (B, H, nb, d), "vp")
    _check_idx(idx, B, H, nb, budget, vp.device)
    cmax = torch.empty(B, H, nb, device=vp.device, dtype=torch.float32)
    csum = torch.empty_like(cmax)
    cvec = torch.empty(B, H, nb, d, device=vp.device, dtype=torch.float32)
    _call("mra_coarse_term", _ptr(scores), _ptr(idx), _ptr(vp), _ptr(cmax), _ptr(csum), _ptr(cvec),
          B, H, nb * BLOCK, d, BLOCK, budget, _stream(vp.device))
    return cmax, csum, cvec


def block_sddmm_spmm(q, k, v, idx, cmax=None, csum=None, cvec=None, out=None, lse_out=None):
    """Selected tiles exp(c Q_x K_y^T) V_y, merged with the coarse term (if
    given) and normalised: the output Z, [B, H, n, d] in the input dtype.
    ``lse_out`` (float32 [B, H, n]) receives each query's log normaliser."""
    ref = _check_qkv(q, k, v)
    B, H, n, d = ref.shape
    nb = n // BLOCK
    budget = idx.shape[-1]
    _check_idx(idx, B, H, nb, budget, ref.device)
    if cmax is not None:
        _check_f32(cmax, (B, H, nb), "cmax")
        _check_f32(csum, (B, H, nb), "csum")
        _check_f32(cvec, (B, H, nb, d), "cvec")
    if out is None:
        out = torch.empty_like(ref)
    if lse_out is not None:
        _check_f32(lse_out, (B, H, n), "lse_out")
    _call("mra_block_sddmm_spmm", _ptr(q), _ptr(k), _ptr(v), _ptr(idx), _ptr(cmax), _ptr(csum),
          _ptr(cvec), _ptr(out), _ptr(lse_out), B, H, n, d, BLOCK, budget, _dtype_code(ref), _stream(ref.device))
    return out


def forward_workspace_bytes(B: int, H: int, n: int, d: int, budget: int, dtype=torch.bfloat16) -> int:
    code = MRA_BF16 if dtype == torch.bfloat16 else MRA_F32
    return int(load().mra_forward_workspace_bytes(B, H, n, d, BLOCK, budget, code))


def attention_forward(q, k, v, budget: int, out=None, idx_out=None, workspace=None, lse_out=None):
    """The whole MRA-2 forward pass. Returns the output Z ([B, H, n, d], input
    dtype); the selection is written to ``idx_out`` and each query's log
    normaliser (float32 [B, H, n]) to ``lse_out`` when given."""
    return _forward("mra_attention_forward", q, k, v, budget, out, idx_out, workspace, lse_out)


def attention_forward_noalloc(q, k, v, budget: int, out=None, idx_out=None, lse_out=None):
    """``attention_forward`` through the entry point that allocates nothing:
    its workspace is the library's static per-GPU scratch (calls on one GPU
    must not overlap). ``out`` is allocated here only when not given."""
    ref = _check_qkv(q, k, v)
    B, H, n, d = ref.shape
    nb = n // BLOCK
    if out is None:
        out = torch.empty_like(ref)
    if idx_out is not None:
        _check_idx(idx_out, B, H, nb, budget, ref.device)
    if lse_out is not None:
        _check_f32(lse_out, (B, H, n), "lse_out")
    _call("mra_attention_forward_noalloc", _ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(idx_out), _ptr(lse_out),
          B, H, n, d, BLOCK, budget, _dtype_code(ref), _stream(ref.device))
    return out


def sparse_attention_forward(q, k, v, budget: int, out=None, idx_out=None, workspace=None, lse_out=None):
    """The sparse-only variant MRA-2-s (Sec. 5): softmax over the selected
    blocks only, no low-resolution term; budget >= 1. Same arguments and
    result as ``attention_forward``."""
    return _forward("mra_sparse_attention_forward", q, k, v, budget, out, idx_out, workspace, lse_out)


def _forward(entry, q, k, v, budget, out, idx_out, workspace, lse_out):
    ref = _check_qkv(q, k, v)
    B, H, n, d = ref.shape
    nb = n // BLOCK
    if out is None:
        out = torch.empty_like(ref)
    if idx_out is not None:
        _check_idx(idx_out, B, H, nb, budget, ref.device)
    if lse_out is not None:
        _check_f32(lse_out, (B, H, n), "lse_out")
    need = forward_workspace_bytes(B, H, n, d, budget, ref.dtype)
    if workspace is None:
        workspace = torch.empty(max(need, 1), device=ref.device, dtype=torch.uint8)
    _call(entry, _ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(idx_out), _ptr(lse_out),
          _ptr(workspace), workspace.numel() * workspace.element_size(),
          B, H, n, d, BLOCK, budget, _dtype_code(ref), _stream(ref.device))
    return out


def forward_global_workspace_bytes(B: int, H: int, n: int, d: int, dtype=torch.bfloat16) -> int:
    code = MRA_BF16 if dtype == torch.bfloat16 else MRA_F32
    return int(load().mra_forward_global_workspace_bytes(B, H, n, d, BLOCK, code))


def attention_forward_global(q, k, v, budget: int, prior_diagonal: bool = False, out=None, idx_out=None,
                             workspace=None, lse_out=None):
    """MRA-2 with the head-wide budget of Alg. 1 (``budget`` blocks per head,
    plus the diagonal with ``prior_diagonal``). Returns Z; the selection
    (int32 [B, H, nb, nb], rows padded with -1) goes to ``idx_out`` and the
    log normalisers to ``lse_out`` when given."""
    ref = _check_qkv(q, k, v)
    B, H, n, d = ref.shape
    nb = n // BLOCK
    if out is None:
        out = torch.empty_like(ref)
    if idx_out is not None:
        _check_idx(idx_out, B, H, nb, nb, ref.device)
    if lse_out is not None:
        _check_f32(lse_out, (B, H, n), "lse_out")
    need = forward_global_workspace_bytes(B, H, n, d, ref.dtype)
    if workspace is None:
        workspace = torch.empty(max(need, 1), device=ref.device, dtype=torch.uint8)
    _call("mra_attention_forward_global", _ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(idx_out), _ptr(lse_out),
          _ptr(workspace), workspace.numel() * workspace.element_size(),
          B, H, n, d, BLOCK, budget, int(bool(prior_diagonal)), _dtype_code(ref), _stream(ref.device))
    return out


def forward_multilevel_workspace_bytes(B: int, H: int, n: int, d: int, coarse_block: int, budget1: int,
                                       budget2: int, dtype=torch.bfloat16) -> int:
    code = MRA_BF16 if dtype == torch.bfloat16 else MRA_F32
    return int(load().mra_forward_multilevel_workspace_bytes(B, H, n, d, BLOCK, coarse_block, budget1, budget2,
                                                             code))


def attention_forward_multilevel(q, k, v, coarse_block: int, budget1: int, budget2: int, out=None,
                                 idx1_out=None, idx2_out=None, lse_out=None, workspace=None):
    """Three resolutions R = {coarse_block, 32, 1} (Alg. 1 with two refinement
    levels, per-row budgets). Returns Z; the selections go to ``idx1_out``
    (int32 [B, H, n/coarse_block, budget1]) and ``idx2_out`` (int32
    [B, H, n/32, budget2]) when given."""
    ref = _check_qkv(q, k, v)
    B, H, n, d = ref.shape
    if out is None:
        out = torch.empty_like(ref)
    if idx1_out is not None:
        _check_idx(idx1_out, B, H, n // coarse_block if coarse_block else 0, budget1, ref.device)
    if idx2_out is not None:
        _check_idx(idx2_out, B, H, n // BLOCK, budget2, ref.device)
    if lse_out is not None:
        _check_f32(lse_out, (B, H, n), "lse_out")
    need = forward_multilevel_workspace_bytes(B, H, n, d, coarse_block, budget1, budget2, ref.dtype)
    if workspace is None:
        workspace = torch.empty(max(need, 1), device=ref.device, dtype=torch.uint8)
    _call("mra_attention_forward_multilevel", _ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(idx1_out),
          _ptr(idx2_out), _ptr(lse_out), _ptr(workspace), workspace.numel() * workspace.element_size(),
          B, H, n, d, BLOCK, coarse_block, budget1, budget2, _dtype_code(ref), _stream(ref.device))
    return out


def _int_array(vals):
    vals = [int(x) for x in vals]
    return (ctypes.c_int * max(len(vals), 1))(*vals)


def forward_levels_workspace_bytes(B: int, H: int, n: int, d: int, scales, budgets, dtype=torch.bfloat16) -> int:
    code = MRA_BF16 if dtype == torch.bfloat16 else MRA_F32
    sc, bu = _int_array(scales), _int_array(budgets)
    return int(load().mra_forward_levels_workspace_bytes(B, H, n, d, BLOCK, len(scales),
                                                         ctypes.cast(sc, _P), ctypes.cast(bu, _P), code))


def attention_forward_levels(q, k, v, scales, budgets, out=None, idx_outs=None, lse_out=None,
                             workspace=None):
    """Any number of resolutions R = {scales[0] > ... > scales[-1] = 32, 1}
    (Alg. 1 refined level by level, a per-row budget at every level). Returns
    Z; level l's selection goes to ``idx_outs[l]`` (int32
    [B, H, n/scales[l], budgets[l]]) when that entry is given."""
    ref = _check_qkv(q, k, v)
    B, H, n, d = ref.shape
    L = len(scales)
    if len(budgets) != L or L < 1:
        raise ValueError("one budget per scale")
    if out is None:
        out = torch.empty_like(ref)
    outs = list(idx_outs) if idx_outs is not None else [None] * L
    if len(outs) != L:
        raise ValueError("one selection output (or None) per scale")
    for l, t in enumerate(outs):
        if t is not None:
            _check_idx(t, B, H, n // int(scales[l]) if int(scales[l]) > 0 else 0, int(budgets[l]), ref.device)
    if lse_out is not None:
        _check_f32(lse_out, (B, H, n), "lse_out")
    need = forward_levels_workspace_bytes(B, H, n, d, scales, budgets, ref.dtype)
    if workspace is None:
        workspace = torch.empty(max(need, 1), device=ref.device, dtype=torch.uint8)
    sc, bu = _int_array(scales), _int_array(budgets)
    ptrs = (ctypes.c_void_p * L)(*[_ptr(t) for t in outs])
    _call("mra_attention_forward_levels", _ptr(q), _ptr(k), _ptr(v), _ptr(out), ctypes.cast(ptrs, _P),
          _ptr(lse_out), _ptr(workspace), workspace.numel() * workspace.element_size(), B, H, n, d, BLOCK,
          L, ctypes.cast(sc, _P), ctypes.cast(bu, _P), _dtype_code(ref), _stream(ref.device))
    return out


def backward_workspace_bytes(B: int, H: int, n: int, d: int, dtype=torch.bfloat16) -> int:
    code = MRA_BF16 if dtype == torch.bfloat16 else MRA_F32
    return int(load().mra_backward_workspace_bytes(B, H, n, d, BLOCK, code))


def forward_pooled_rows(workspace, B: int, H: int, n: int, d: int):
    """The block means (Q~, K~, V~: float32 [B, H, nb, d] each) that
    ``attention_forward`` or ``attention_forward_global`` left in
    ``workspace`` (a uint8 device tensor) for these sizes, as views of it (no
    copy); they change when the workspace is used again."""
    if workspace.dtype != torch.uint8 or not workspace.is_contiguous():
        raise ValueError("workspace must be a contiguous uint8 tensor")
    nb = n // BLOCK
    if B * H * nb * d == 0:
        return tuple(torch.empty(B, H, nb, d, dtype=torch.float32, device=workspace.device) for _ in range(3))
    ptrs = [ctypes.c_void_p() for _ in range(3)]
    _call("mra_forward_pooled_rows", _ptr(workspace), B, H, n, d, BLOCK, *(ctypes.byref(p) for p in ptrs))
    size = B * H * nb * d * 4
    views = []
    for p in ptrs:
        off = (p.value or 0) - workspace.data_ptr()
        if p.value is None or off < 0 or off + size > workspace.numel():
            raise ValueError("workspace too small for the pooled rows of these sizes")
        views.append(workspace[off:off + size].view(torch.float32).view(B, H, nb, d))
    return tuple(views)


def attention_backward(q, k, v, out, dout, lse, idx, coarse: bool = True, dq=None, dk=None, dv=None,
                       workspace=None, pooled=None):
    """Gradients (dq, dk, dv) through one forward (``coarse=True``: MRA-2,
    per-row or head-wide budget; ``False``: MRA-2-s) with its selection
    ``idx`` (int32 [B, H, nb, width]) held fixed; ``out`` and ``lse`` are the
    forward's output and log normalisers, ``dout`` the gradient of the output.
    ``pooled``: the block means of q, k, v (float32 [B, H, nb, d] each, e.g.
    from ``forward_pooled_rows``), so that the backward does not compute them
    again; the gradients are the same bits either way."""
    ref = _check_qkv(q, k, v, out, dout)
    B, H, n, d = ref.shape
    nb = n // BLOCK
    width = idx.shape[-1]
    _check_idx(idx, B, H, nb, width, ref.device)
    _check_f32(lse, (B, H, n), "lse")
    dq = torch.empty_like(ref) if dq is None else dq
    dk = torch.empty_like(ref) if dk is None else dk
    dv = torch.empty_like(ref) if dv is None else dv
    _check_qkv(ref, dq, dk, dv)
    need = backward_workspace_bytes(B, H, n, d, ref.dtype)
    if workspace is None:
        workspace = torch.empty(max(need, 1), device=ref.device, dtype=torch.uint8)
    head = (_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(dout), _ptr(lse), _ptr(idx))
    tail = (_ptr(dq), _ptr(dk), _ptr(dv), _ptr(workspace), workspace.numel() * workspace.element_size(),
            B, H, n, d, BLOCK, width, int(bool(coarse)), _dtype_code(ref), _stream(ref.device))
    if pooled is None:
        _call("mra_attention_backward", *head, *tail)
    else:
        for name, t in zip(("qp", "kp", "vp"), pooled):
            _check_f32(t, (B, H, nb, d), name)
            if t.device != ref.device:
                raise ValueError(f"{name} must be on {ref.device}")
        _call("mra_attention_backward_pooled", *head, *(_ptr(t) for t in pooled), *tail)
    return dq, dk, dv


class MraAttention(torch.autograd.Function):
    """Z = MRA-2 attention of (q, k, v) as a differentiable op: the forward
    keeps its selection and log normalisers, the backward hands them to
    ``attention_backward`` (selection held fixed). ``variant`` is "mra2"
    (per-row budget), "mra2s" (sparse only) or "global" (head-wide budget,
    with ``prior_diagonal``)."""

    @staticmethod
    def forward(ctx, q, k, v, budget: int, variant: str = "mra2", prior_diagonal: bool = False):
        ref = _check_qkv(q, k, v)
        B, H, n, d = ref.shape
        nb = n // BLOCK
        lse = torch.empty(B, H, n, device=ref.device, dtype=torch.float32)
        pooled = ()
        if variant == "global":
            idx = torch.empty(B, H, nb, nb, device=ref.device, dtype=torch.int32)
            ws = torch.empty(max(forward_global_workspace_bytes(B, H, n, d, ref.dtype), 1), device=ref.device,
                             dtype=torch.uint8)
            out = attention_forward_global(q, k, v, budget, prior_diagonal, idx_out=idx, workspace=ws, lse_out=lse)
            pooled = forward_pooled_rows(ws, B, H, n, d)
        elif variant == "mra2":
            idx = torch.empty(B, H, nb, budget, device=ref.device, dtype=torch.int32)
            ws = torch.empty(max(forward_workspace_bytes(B, H, n, d, budget, ref.dtype), 1), device=ref.device,
                             dtype=torch.uint8)
            out = attention_forward(q, k, v, budget, idx_out=idx, workspace=ws, lse_out=lse)
            pooled = forward_pooled_rows(ws, B, H, n, d)
        elif variant == "mra2s":
            idx = torch.empty(B, H, nb, budget, device=ref.device, dtype=torch.int32)
            out = sparse_attention_forward(q, k, v, budget, idx_out=idx, lse_out=lse)
        else:
            raise ValueError(f"unknown variant {variant!r}")
        # the forward's block means (views of its workspace) go to the backward
        ctx.save_for_backward(q, k, v, out, lse, idx, *pooled)
        ctx.coarse = variant != "mra2s"
        return out

    @staticmethod
    def backward(ctx, dout):
        q, k, v, out, lse, idx, *pooled = ctx.saved_tensors
        dq, dk, dv = attention_backward(q, k, v, out, dout.contiguous(), lse, idx, coarse=ctx.coarse,
                                        pooled=tuple(pooled) if pooled else None)
        return dq, dk, dv, None, None, None


def mra_attention(q, k, v, budget: int, variant: str = "mra2", prior_diagonal: bool = False):
    """Differentiable MRA-2 attention (see ``MraAttention``)."""
    return MraAttention.apply(q, k, v, budget, variant, prior_diagonal)
