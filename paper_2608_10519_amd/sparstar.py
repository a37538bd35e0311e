"""Python binding of libsparstar (argument marshalling only).

Each function mirrors the C entry point of the same name in include/sparstar.h.
torch supplies device memory and the current HIP stream; every step of the
computation runs in the library's HIP kernels.  There is no fallback: if the
library cannot be loaded, every call raises.
"""
from __future__ import annotations

import ctypes
import os
from typing import Sequence

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libsparstar.so")

OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_WORKSPACE, ERR_HIP = 0, -1, -2, -3, -4
MAX_KEEP_RANGES = 8
FUSED_MAX_BLOCKS = 2304  # SPARSTAR_FUSED_MAX_BLOCKS
MAX_MASS_ROWS = 16
STATIC_SCRATCH_BYTES = 64 << 20  # SPARSTAR_STATIC_SCRATCH_BYTES

_lib = None


class SparstarError(RuntimeError):
    def __init__(self, fn: str, code: int, msg: str):
        super().__init__(f"{fn} failed with code {code}: {msg}")
        self.code = code


class Range(ctypes.Structure):
    _fields_ = [("begin", ctypes.c_int64), ("end", ctypes.c_int64)]


def load(path: str | None = None) -> ctypes.CDLL:
    """Load the HIP library (once).  Raises if it is not built."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise RuntimeError(f"libsparstar.so not found at {p}; build it with "
                           "`python -m paper_2608_10519_amd.build`")
    lib = ctypes.CDLL(p)
    c_i, c_i64, c_sz, c_p, c_f = ctypes.c_int, ctypes.c_int64, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_float
    c_dp, c_rp = ctypes.POINTER(ctypes.c_double), ctypes.POINTER(Range)
    lib.sparstar_score_workspace_bytes.argtypes = [c_i, c_i, c_i64, c_i64, c_i, c_i]
    lib.sparstar_score_workspace_bytes.restype = c_sz
    lib.sparstar_kv_stride.argtypes = [c_i, c_i64, c_i, c_dp, c_i, c_rp, c_i]
    lib.sparstar_kv_stride.restype = c_i64
    lib.sparstar_score_blocks.argtypes = [c_p, c_p, c_i, c_i, c_i64, c_i64, c_i, c_i, c_dp, c_i, c_rp, c_i,
                                          c_p, c_p, c_i, c_p, c_p, c_sz, c_p]
    lib.sparstar_score_blocks.restype = c_i
    lib.sparstar_score_blocks_fused.argtypes = [c_p, c_p, c_i, c_i, c_i64, c_i64, c_i, c_i, c_dp, c_i, c_rp, c_i,
                                                c_p, c_p, c_i, c_p, c_sz, c_p]
    lib.sparstar_score_blocks_fused.restype = c_i
    lib.sparstar_score_blocks_static.argtypes = [c_p, c_p, c_i, c_i, c_i64, c_i64, c_i, c_i, c_dp, c_i, c_rp, c_i,
                                                 c_p, c_p, c_i, c_p, c_p]
    lib.sparstar_score_blocks_static.restype = c_i
    lib.sparstar_attn_workspace_bytes.argtypes = [c_i, c_i, c_i64, c_i64, c_i, c_i]
    lib.sparstar_attn_workspace_bytes.restype = c_sz
    lib.sparstar_sparse_attn_fwd.argtypes = [c_p, c_p, c_p, c_i, c_i, c_i64, c_i64, c_i, c_i, c_p, c_p, c_i,
                                             c_f, c_p, c_p, c_p, c_sz, c_p]
    lib.sparstar_sparse_attn_fwd.restype = c_i
    lib.sparstar_dense_attn_fwd.argtypes = [c_p, c_p, c_p, c_i, c_i, c_i64, c_i64, c_i, c_i, c_f, c_p, c_p, c_p,
                                            c_sz, c_p]
    lib.sparstar_dense_attn_fwd.restype = c_i
    lib.sparstar_retained_mass.argtypes = [c_p, c_p, c_i64, c_p, c_p]
    lib.sparstar_retained_mass.restype = c_i
    lib.sparstar_token_topk_workspace_bytes.argtypes = [c_i, c_i, c_i64, c_i]
    lib.sparstar_token_topk_workspace_bytes.restype = c_sz
    lib.sparstar_token_topk_mass.argtypes = [c_p, c_p, c_i, c_i, c_i64, c_i64, c_i, ctypes.POINTER(ctypes.c_int64),
                                             c_i, c_p, c_p, c_f, c_p, c_p, c_sz, c_p]
    lib.sparstar_token_topk_mass.restype = c_i
    lib.sparstar_last_error.argtypes = []
    lib.sparstar_last_error.restype = ctypes.c_char_p
    lib.sparstar_clip_keep_ranges.argtypes = [c_i, Range, Range, c_rp, c_i]
    lib.sparstar_clip_keep_ranges.restype = c_i
    lib.sparstar_scale_densities.argtypes = [ctypes.POINTER(ctypes.c_int64), c_i, c_dp, c_i, c_dp]
    lib.sparstar_scale_densities.restype = c_i
    if path is None:
        _lib = lib
    return lib


def last_error() -> str:
    return load().sparstar_last_error().decode()


def _check(fn: str, rc: int) -> None:
    if rc != OK:
        raise SparstarError(fn, rc, last_error())


def _budget_array(budget) -> tuple[ctypes.Array, int]:
    vals = [float(budget)] if isinstance(budget, (int, float)) else [float(x) for x in budget]
    return (ctypes.c_double * len(vals))(*vals), len(vals)


def _keep_array(keep: Sequence[tuple[int, int]]):
    keep = list(keep)
    if not keep:
        return None, 0
    return (Range * len(keep))(*[Range(int(a), int(b)) for a, b in keep]), len(keep)


def _stream() -> int:
    return torch.cuda.current_stream().cuda_stream


def _bhld(t: torch.Tensor, name: str) -> tuple[int, int, int, int]:
    if t.dtype != torch.bfloat16 or not t.is_cuda or not t.is_contiguous() or t.dim() != 4:
        raise ValueError(f"{name} must be a contiguous 4-D bf16 tensor on the GPU [B, H, L, D]")
    return tuple(t.shape)


def sparstar_score_workspace_bytes(B: int, H: int, Lq: int, Lk: int, D: int, block_size: int) -> int:
    return int(load().sparstar_score_workspace_bytes(B, H, Lq, Lk, D, block_size))


def sparstar_attn_workspace_bytes(B: int, H: int, Lq: int, Lk: int, D: int, block_size: int) -> int:
    return int(load().sparstar_attn_workspace_bytes(B, H, Lq, Lk, D, block_size))


def _attn_workspace(workspace, split: bool, B, H, Lq, Lk, D, block_size, device):
    """(pointer, bytes) of the attention workspace: the caller's, a fresh one, or none."""
    if not split:
        return None, 0
    if workspace is None:
        n = sparstar_attn_workspace_bytes(B, H, Lq, Lk, D, block_size)
        if n == 0:
            return None, 0
        workspace = torch.empty(n, dtype=torch.uint8, device=device)
    return workspace.data_ptr(), workspace.numel() * workspace.element_size()


def sparstar_kv_stride(H: int, Lk: int, block_size: int, budget, keep=()) -> int:
    b, nb = _budget_array(budget)
    kr, nk = _keep_array(keep)
    r = int(load().sparstar_kv_stride(H, Lk, block_size, b, nb, kr, nk))
    if r < 0:
        raise SparstarError("sparstar_kv_stride", r, last_error())
    return r


# The paper's 720p schedule: densities of the four finest scales, in order of
# increasing token count (Section 5.2; supplement, sparsity schedule).
PAPER_720P_FINEST_DENSITIES = (0.625, 0.1875, 0.1875, 0.09375)


def sparstar_clip_keep_ranges(clip: int, text: tuple[int, int], ref: tuple[int, int]) -> list[tuple[int, int]]:
    """Forced token ranges of Eq. 3 for clip `clip` (text first)."""
    out = (Range * 2)()
    n = load().sparstar_clip_keep_ranges(int(clip), Range(*map(int, text)), Range(*map(int, ref)), out, 2)
    if n < 0:
        raise SparstarError("sparstar_clip_keep_ranges", n, last_error())
    return [(out[i].begin, out[i].end) for i in range(n)]


def sparstar_scale_densities(scale_lq: Sequence[int], finest_rho: Sequence[float]) -> list[float | None]:
    """rho of every scale of one clip group (None: the scale stays dense)."""
    n, m = len(scale_lq), len(finest_rho)
    lq = (ctypes.c_int64 * max(n, 1))(*map(int, scale_lq))
    rho = (ctypes.c_double * max(m, 1))(*map(float, finest_rho))
    out = (ctypes.c_double * max(n, 1))()
    _check("sparstar_scale_densities", load().sparstar_scale_densities(lq, n, rho, m, out))
    return [None if out[i] < 0 else out[i] for i in range(n)]


def sparstar_score_blocks(q: torch.Tensor, k: torch.Tensor, block_size: int, budget, keep=(), *,
                          kv_stride: int | None = None, scores: torch.Tensor | None = None,
                          workspace: torch.Tensor | None = None, out=None, fused: bool = False):
    """Selector: returns (kv_num_blocks [B,H,n_q] int32, kv_indices [B,H,n_q,kv_stride] int32).

    fused=True runs sparstar_score_blocks_fused (scores and selection in one
    kernel, S kept in LDS; no `scores` output)."""
    B, H, Lq, D = _bhld(q, "q")
    Bk, Hk, Lk, Dk = _bhld(k, "k")
    if (B, H, D) != (Bk, Hk, Dk):
        raise ValueError("q and k disagree on B, H or D")
    lib = load()
    bud, nb = _budget_array(budget)
    kr, nkeep = _keep_array(keep)
    if kv_stride is None:
        kv_stride = sparstar_kv_stride(H, Lk, block_size, budget, keep)
    n_q = -(-Lq // block_size)
    if out is None:
        num = torch.empty((B, H, n_q), dtype=torch.int32, device=q.device)
        idx = torch.empty((B, H, n_q, kv_stride), dtype=torch.int32, device=q.device)
    else:
        num, idx = out
    ws_bytes = sparstar_score_workspace_bytes(B, H, Lq, Lk, D, block_size)
    if workspace is None:
        workspace = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device=q.device)
    ws_n = workspace.numel() * workspace.element_size()
    if fused:
        if scores is not None:
            raise ValueError("the fused selector writes no scores")
        rc = lib.sparstar_score_blocks_fused(q.data_ptr(), k.data_ptr(), B, H, Lq, Lk, D, block_size, bud, nb, kr,
                                             nkeep, num.data_ptr(), idx.data_ptr(), kv_stride, workspace.data_ptr(),
                                             ws_n, _stream())
        _check("sparstar_score_blocks_fused", rc)
    else:
        rc = lib.sparstar_score_blocks(q.data_ptr(), k.data_ptr(), B, H, Lq, Lk, D, block_size, bud, nb, kr, nkeep,
                                       num.data_ptr(), idx.data_ptr(), kv_stride,
                                       scores.data_ptr() if scores is not None else None,
                                       workspace.data_ptr(), ws_n, _stream())
        _check("sparstar_score_blocks", rc)
    return num, idx


def sparstar_score_blocks_static(q: torch.Tensor, k: torch.Tensor, block_size: int, budget, keep=(), *,
                                 kv_stride: int | None = None, scores: torch.Tensor | None = None, out=None):
    """The selector with its scratch in the library's static per-GPU buffer
    (sparstar_score_blocks_static): the C call allocates nothing.  Pass `out`
    (and `scores` where S does not fit the scratch) to allocate nothing here
    either.  Returns (kv_num_blocks, kv_indices)."""
    B, H, Lq, D = _bhld(q, "q")
    Bk, Hk, Lk, Dk = _bhld(k, "k")
    if (B, H, D) != (Bk, Hk, Dk):
        raise ValueError("q and k disagree on B, H or D")
    bud, nb = _budget_array(budget)
    kr, nkeep = _keep_array(keep)
    if kv_stride is None:
        kv_stride = sparstar_kv_stride(H, Lk, block_size, budget, keep)
    n_q = -(-Lq // block_size)
    if out is None:
        num = torch.empty((B, H, n_q), dtype=torch.int32, device=q.device)
        idx = torch.empty((B, H, n_q, kv_stride), dtype=torch.int32, device=q.device)
    else:
        num, idx = out
    rc = load().sparstar_score_blocks_static(q.data_ptr(), k.data_ptr(), B, H, Lq, Lk, D, block_size, bud, nb, kr,
                                             nkeep, num.data_ptr(), idx.data_ptr(), kv_stride,
                                             scores.data_ptr() if scores is not None else None, _stream())
    _check("sparstar_score_blocks_static", rc)
    return num, idx


def sparstar_sparse_attn_fwd(q, k, v, kv_num_blocks, kv_indices, block_size: int, softmax_scale: float = 0.0, *,
                             out: torch.Tensor | None = None, lse: torch.Tensor | None = None,
                             return_lse: bool = True, split: bool = True, workspace: torch.Tensor | None = None):
    """Block-sparse forward: returns (O [B,H,Lq,D] bf16, lse [B,H,Lq] fp32 or None).

    split=True runs the key-range split (allocating its workspace unless one is
    given); split=False runs the single-pass kernel."""
    B, H, Lq, D = _bhld(q, "q")
    _, _, Lk, _ = _bhld(k, "k")
    _bhld(v, "v")
    if kv_indices.dtype != torch.int32 or kv_num_blocks.dtype != torch.int32:
        raise ValueError("block lists must be int32")
    if not kv_indices.is_contiguous() or not kv_num_blocks.is_contiguous():
        raise ValueError("block lists must be contiguous")
    o = torch.empty_like(q) if out is None else out
    if lse is None and return_lse:
        lse = torch.empty((B, H, Lq), dtype=torch.float32, device=q.device)
    wp, wn = _attn_workspace(workspace, split, B, H, Lq, Lk, D, block_size, q.device)
    rc = load().sparstar_sparse_attn_fwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), B, H, Lq, Lk, D, block_size,
                                         kv_num_blocks.data_ptr(), kv_indices.data_ptr(), kv_indices.shape[-1],
                                         float(softmax_scale), o.data_ptr(),
                                         lse.data_ptr() if lse is not None else None, wp, wn, _stream())
    _check("sparstar_sparse_attn_fwd", rc)
    return o, lse


def sparstar_dense_attn_fwd(q, k, v, block_size: int = 64, softmax_scale: float = 0.0, *,
                            out: torch.Tensor | None = None, lse: torch.Tensor | None = None,
                            return_lse: bool = True, split: bool = True, workspace: torch.Tensor | None = None):
    """Dense forward with the same tile engine: returns (O, lse)."""
    B, H, Lq, D = _bhld(q, "q")
    _, _, Lk, _ = _bhld(k, "k")
    _bhld(v, "v")
    o = torch.empty_like(q) if out is None else out
    if lse is None and return_lse:
        lse = torch.empty((B, H, Lq), dtype=torch.float32, device=q.device)
    wp, wn = _attn_workspace(workspace, split, B, H, Lq, Lk, D, block_size, q.device)
    rc = load().sparstar_dense_attn_fwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), B, H, Lq, Lk, D, block_size,
                                        float(softmax_scale), o.data_ptr(),
                                        lse.data_ptr() if lse is not None else None, wp, wn, _stream())
    _check("sparstar_dense_attn_fwd", rc)
    return o, lse


def sparstar_retained_mass(lse_sel: torch.Tensor, lse_all: torch.Tensor, *, out: torch.Tensor | None = None):
    """exp(lse_sel - lse_all) elementwise (0 where lse_sel is -inf): the share of
    each query's dense softmax mass its block selection keeps."""
    for t, name in ((lse_sel, "lse_sel"), (lse_all, "lse_all")):
        if t.dtype != torch.float32 or not t.is_cuda or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous fp32 tensor on the GPU")
    if lse_sel.shape != lse_all.shape:
        raise ValueError("lse_sel and lse_all differ in shape")
    mass = torch.empty_like(lse_sel) if out is None else out
    rc = load().sparstar_retained_mass(lse_sel.data_ptr(), lse_all.data_ptr(), lse_sel.numel(), mass.data_ptr(),
                                       _stream())
    _check("sparstar_retained_mass", rc)
    return mass


def sparstar_token_topk_workspace_bytes(B: int, H: int, Lk: int, n_rows: int) -> int:
    return int(load().sparstar_token_topk_workspace_bytes(B, H, Lk, n_rows))


def sparstar_token_topk_mass(q: torch.Tensor, k: torch.Tensor, rows: Sequence[int], n_tokens: torch.Tensor,
                             lse_all: torch.Tensor, softmax_scale: float = 0.0, *,
                             workspace: torch.Tensor | None = None):
    """Sum of the n_tokens[b,h,r] largest dense softmax weights of query rows[r]:
    the token-wise upper bound of the retained mass.  Returns [B, H, len(rows)] fp32."""
    B, H, Lq, D = _bhld(q, "q")
    _, _, Lk, _ = _bhld(k, "k")
    n = len(rows)
    if n_tokens.dtype != torch.int32 or not n_tokens.is_contiguous() or tuple(n_tokens.shape) != (B, H, n):
        raise ValueError("n_tokens must be a contiguous int32 tensor [B, H, len(rows)]")
    if lse_all.dtype != torch.float32 or not lse_all.is_contiguous() or tuple(lse_all.shape) != (B, H, Lq):
        raise ValueError("lse_all must be a contiguous fp32 tensor [B, H, Lq]")
    r = (ctypes.c_int64 * max(n, 1))(*[int(x) for x in rows])
    need = sparstar_token_topk_workspace_bytes(B, H, Lk, n)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=q.device)
    mass = torch.empty((B, H, n), dtype=torch.float32, device=q.device)
    rc = load().sparstar_token_topk_mass(q.data_ptr(), k.data_ptr(), B, H, Lq, Lk, D, r, n, n_tokens.data_ptr(),
                                         lse_all.data_ptr(), float(softmax_scale), mass.data_ptr(),
                                         workspace.data_ptr(), workspace.numel() * workspace.element_size(),
                                         _stream())
    _check("sparstar_token_topk_mass", rc)
    return mass
