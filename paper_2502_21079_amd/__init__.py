"""Python binding of libadaspa, the MI355X (gfx950) AdaSpa attention hot path.

Argument marshalling only: every step runs in the HIP kernels of
``libadaspa.so``.  PyTorch provides device memory and the current stream.
The three calls mirror the C ABI in ``include/adaspa.h``:

* :func:`dense_attn_lse`     dense attention + LSE (Sec. 2.2; Algorithm 1 pass 1)
* :func:`block_search`       block masses from a given LSE (Algorithm 1 pass 2 /
                             Algorithm 2) and per-head block selection
                             (Sec. 4.1 optimal indices, Sec. 4.3 text sink and
                             row-wise uniform selection)
* :func:`block_sparse_attn`  blockified sparse attention (Sec. 4.1)
* :func:`fused_online_search`  Algorithm 1 in one launch: dense attention +
                             LSE and the masses of the same rows, then the
                             selection (bitwise what the first two give)

There is no CPU fallback: if the library is missing, every call raises.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional, Sequence

import torch

__all__ = ["dense_attn_lse", "dense_attn_workspace", "block_search", "block_sparse_attn",
           "block_sparse_attn_workspace", "block_sparse_attn_noalloc", "SearchResult",
           "library_path", "load_library", "AdaspaError", "EXPORTED_SYMBOLS",
           "block_search_workspace", "block_search_capacity", "fused_online_search",
           "single_pass_online_search", "single_pass_online_search_workspace",
           "single_pass_online_search_min_workspace"]

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_NAME = "libadaspa.so"

EXPORTED_SYMBOLS = ("adaspa_status_string", "adaspa_dense_attn_workspace", "adaspa_dense_attn_lse",
                    "adaspa_block_search_workspace", "adaspa_block_search_capacity",
                    "adaspa_block_search", "adaspa_block_sparse_attn_workspace",
                    "adaspa_block_sparse_attn", "adaspa_block_sparse_attn_noalloc",
                    "adaspa_fused_online_search", "adaspa_single_pass_online_search_workspace",
                    "adaspa_single_pass_online_search_min_workspace", "adaspa_single_pass_online_search")

SELECT_TOPK = 0
SELECT_COVERAGE = 1
SELECT_HIERARCHICAL = 2
F_TEXT_SINK = 1
F_SCORES_GIVEN = 2


class AdaspaError(RuntimeError):
    pass


class _Problem(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("heads", ctypes.c_int32),
                ("seqlen", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("block", ctypes.c_int32), ("text_start", ctypes.c_int32),
                ("text_len", ctypes.c_int32), ("softmax_scale", ctypes.c_float)]


class _Select(ctypes.Structure):
    _fields_ = [("mode", ctypes.c_int32), ("flags", ctypes.c_int32),
                ("head_param_bp", ctypes.POINTER(ctypes.c_int32)),
                ("base_sparsity_bp", ctypes.c_int32), ("recall_threshold_bp", ctypes.c_int32)]


_lib = None


def library_path() -> str:
    return os.environ.get("ADASPA_LIB", os.path.join(_HERE, _LIB_NAME))


def load_library():
    """Load libadaspa.so (once).  Raises if it is missing: there is no fallback."""
    global _lib
    if _lib is not None:
        return _lib
    path = library_path()
    if not os.path.exists(path):
        raise AdaspaError(f"{path} not found; build it with "
                          f"`python -m paper_2502_21079_amd.build`")
    lib = ctypes.CDLL(path)
    P, S = ctypes.POINTER(_Problem), ctypes.POINTER(_Select)
    vp, i32p, f32p = ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p
    lib.adaspa_status_string.restype = ctypes.c_char_p
    lib.adaspa_status_string.argtypes = [ctypes.c_int]
    lib.adaspa_dense_attn_workspace.restype = ctypes.c_size_t
    lib.adaspa_dense_attn_workspace.argtypes = [P]
    lib.adaspa_dense_attn_lse.restype = ctypes.c_int
    lib.adaspa_dense_attn_lse.argtypes = [P, vp, vp, vp, vp, f32p, vp, ctypes.c_size_t, vp]
    lib.adaspa_block_search_workspace.restype = ctypes.c_size_t
    lib.adaspa_block_search_workspace.argtypes = [P, S]
    lib.adaspa_block_search_capacity.restype = ctypes.c_int64
    lib.adaspa_block_search_capacity.argtypes = [P, S]
    lib.adaspa_block_search.restype = ctypes.c_int
    lib.adaspa_block_search.argtypes = [P, vp, vp, f32p, S, f32p, i32p, i32p, ctypes.c_int64,
                                        i32p, f32p, vp, ctypes.c_size_t, vp]
    lib.adaspa_fused_online_search.restype = ctypes.c_int
    lib.adaspa_fused_online_search.argtypes = [P, vp, vp, vp, vp, f32p, S, f32p, i32p, i32p,
                                               ctypes.c_int64, i32p, f32p, vp, ctypes.c_size_t, vp]
    lib.adaspa_single_pass_online_search_workspace.restype = ctypes.c_size_t
    lib.adaspa_single_pass_online_search_workspace.argtypes = [P, S]
    lib.adaspa_single_pass_online_search_min_workspace.restype = ctypes.c_size_t
    lib.adaspa_single_pass_online_search_min_workspace.argtypes = [P, S]
    lib.adaspa_single_pass_online_search.restype = ctypes.c_int
    lib.adaspa_single_pass_online_search.argtypes = [P, vp, vp, vp, vp, f32p, S, f32p, i32p, i32p,
                                                     ctypes.c_int64, i32p, f32p, vp, ctypes.c_size_t, vp]
    lib.adaspa_block_sparse_attn_workspace.restype = ctypes.c_size_t
    lib.adaspa_block_sparse_attn_workspace.argtypes = [P]
    lib.adaspa_block_sparse_attn.restype = ctypes.c_int
    lib.adaspa_block_sparse_attn.argtypes = [P, vp, vp, vp, i32p, i32p, ctypes.c_int64, vp,
                                             f32p, vp, ctypes.c_size_t, vp]
    lib.adaspa_block_sparse_attn_noalloc.restype = ctypes.c_int
    lib.adaspa_block_sparse_attn_noalloc.argtypes = [P, vp, vp, vp, i32p, i32p, ctypes.c_int64,
                                                     vp, f32p, vp]
    _lib = lib
    return lib


def _check(status: int):
    if status != 0:
        msg = load_library().adaspa_status_string(status).decode()
        raise AdaspaError(f"libadaspa status {status}: {msg}")


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(device) -> ctypes.c_void_p:
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _problem(q: torch.Tensor, block: int, text_start: int, text_len: int,
             scale: Optional[float]) -> _Problem:
    B, H, L, D = q.shape
    return _Problem(B, H, L, D, block, text_start, text_len,
                    0.0 if scale is None else float(scale))


def _check_qkv(*ts):
    ref = ts[0]
    for t in ts:
        if t is None:
            continue
        if t.dtype != torch.bfloat16 or t.device.type != "cuda" or not t.is_contiguous():
            raise AdaspaError("q, k, v must be contiguous bf16 CUDA tensors [B, H, L, D]")
        if t.shape != ref.shape:
            raise AdaspaError(f"shape mismatch {tuple(t.shape)} vs {tuple(ref.shape)}")


def _check_outputs(q, out, lse):
    """Caller-provided outputs must have the shapes the kernels write: the
    library sees only pointers, so a smaller buffer would be written past its
    end on the device."""
    B, H, L, D = q.shape
    if out is not None and (out.dtype != torch.bfloat16 or tuple(out.shape) != (B, H, L, D)
                            or not out.is_contiguous() or out.device != q.device):
        raise AdaspaError(f"out must be a contiguous bf16 [B, H, L, D] = {(B, H, L, D)} tensor on q's device")
    if lse is not None and (lse.dtype != torch.float32 or tuple(lse.shape) != (B, H, L)
                            or not lse.is_contiguous() or lse.device != q.device):
        raise AdaspaError(f"lse must be a contiguous fp32 [B, H, L] = {(B, H, L)} tensor on q's device")


def _workspace_bytes(workspace, dev) -> int:
    """Bytes of a caller's workspace tensor (any dtype), which must be a
    contiguous tensor on the inputs' device: the library sees only its
    pointer and size."""
    if workspace.device != dev or not workspace.is_contiguous():
        raise AdaspaError("workspace must be a contiguous tensor on q's device")
    return workspace.numel() * workspace.element_size()


def _select(mode: str, head_param_bp: Optional[Sequence[int]], text_sink: bool,
            scores_given: bool, base_sparsity_bp: int = 8000, recall_threshold_bp: int = 8000,
            heads: Optional[int] = None):
    modes = {"topk": SELECT_TOPK, "coverage": SELECT_COVERAGE, "hierarchical": SELECT_HIERARCHICAL}
    if mode not in modes:
        raise AdaspaError(f"unknown selection mode {mode!r}")
    m = modes[mode]
    params = list(head_param_bp) if head_param_bp is not None else []
    # The library reads head_param_bp[0 .. H-1] in the per-head modes: a shorter
    # list would be read past its end.
    if m != SELECT_HIERARCHICAL and heads is not None and len(params) != heads:
        raise AdaspaError(f"head_param_bp needs one entry per head ({heads}), got {len(params)}")
    arr = (ctypes.c_int32 * max(1, len(params)))(*[int(x) for x in params])
    ptr = ctypes.cast(arr, ctypes.POINTER(ctypes.c_int32)) if params else None
    flags = (F_TEXT_SINK if text_sink else 0) | (F_SCORES_GIVEN if scores_given else 0)
    return _Select(m, flags, ptr, int(base_sparsity_bp), int(recall_threshold_bp)), arr


def dense_attn_lse(q, k, v, *, scale: Optional[float] = None, out=None, lse=None,
                   want_lse: bool = True, workspace=None, balance: bool = True):
    """Dense attention and per-row natural-log LSE.  Returns (out, lse).

    With ``balance`` (the default) the XCDs share the work through per-XCD
    work queues whose counters live in ``workspace`` (uint8 CUDA tensor of at
    least ``dense_attn_workspace(q.shape)`` bytes; allocated here when not
    given); ``balance=False`` splits the work statically.  The results are
    the same either way."""
    _check_qkv(q, k, v)
    _check_outputs(q, out, lse)
    lib = load_library()
    B, H, L, D = q.shape
    if out is None:
        out = torch.empty_like(q)
    if lse is None and want_lse:
        lse = torch.empty(B, H, L, dtype=torch.float32, device=q.device)
    prob = _problem(q, 128, 0, 0, scale)
    ws_bytes = 0
    if balance:
        ws_bytes = int(lib.adaspa_dense_attn_workspace(ctypes.byref(prob)))
        if workspace is None:
            workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=q.device)
        ws_bytes = _workspace_bytes(workspace, q.device)
    else:
        workspace = None
    _check(lib.adaspa_dense_attn_lse(ctypes.byref(prob), _ptr(q), _ptr(k), _ptr(v), _ptr(out),
                                     _ptr(lse), _ptr(workspace), ctypes.c_size_t(ws_bytes),
                                     _stream(q.device)))
    return out, lse


def dense_attn_workspace(shape, scale: Optional[float] = None) -> int:
    """Bytes of the work-queue workspace of :func:`dense_attn_lse`."""
    B, H, L, D = shape
    prob = _Problem(B, H, L, D, 128, 0, 0, 0.0 if scale is None else float(scale))
    return int(load_library().adaspa_dense_attn_workspace(ctypes.byref(prob)))


@dataclass
class SearchResult:
    block_mass: torch.Tensor      # fp32 [B, H, NB, NB]
    row_ptr: torch.Tensor         # int32 [B*H*NB + 1]
    col_idx: torch.Tensor         # int32 [capacity]; valid prefix row_ptr[-1]
    head_k: torch.Tensor          # int32 [B, H]
    head_recall: torch.Tensor     # fp32 [B, H]

    def nnz(self) -> int:
        return int(self.row_ptr[-1].item())


def _problem_shape(B, H, L, D, block, text_start, text_len, scale):
    return _Problem(B, H, L, D, block, text_start, text_len, 0.0 if scale is None else float(scale))


def block_search_workspace(shape, block, text_start, text_len, mode, head_param_bp,
                           text_sink=True) -> int:
    B, H, L, D = shape
    prob = _problem_shape(B, H, L, D, block, text_start, text_len, None)
    sel, _keep = _select(mode, head_param_bp, text_sink, False, heads=H)
    return int(load_library().adaspa_block_search_workspace(ctypes.byref(prob), ctypes.byref(sel)))


def block_search_capacity(shape, block, text_start, text_len, mode, head_param_bp,
                          text_sink=True) -> int:
    B, H, L, D = shape
    prob = _problem_shape(B, H, L, D, block, text_start, text_len, None)
    sel, _keep = _select(mode, head_param_bp, text_sink, False, heads=H)
    return int(load_library().adaspa_block_search_capacity(ctypes.byref(prob), ctypes.byref(sel)))


def block_search(q, k, lse, *, block: int, text_start: int, text_len: int,
                 mode: str, head_param_bp: Optional[Sequence[int]] = None, text_sink: bool = True,
                 scale: Optional[float] = None, scores: Optional[torch.Tensor] = None,
                 shape=None, workspace: Optional[torch.Tensor] = None,
                 base_sparsity_bp: int = 8000, recall_threshold_bp: int = 8000,
                 result: Optional["SearchResult"] = None) -> SearchResult:
    """Block masses W_sum_attn from ``lse`` (fresh or cached) and the per-head
    selection.  ``mode`` is "topk" or "coverage" (per-head ``head_param_bp``)
    or "hierarchical" (``base_sparsity_bp``, ``recall_threshold_bp``, Sec. 4.2).
    With ``scores`` given (fp32 [B, H, NB, NB]) the mass pass is skipped and
    those masses are selected from (then q, k, lse may be None and ``shape`` =
    (B, H, L, D) is required).  ``result`` (an earlier SearchResult of the same
    problem and selection) is filled in place instead of new outputs."""
    lib = load_library()
    given = scores is not None
    if given:
        B, H, L, D = shape if shape is not None else q.shape
        dev = scores.device
    else:
        _check_qkv(q, k)
        B, H, L, D = q.shape
        dev = q.device
        if lse.dtype != torch.float32 or not lse.is_contiguous() or lse.shape != (B, H, L):
            raise AdaspaError("lse must be contiguous fp32 [B, H, L]")
    nb = (L + block - 1) // block
    prob = _problem_shape(B, H, L, D, block, text_start, text_len, scale)
    sel, _keep = _select(mode, head_param_bp, text_sink, given, base_sparsity_bp,
                         recall_threshold_bp, heads=H)
    cap = lib.adaspa_block_search_capacity(ctypes.byref(prob), ctypes.byref(sel))
    wsb = lib.adaspa_block_search_workspace(ctypes.byref(prob), ctypes.byref(sel))
    if cap < 0 or wsb == 0:
        _check(lib.adaspa_block_search(ctypes.byref(prob), None, None, None, ctypes.byref(sel),
                                       None, None, None, 0, None, None, None, 0, None))
        raise AdaspaError("invalid block_search arguments")
    res = _search_outputs(B, H, nb, cap, dev, result, scores)
    if workspace is None or _workspace_bytes(workspace, dev) < wsb:
        workspace = torch.empty(int(wsb), dtype=torch.uint8, device=dev)
    _check(lib.adaspa_block_search(ctypes.byref(prob), _ptr(q), _ptr(k), _ptr(lse),
                                   ctypes.byref(sel), _ptr(res.block_mass), _ptr(res.row_ptr),
                                   _ptr(res.col_idx), int(res.col_idx.numel()), _ptr(res.head_k),
                                   _ptr(res.head_recall), _ptr(workspace), _workspace_bytes(workspace, dev),
                                   _stream(dev)))
    return res


def _search_outputs(B, H, nb, cap, dev, result, scores=None) -> SearchResult:
    """The outputs of a search: ``result`` checked against the problem, or new
    tensors (with ``scores`` as the masses when they are given)."""
    if result is not None:
        ok = (result.block_mass.shape == (B, H, nb, nb) and result.row_ptr.numel() == B * H * nb + 1
              and result.col_idx.numel() >= cap and result.head_k.shape == (B, H)
              and result.block_mass.device == dev and scores is None)
        if not ok:
            raise AdaspaError("result does not fit this search (shape, capacity or device)")
        return result
    if scores is not None:
        if scores.dtype != torch.float32 or scores.shape != (B, H, nb, nb) or not scores.is_contiguous():
            raise AdaspaError("scores must be contiguous fp32 [B, H, NB, NB]")
        mass = scores
    else:
        mass = torch.empty(B, H, nb, nb, dtype=torch.float32, device=dev)
    return SearchResult(mass, torch.empty(B * H * nb + 1, dtype=torch.int32, device=dev),
                        torch.empty(max(int(cap), 1), dtype=torch.int32, device=dev),
                        torch.empty(B, H, dtype=torch.int32, device=dev),
                        torch.empty(B, H, dtype=torch.float32, device=dev))


def fused_online_search(q, k, v, *, block: int, text_start: int, text_len: int, mode: str,
                        head_param_bp: Optional[Sequence[int]] = None, text_sink: bool = True,
                        scale: Optional[float] = None, out=None, lse=None, want_lse: bool = True,
                        workspace: Optional[torch.Tensor] = None, base_sparsity_bp: int = 8000,
                        recall_threshold_bp: int = 8000,
                        result: Optional["SearchResult"] = None):
    """Algorithm 1 (fused online search) in one kernel launch, then the
    selection: returns (out, lse, SearchResult), bit for bit what
    :func:`dense_attn_lse` followed by :func:`block_search` with that LSE
    return.  Arguments as in those two calls; ``lse`` may be skipped
    (``want_lse=False``) and the masses still use the fresh LSE."""
    _check_qkv(q, k, v)
    lib = load_library()
    B, H, L, D = q.shape
    dev = q.device
    nb = (L + block - 1) // block
    prob = _problem_shape(B, H, L, D, block, text_start, text_len, scale)
    sel, _keep = _select(mode, head_param_bp, text_sink, False, base_sparsity_bp,
                         recall_threshold_bp, heads=H)
    cap = lib.adaspa_block_search_capacity(ctypes.byref(prob), ctypes.byref(sel))
    wsb = lib.adaspa_block_search_workspace(ctypes.byref(prob), ctypes.byref(sel))
    if cap < 0 or wsb == 0:
        _check(lib.adaspa_fused_online_search(ctypes.byref(prob), None, None, None, None, None,
                                              ctypes.byref(sel), None, None, None, 0, None, None,
                                              None, 0, None))
        raise AdaspaError("invalid fused_online_search arguments")
    _check_outputs(q, out, lse)
    if out is None:
        out = torch.empty_like(q)
    if lse is None and want_lse:
        lse = torch.empty(B, H, L, dtype=torch.float32, device=dev)
    res = _search_outputs(B, H, nb, cap, dev, result)
    if workspace is None or _workspace_bytes(workspace, dev) < wsb:
        workspace = torch.empty(int(wsb), dtype=torch.uint8, device=dev)
    _check(lib.adaspa_fused_online_search(ctypes.byref(prob), _ptr(q), _ptr(k), _ptr(v), _ptr(out),
                                          _ptr(lse), ctypes.byref(sel), _ptr(res.block_mass),
                                          _ptr(res.row_ptr), _ptr(res.col_idx),
                                          int(res.col_idx.numel()), _ptr(res.head_k),
                                          _ptr(res.head_recall), _ptr(workspace),
                                          _workspace_bytes(workspace, dev), _stream(dev)))
    return out, lse, res


def single_pass_online_search_workspace(shape, block, text_start, text_len, mode, head_param_bp=None,
                                        text_sink=True, base_sparsity_bp: int = 8000,
                                        recall_threshold_bp: int = 8000) -> int:
    """Bytes of the workspace of :func:`single_pass_online_search`: the
    search's scratch plus B*H*NB*L floats of per-row block masses."""
    B, H, L, D = shape
    prob = _problem_shape(B, H, L, D, block, text_start, text_len, None)
    sel, _keep = _select(mode, head_param_bp, text_sink, False, base_sparsity_bp, recall_threshold_bp,
                         heads=H)
    return int(load_library().adaspa_single_pass_online_search_workspace(ctypes.byref(prob),
                                                                         ctypes.byref(sel)))


def single_pass_online_search_min_workspace(shape, block, text_start, text_len, mode, head_param_bp=None,
                                            text_sink=True, base_sparsity_bp: int = 8000,
                                            recall_threshold_bp: int = 8000) -> int:
    """The least workspace :func:`single_pass_online_search` accepts (one
    (batch, head) pair's per-row block masses); with less than the full size
    the call runs the (batch, head) pairs in groups, with the same results."""
    B, H, L, D = shape
    prob = _problem_shape(B, H, L, D, block, text_start, text_len, None)
    sel, _keep = _select(mode, head_param_bp, text_sink, False, base_sparsity_bp, recall_threshold_bp,
                         heads=H)
    return int(load_library().adaspa_single_pass_online_search_min_workspace(ctypes.byref(prob),
                                                                             ctypes.byref(sel)))


def single_pass_online_search(q, k, v, *, block: int, text_start: int, text_len: int, mode: str,
                              head_param_bp: Optional[Sequence[int]] = None, text_sink: bool = True,
                              scale: Optional[float] = None, out=None, lse=None, want_lse: bool = True,
                              workspace: Optional[torch.Tensor] = None, base_sparsity_bp: int = 8000,
                              recall_threshold_bp: int = 8000,
                              result: Optional["SearchResult"] = None):
    """Algorithm 1 with one pass over Q K^T: dense attention with its LSE, the
    block masses of that LSE (added per key block from the attention pass's
    own exponentials) and the selection.  Returns (out, lse, SearchResult):
    out and lse bit for bit those of :func:`dense_attn_lse`; the masses are
    normalised by the LSE of the unrounded row sum, so they differ from
    :func:`block_search`'s given that lse (the LSE of the bf16-rounded
    weights) by up to 2^-9 relative.  ``workspace`` is a uint8 CUDA tensor:
    with :func:`single_pass_online_search_workspace` bytes every (batch, head)
    pair runs in one launch, with fewer (at least
    :func:`single_pass_online_search_min_workspace`) in groups; when not given
    (or below the minimum) the full size is allocated here."""
    _check_qkv(q, k, v)
    lib = load_library()
    B, H, L, D = q.shape
    dev = q.device
    nb = (L + block - 1) // block
    prob = _problem_shape(B, H, L, D, block, text_start, text_len, scale)
    sel, _keep = _select(mode, head_param_bp, text_sink, False, base_sparsity_bp,
                         recall_threshold_bp, heads=H)
    cap = lib.adaspa_block_search_capacity(ctypes.byref(prob), ctypes.byref(sel))
    wsb = lib.adaspa_single_pass_online_search_workspace(ctypes.byref(prob), ctypes.byref(sel))
    wsb_min = lib.adaspa_single_pass_online_search_min_workspace(ctypes.byref(prob), ctypes.byref(sel))
    if cap < 0 or wsb == 0:
        _check(lib.adaspa_single_pass_online_search(ctypes.byref(prob), None, None, None, None, None,
                                                    ctypes.byref(sel), None, None, None, 0, None, None,
                                                    None, 0, None))
        raise AdaspaError("invalid single_pass_online_search arguments")
    _check_outputs(q, out, lse)
    if out is None:
        out = torch.empty_like(q)
    if lse is None and want_lse:
        lse = torch.empty(B, H, L, dtype=torch.float32, device=dev)
    res = _search_outputs(B, H, nb, cap, dev, result)
    if workspace is None or _workspace_bytes(workspace, dev) < wsb_min:
        workspace = torch.empty(int(wsb), dtype=torch.uint8, device=dev)
    _check(lib.adaspa_single_pass_online_search(ctypes.byref(prob), _ptr(q), _ptr(k), _ptr(v), _ptr(out),
                                                _ptr(lse), ctypes.byref(sel), _ptr(res.block_mass),
                                                _ptr(res.row_ptr), _ptr(res.col_idx),
                                                int(res.col_idx.numel()), _ptr(res.head_k),
                                                _ptr(res.head_recall), _ptr(workspace),
                                                _workspace_bytes(workspace, dev), _stream(dev)))
    return out, lse, res


def block_sparse_attn(q, k, v, row_ptr, col_idx, *, block: int, scale: Optional[float] = None,
                      out=None, lse=None, want_lse: bool = True, text_start: int = 0,
                      text_len: int = 0, workspace=None, balance: bool = True):
    """Blockified sparse attention over the CSR key-block lists.  Returns (out, lse).
    ``text_start``/``text_len`` only order the work (text query blocks first).
    With ``balance`` (the default) the last tenth of the query blocks goes to
    the XCDs that run ahead, through per-XCD work queues whose counters live
    in ``workspace`` (uint8 CUDA tensor of at least
    ``block_sparse_attn_workspace(q.shape, block)`` bytes; allocated here when
    not given); ``balance=False`` splits the work statically.  The results
    are the same either way."""
    _check_qkv(q, k, v)
    lib = load_library()
    B, H, L, D = q.shape
    nb = (L + block - 1) // block
    for t in (row_ptr, col_idx):
        if t.dtype != torch.int32 or t.device != q.device or not t.is_contiguous():
            raise AdaspaError("row_ptr and col_idx must be contiguous int32 on q's device")
    if row_ptr.numel() != B * H * nb + 1:
        raise AdaspaError(f"row_ptr must have B*H*NB+1 = {B * H * nb + 1} entries")
    _check_outputs(q, out, lse)
    if out is None:
        out = torch.empty_like(q)
    if lse is None and want_lse:
        lse = torch.empty(B, H, L, dtype=torch.float32, device=q.device)
    prob = _problem(q, block, text_start, text_len, scale)
    ws_bytes = 0
    if balance:
        ws_bytes = int(lib.adaspa_block_sparse_attn_workspace(ctypes.byref(prob)))
        if workspace is None:
            workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=q.device)
        ws_bytes = _workspace_bytes(workspace, q.device)
    else:
        workspace = None
    _check(lib.adaspa_block_sparse_attn(ctypes.byref(prob), _ptr(q), _ptr(k), _ptr(v),
                                        _ptr(row_ptr), _ptr(col_idx), int(col_idx.numel()),
                                        _ptr(out), _ptr(lse), _ptr(workspace),
                                        ctypes.c_size_t(ws_bytes), _stream(q.device)))
    return out, lse


def block_sparse_attn_workspace(shape, block: int = 128, scale: Optional[float] = None) -> int:
    """Bytes of the work-queue workspace of :func:`block_sparse_attn`."""
    B, H, L, D = shape
    prob = _Problem(B, H, L, D, block, 0, 0, 0.0 if scale is None else float(scale))
    return int(load_library().adaspa_block_sparse_attn_workspace(ctypes.byref(prob)))


def block_sparse_attn_noalloc(q, k, v, row_ptr, col_idx, *, block: int, out, lse=None,
                              scale: Optional[float] = None, text_start: int = 0,
                              text_len: int = 0):
    """:func:`block_sparse_attn` through the allocation-free entry point: the
    caller passes ``out`` (and ``lse``, or None to skip it) and nothing is
    allocated, here or in the library, whose per-XCD work-queue counters sit
    in a small array of its own on each GPU.  Results are bitwise those of
    :func:`block_sparse_attn` with a workspace.  Calls on one GPU must not
    overlap (they share that GPU's counters)."""
    _check_qkv(q, k, v, out)
    lib = load_library()
    B, H, L, D = q.shape
    nb = (L + block - 1) // block
    for t in (row_ptr, col_idx):
        if t.dtype != torch.int32 or t.device != q.device or not t.is_contiguous():
            raise AdaspaError("row_ptr and col_idx must be contiguous int32 on q's device")
    if row_ptr.numel() != B * H * nb + 1:
        raise AdaspaError(f"row_ptr must have B*H*NB+1 = {B * H * nb + 1} entries")
    _check_outputs(q, out, lse)
    prob = _problem(q, block, text_start, text_len, scale)
    _check(lib.adaspa_block_sparse_attn_noalloc(ctypes.byref(prob), _ptr(q), _ptr(k), _ptr(v),
                                                _ptr(row_ptr), _ptr(col_idx), int(col_idx.numel()),
                                                _ptr(out), _ptr(lse), _stream(q.device)))
    return out, lse

