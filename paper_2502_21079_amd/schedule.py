"""Denoising-step schedule of AdaSpa's two-phase online search.

The paper runs the search only at a few denoising steps and reuses its result
in between, because the sparse pattern and the LSE of an attention head stay
nearly invariant across steps (Sec. 3, Solution 2).  Its overview figure and
Sec. 4.2 ("Fused LSE-Cached Online Search") give the schedule: a set of
search steps T_s = {t_s^1, t_s^2, ...}; before t_s^1 every step runs full
attention (warm-up); at t_s^1 the fused search (Algorithm 1) runs full
attention, keeps its LSE and selects the block pattern from the masses of
that fresh LSE; the steps after it run block-sparse attention with that
pattern; at every later t_s^i the LSE-cached search (Algorithm 2) selects a
new pattern from the current Q, K and the LSE kept at t_s^1, and step t_s^i
and the steps after it use the new pattern.  Sec. 5 uses T_s = {10, 30}
with the first 10 steps at full attention.

Step indices here are 0-based (t = 0 .. T-1): with T_s = {10, 30}, steps
0-9 run full attention (the paper's ten warm-up steps), step 10 the fused
search (its output is full attention), steps 11-29 sparse attention with
the first pattern, step 30 the cached search and sparse attention with the
second pattern, which the later steps keep.  T_s = {0, 30} (the paper's
length-scaling setting) has no warm-up.

Every computation runs in the HIP library through the C ABI calls; this
module only decides which call each step makes and owns the buffers the
steps share (the cached LSE, the current pattern, the workspaces).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional, Sequence, Tuple

import torch

from . import (AdaspaError, SearchResult, block_search, block_search_workspace,
               block_sparse_attn, block_sparse_attn_workspace, dense_attn_lse,
               dense_attn_workspace, fused_online_search, single_pass_online_search,
               single_pass_online_search_workspace)

__all__ = ["DENSE", "FUSED_SEARCH", "CACHED_SEARCH", "SPARSE", "SearchSchedule",
           "AdaSpaAttention", "SEARCH_KERNELS"]

DENSE = "dense"                   # warm-up: full attention
FUSED_SEARCH = "fused_search"     # Algorithm 1: full attention + LSE + search from the fresh LSE
CACHED_SEARCH = "cached_search"   # Algorithm 2: search from the cached LSE, then sparse attention
SPARSE = "sparse"                 # block-sparse attention with the current pattern

# How the fused search step (Algorithm 1) runs: as one pass over Q K^T
# (single_pass_online_search: the attention pass also adds its exponentials
# per key block), as one launch of both passes (fused_online_search), or as
# dense attention followed by the search.  All give the same output and LSE;
# the single pass's masses are normalised by the unrounded row sum, the
# others' by the stored LSE, so they differ by up to 2^-9 relative.
SEARCH_KERNELS = ("single_pass", "fused", "two_calls")


@dataclass(frozen=True)
class SearchSchedule:
    """Which call each denoising step makes, from the search steps T_s."""
    search_steps: Tuple[int, ...] = (10, 30)

    def __post_init__(self):
        s = tuple(sorted(set(int(t) for t in self.search_steps)))
        if not s or s[0] < 0:
            raise AdaspaError("search_steps needs at least one step, all >= 0")
        object.__setattr__(self, "search_steps", s)

    @property
    def warmup(self) -> int:
        """Number of full-attention steps before the fused search."""
        return self.search_steps[0]

    def action(self, t: int) -> str:
        first = self.search_steps[0]
        if t < first:
            return DENSE
        if t == first:
            return FUSED_SEARCH
        if t in self.search_steps:
            return CACHED_SEARCH
        return SPARSE

    def pattern_step(self, t: int) -> Optional[int]:
        """The search step whose pattern step t's sparse attention uses (None
        for the steps that run full attention)."""
        if t <= self.search_steps[0]:
            return None
        return max(s for s in self.search_steps if s <= t)


@dataclass
class AdaSpaAttention:
    """AdaSpa state of one attention layer across the denoising steps.

    ``step(t, q, k, v)`` makes the call the schedule names for step t and
    returns the attention output; the LSE of the fused search and the
    current block pattern persist between steps.  ``shape`` is (B, H, L, D);
    the selection arguments are those of :func:`block_search`.
    ``search_kernel`` (one of SEARCH_KERNELS) chooses how the fused search
    step runs.  The default, "single_pass", takes one pass over Q K^T and is
    the fastest on MI355X (110K tokens, block 128: about 0.1 of a dense pass
    on top of it, against 0.55 for the two calls); it needs a workspace of
    B*H*NB*L floats (9.1 GB at that size).  "fused" runs both passes in one
    launch and "two_calls" dense attention followed by the search; those
    two give bitwise the same results as each other.

    The search workspace is scratch (nothing in it is read by a later call),
    so the layers of a model that run one after another can share one:
    pass ``search_workspace`` (uint8, at least :meth:`search_workspace_bytes`
    bytes, on the layer's device); otherwise each layer allocates its own.
    The LSE and the pattern, which persist between steps, stay per layer."""
    shape: Tuple[int, int, int, int]
    block: int
    text_start: int
    text_len: int
    mode: str = "coverage"
    head_param_bp: Optional[Sequence[int]] = None
    base_sparsity_bp: int = 8000
    recall_threshold_bp: int = 8000
    schedule: SearchSchedule = field(default_factory=SearchSchedule)
    scale: Optional[float] = None
    device: str = "cuda"
    search_kernel: str = "single_pass"
    search_workspace: Optional[torch.Tensor] = None

    def search_workspace_bytes(self) -> int:
        """Bytes of scratch the searches of this layer need."""
        wsb = block_search_workspace(self.shape, self.block, self.text_start, self.text_len, self.mode,
                                     self.head_param_bp)
        if self.search_kernel == "single_pass":
            wsb = max(wsb, single_pass_online_search_workspace(
                self.shape, self.block, self.text_start, self.text_len, self.mode, self.head_param_bp,
                base_sparsity_bp=self.base_sparsity_bp, recall_threshold_bp=self.recall_threshold_bp))
        return int(wsb)

    def __post_init__(self):
        if self.search_kernel not in SEARCH_KERNELS:
            raise AdaspaError(f"search_kernel must be one of {SEARCH_KERNELS}, got {self.search_kernel!r}")
        B, H, L, D = self.shape
        dev = self.device
        self.lse = torch.empty(B, H, L, dtype=torch.float32, device=dev)   # the cached LSE
        self.search: Optional[SearchResult] = None                          # the current pattern
        self.search_step: Optional[int] = None
        self.lse_step: Optional[int] = None
        # The single pass's workspace holds the search's, so one buffer serves
        # both searches.
        wsb = self.search_workspace_bytes()
        ws = self.search_workspace
        if ws is not None:
            if ws.dtype != torch.uint8 or ws.numel() < wsb or ws.device != torch.device(dev) or \
                    not ws.is_contiguous():
                raise AdaspaError(f"search_workspace must be contiguous uint8 of at least {wsb} bytes on {dev}")
            self._ws_search = ws
        else:
            self._ws_search = torch.empty(wsb, dtype=torch.uint8, device=dev)
        self._ws_dense = torch.empty(dense_attn_workspace(self.shape, self.scale), dtype=torch.uint8,
                                     device=dev)
        self._ws_sparse = torch.empty(block_sparse_attn_workspace(self.shape, self.block, self.scale),
                                      dtype=torch.uint8, device=dev)

    def _search(self, q, k):
        self.search = block_search(q, k, self.lse, block=self.block, text_start=self.text_start,
                                   text_len=self.text_len, mode=self.mode,
                                   head_param_bp=self.head_param_bp, scale=self.scale,
                                   workspace=self._ws_search, base_sparsity_bp=self.base_sparsity_bp,
                                   recall_threshold_bp=self.recall_threshold_bp, result=self.search)

    def step(self, t: int, q, k, v, out=None):
        """Run step t; returns (out, action)."""
        if tuple(q.shape) != tuple(self.shape):
            raise AdaspaError(f"q has shape {tuple(q.shape)}, the layer was set up for {self.shape}")
        a = self.schedule.action(t)
        if out is None:
            out = torch.empty_like(q)
        if a == DENSE:
            dense_attn_lse(q, k, v, scale=self.scale, out=out, want_lse=False,
                           workspace=self._ws_dense)
            return out, a
        if a == FUSED_SEARCH:
            if self.search_kernel in ("single_pass", "fused"):
                fn = single_pass_online_search if self.search_kernel == "single_pass" else fused_online_search
                _, _, self.search = fn(
                    q, k, v, block=self.block, text_start=self.text_start, text_len=self.text_len,
                    mode=self.mode, head_param_bp=self.head_param_bp, scale=self.scale, out=out,
                    lse=self.lse, workspace=self._ws_search, base_sparsity_bp=self.base_sparsity_bp,
                    recall_threshold_bp=self.recall_threshold_bp, result=self.search)
            else:
                dense_attn_lse(q, k, v, scale=self.scale, out=out, lse=self.lse,
                               workspace=self._ws_dense)
                self._search(q, k)
            self.lse_step = t
            self.search_step = t
            return out, a
        if self.search is None:
            raise AdaspaError(f"step {t}: no search has run yet (search steps {self.schedule.search_steps})")
        if a == CACHED_SEARCH:
            self._search(q, k)            # masses from the LSE kept at the fused search
            self.search_step = t
        block_sparse_attn(q, k, v, self.search.row_ptr, self.search.col_idx, block=self.block,
                          scale=self.scale, out=out, want_lse=False, text_start=self.text_start,
                          text_len=self.text_len, workspace=self._ws_sparse)
        return out, a
