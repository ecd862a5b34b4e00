"""Seeded synthetic inputs shaped like the token sequences of a 720p video DiT.

This module is shared by the tests, the benchmark and the CPU oracle's callers.
It holds no arithmetic of the attention method itself: it only draws random
tensors and describes the workload shapes.

Token layout (the paper's sequence-length equation, Sec. 2.1): a sequence of
``L = f*h*w + t`` tokens, ``t`` text tokens and ``f`` latent frames of
``h*w`` patches each.  Video token ``v`` (0-based among the video tokens)
belongs to frame ``v // P`` and patch position ``v % P`` with ``P = h*w``.

Structure (imitating the hierarchical frame/text structure of Sec. 3,
Observation 1): for each (batch, head) one set of frame vectors ``U[f]`` and
one of patch-position vectors ``W[s]`` is drawn, shared by Q, K and V, and

    video token:  X = N_X + 0.8 * U[frame] + 0.6 * W[patch]
    text token:   X = N_X

with every entry of ``N_X``, ``U`` and ``W`` i.i.d. N(0, 1) and ``N_X``
independent per tensor (``head_structure`` scales the shared part per head).  The result is rounded to bf16 (round to nearest even,
torch's conversion).  Same-frame keys therefore gain about ``0.64*sqrt(D)`` in
the scaled score and same-patch keys about ``0.36*sqrt(D)``, which gives the
frame blocks, diagonals and stripes the paper describes.

Random draws use ``torch.Generator`` seeded per (workload seed, stream), on
the device the tensors are made on; results on CPU and GPU differ, so callers
that compare two implementations give both the same tensors.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional

import torch

__all__ = ["Workload", "TINY", "MODERATE", "LONG", "WORKLOADS", "make_qkv",
           "make_drift_noise", "text_blocks", "num_blocks", "random_block_lists",
           "random_block_masses"]


@dataclasses.dataclass(frozen=True)
class Workload:
    """Shape of one synthetic attention problem (one DiT attention call)."""
    name: str
    batch: int
    heads: int
    head_dim: int
    seqlen: int
    text_len: int
    frames: int           # latent frames f (the last one may be partial)
    patches: int          # patches per frame P = h*w
    block: int            # square block size of the sparse pattern
    seed: int
    coverage_bp: int = 9000          # per-head coverage target, basis points
    text_first: bool = True          # text tokens at [0, t) (else at the end)
    # Per-head weight of the shared frame/patch component, cycled over the
    # heads (empty: weight 1 for every head).  Unequal weights make heads of
    # different concentration: a weak structure spreads a row's mass over
    # many key blocks, a strong one gathers it in the frame and stripe blocks.
    head_structure: tuple = ()

    def __post_init__(self):
        # Every video token must fall in one of the drawn frames: make_qkv
        # indexes the frame table by v // patches, and on a GPU an index past
        # the table is a memory fault, not an error.
        if not (0 <= self.text_len <= self.seqlen):
            raise ValueError(f"{self.name}: text_len {self.text_len} outside [0, {self.seqlen}]")
        if self.patches < 1 or self.frames * self.patches < self.seqlen - self.text_len:
            raise ValueError(f"{self.name}: {self.frames} frames x {self.patches} patches hold fewer "
                             f"than the {self.seqlen - self.text_len} video tokens")

    @property
    def text_start(self) -> int:
        return 0 if self.text_first else self.seqlen - self.text_len

    @property
    def video_len(self) -> int:
        return self.seqlen - self.text_len

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.head_dim)

    @property
    def nblocks(self) -> int:
        return num_blocks(self.seqlen, self.block)

    def replace(self, **kw) -> "Workload":
        return dataclasses.replace(self, **kw)


# B=1, H=2, d=64, L=2048 = 64 text + 4 frames x 496 patches, block 64.
TINY = Workload("tiny_L2048_H2_d64_b64", 1, 2, 64, 2048, 64, 4, 496, 64, seed=0)
# B=1, H=48, d=64, L=17,920 = 256 text + 17,664 video, block 128.  17,664 video
# tokens at 1,358 patches per frame are 13 full frames plus 10 tokens of a 14th.
MODERATE = Workload("moderate_L17920_H48_d64_b128", 1, 48, 64, 17920, 256, 14, 1358,
                    128, seed=1)
# B=1, H=24, d=128, L=110,336 = 256 text + 32 frames x 3,440 patches, block 128.
LONG = Workload("long_L110336_H24_d128_b128", 1, 24, 128, 110336, 256, 32, 3440,
                128, seed=2)

WORKLOADS = {w.name: w for w in (TINY, MODERATE, LONG)}


def num_blocks(seqlen: int, block: int) -> int:
    return (seqlen + block - 1) // block


def text_blocks(seqlen: int, block: int, text_start: int, text_len: int) -> list[int]:
    """Indices of the blocks whose token range overlaps the text range."""
    if text_len <= 0:
        return []
    first = text_start // block
    last = (text_start + text_len - 1) // block
    return list(range(first, last + 1))


def _gen(seed: int, stream: int, device) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed * 1_000_003 + stream)
    return g


def make_qkv(w: Workload, device="cpu", heads: Optional[range] = None,
             fp32: bool = False):
    """Return (q, k, v), each [B, H, L, D] bf16 (or fp32 before rounding).

    ``heads`` restricts generation to a subset of heads (same values as the
    full draw for those heads, since every (b, h) uses its own streams).
    """
    hs = list(range(w.heads)) if heads is None else list(heads)
    B, L, D = w.batch, w.seqlen, w.head_dim
    out = [torch.empty(B, len(hs), L, D, dtype=torch.float32 if fp32 else torch.bfloat16,
                       device=device) for _ in range(3)]
    vid = torch.arange(w.video_len, device=device)
    frame = vid // w.patches
    patch = vid % w.patches
    t0 = w.text_start
    v0 = w.text_len if w.text_first else 0
    for b in range(B):
        for hi, h in enumerate(hs):
            base = (b * 65536 + h) * 8
            U = torch.randn(w.frames, D, generator=_gen(w.seed, base + 0, device), device=device)
            W = torch.randn(w.patches, D, generator=_gen(w.seed, base + 1, device), device=device)
            shared = 0.8 * U[frame] + 0.6 * W[patch]
            if w.head_structure:
                shared *= w.head_structure[h % len(w.head_structure)]
            for ti in range(3):
                x = torch.randn(L, D, generator=_gen(w.seed, base + 2 + ti, device), device=device)
                x[v0:v0 + w.video_len] += shared
                out[ti][b, hi].copy_(x)
            del shared
    assert 0 <= t0 <= L
    return tuple(out)


def make_drift_noise(w: Workload, device="cpu", seed: int = 4):
    """One fixed N(0,1) draw E per tensor for the denoising-drift workload,
    X_t = X_0 + (0.05 * t / 50) * E.  Returns fp32 [B, H, L, D] x 3."""
    B, H, L, D = w.batch, w.heads, w.seqlen, w.head_dim
    outs = []
    for ti in range(3):
        g = _gen(seed, 7919 + ti, device)
        outs.append(torch.randn(B, H, L, D, generator=g, device=device))
    return tuple(outs)


def random_block_masses(shape, seed: int, ties: bool = False) -> torch.Tensor:
    """fp32 block-mass-like values for selection tests (non-negative).

    With ``ties`` the values are drawn from a handful of levels, so many
    entries are exactly equal (exercises the lowest-index tie-break)."""
    g = _gen(seed, 31337, "cpu")
    if ties:
        lv = torch.tensor([0.0, 0.25, 0.5, 1.0, 2.0], dtype=torch.float32)
        idx = torch.randint(0, len(lv), shape, generator=g)
        return lv[idx]
    x = torch.rand(shape, generator=g, dtype=torch.float64)
    return (x ** 4 * 8.0).to(torch.float32)


def random_block_lists(nrows: int, nblocks: int, k: int, seed: int,
                       always: list[int] | None = None):
    """A seeded CSR block pattern: every row keeps ``k`` distinct key blocks
    (``always`` first), indices ascending.  Returns (row_ptr, col_idx) int32."""
    g = _gen(seed, 4242, "cpu")
    always = sorted(set(always or []))
    k = max(k, len(always))
    cols = []
    for _ in range(nrows):
        perm = torch.randperm(nblocks, generator=g).tolist()
        chosen = list(always)
        for c in perm:
            if len(chosen) >= k:
                break
            if c not in always:
                chosen.append(c)
        cols.append(sorted(chosen))
    row_ptr = torch.zeros(nrows + 1, dtype=torch.int32)
    row_ptr[1:] = torch.tensor([len(c) for c in cols], dtype=torch.int64).cumsum(0).to(torch.int32)
    col_idx = torch.tensor([c for row in cols for c in row], dtype=torch.int32)
    return row_ptr, col_idx


EXTREME_KINDS = ("negative", "rising", "spiky")


def make_extreme_qkv(kind: str, heads: int, seqlen: int, head_dim: int, seed: int = 11,
                     device="cpu"):
    """Seeded [1, H, L, D] bf16 inputs whose attention scores stress the
    softmax bookkeeping.  Each kind comes with the softmax scale it is meant
    for (returned second):

    - ``negative``: q ~ -2 + 0.3 N, k ~ 2 + 0.3 N, scale 1, so every scaled
      score of every row lies near -4 D, far below the fp32 exponent range;
    - ``rising``: q ~ 2 + 0.3 N, key j ~ a j + 0.3 N, default scale 1/sqrt(D),
      with a set so the scores rise by about 20 per 64 keys (the row maximum
      moves on every tile, by far more than a tile's probabilities allow);
    - ``spiky``: q, k ~ 2 N, scale 1, so scores spread by about 4 sqrt(D)
      times their own scale: large, random jumps of the row maximum.

    V is N(0, 1) throughout."""
    assert kind in EXTREME_KINDS
    H, L, D = heads, seqlen, head_dim
    g = _gen(seed, 5150 + EXTREME_KINDS.index(kind), device)
    nq = torch.randn(1, H, L, D, generator=g, device=device)
    nk = torch.randn(1, H, L, D, generator=g, device=device)
    v = torch.randn(1, H, L, D, generator=g, device=device)
    if kind == "negative":
        q, k, scale = -2.0 + 0.3 * nq, 2.0 + 0.3 * nk, 1.0
    elif kind == "rising":
        a = 20.0 / (64 * 2.0 * D ** 0.5)
        j = torch.arange(L, device=device, dtype=torch.float32).view(1, 1, L, 1)
        q, k, scale = 2.0 + 0.3 * nq, a * j + 0.3 * nk, D ** -0.5
    else:
        q, k, scale = 2.0 * nq, 2.0 * nk, 1.0
    bf = torch.bfloat16
    return (q.to(bf).contiguous(), k.to(bf).contiguous(), v.to(bf).contiguous()), scale
