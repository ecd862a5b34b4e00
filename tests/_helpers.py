"""Shared helpers of the GPU parity tests: tolerances and the oracle on sampled
rows.  Inputs come from the seeded generators in ``workloads``; expected
values come only from ``oracle``."""
from __future__ import annotations

import numpy as np
import torch

import oracle

# Tolerances fixed by the build target for bf16 attention outputs, LSE and
# block masses.  The mass floor guards fp32 underflow of negligible blocks.
OUT_MAX_ABS = 2e-2
OUT_MEAN_ABS = 2e-3
LSE_REL = 1e-3
MASS_REL = 1e-3
MASS_ABS_FLOOR = 1e-30


def f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def check_out(got: torch.Tensor, ref: np.ndarray, what: str = "out"):
    g = f64(got)
    err = np.abs(g - ref)
    assert np.all(np.isfinite(g)), f"{what}: non-finite output"
    mx, mean = float(err.max()), float(err.mean())
    assert mx <= OUT_MAX_ABS, f"{what}: max abs err {mx:.3e} (|ref| max {np.abs(ref).max():.2f})"
    assert mean <= OUT_MEAN_ABS, f"{what}: mean abs err {mean:.3e}"
    return mx, mean


def check_lse(got: torch.Tensor, ref: np.ndarray, what: str = "lse"):
    g = f64(got)
    fin = np.isfinite(ref)
    assert np.array_equal(np.isfinite(g), fin), f"{what}: finiteness differs"
    if fin.any():
        rel = np.abs(g[fin] - ref[fin]) / np.maximum(np.abs(ref[fin]), 1e-30)
        assert rel.max() <= LSE_REL, f"{what}: max rel err {rel.max():.3e}"
    assert np.all(g[~fin] == ref[~fin])


def check_mass(got, ref: np.ndarray, what: str = "mass"):
    g = f64(got) if isinstance(got, torch.Tensor) else np.asarray(got, np.float64)
    err = np.abs(g - ref)
    bound = MASS_REL * np.abs(ref) + MASS_ABS_FLOOR
    bad = err > bound
    assert not bad.any(), (f"{what}: {int(bad.sum())} entries off; worst rel "
                           f"{float((err / np.maximum(np.abs(ref), 1e-300)).max()):.3e}")


def oracle_rows(q, k, v, bh: tuple, rows: np.ndarray, scale: float):
    """Oracle dense output and LSE for the given query rows of head (b, h)."""
    b, h = bh
    qq = f64(q[b, h, torch.as_tensor(rows, device=q.device)])
    return oracle.dense_attention(qq, f64(k[b, h]), f64(v[b, h]), scale)


def csr_rows(row_ptr: torch.Tensor, col_idx: torch.Tensor):
    rp = row_ptr.cpu().numpy().astype(np.int64)
    ci = col_idx[: int(rp[-1])].cpu().numpy()
    return rp, ci


def sample_blocks(nb: int, n: int, seed: int, always=(0,)):
    rng = np.random.default_rng(seed)
    pick = set(int(x) for x in always if 0 <= x < nb)
    pick.add(nb - 1)
    rest = [p for p in range(nb) if p not in pick]
    if n > len(pick) and rest:
        pick.update(int(x) for x in rng.choice(rest, size=min(n - len(pick), len(rest)), replace=False))
    return sorted(pick)
