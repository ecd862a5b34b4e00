"""Plain fp64 CPU oracle for AdaSpa's attention hot path (arXiv 2502.21079).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports, calls or links
this package: only the tests, the smoke check and the benchmark's CPU-baseline
leg use it.  It shares no code with the HIP library.

Every function computes the plain definition from the paper, in float64, on
the exact values of its (bf16) inputs, without blocking, fusion or online
rescaling:

* scores, LSE, dense attention ........ Sec. 2.2 (attention weights equation,
                                          LSE equation, safe softmax)
* block attention mass W_sum_attn ..... Sec. 4.1, definition of W_sum_attn;
                                          Algorithms 1 and 2 (second pass)
* optimal block selection S* .......... Sec. 4.1, optimal-sparse-indices
                                          equation; Sec. 4.3 text sink and
                                          row-wise uniform selection;
                                          Sec. 4.2 head-adaptive sparsity
* masked (block-sparse) attention ..... Sec. 4.1, blockified sparse attention
                                          with bias -c(1 - M) and c -> inf
* Recall .............................. Sec. 2.3, Recall equation

Readings of points the paper leaves open (see the numbered list in the module
``READINGS``) are shared with the HIP path only through this docstring and the
header that documents the library; no code is shared.

Parity status: every function here is pinned by the CPU tests against closed
forms, invariants, brute force and a hand-derived worked example.  The paper
prints no intermediate value (no LSE, mass or index list) of its own runs, so
nothing ties the oracle to the authors' numbers.
"""
from __future__ import annotations

import math
from typing import Sequence

import numpy as np

READINGS = """
R1  Algorithm 1 initialises row_max to 1: read as -infinity (a max starts empty).
R2  Algorithm 1's running sum and accumulator are not rescaled when the max
    changes: read as the standard online softmax (the cited Milakov and
    Gimelshein normaliser), which equals the plain LSE definition.
R3  Algorithm 1 returns acc unnormalised: read Out = acc / (row sum).
R4  Algorithms 1 and 2 take Dot(q, k) without 1/sqrt(D): the scale of the
    attention-weights equation applies (s = scale * q.k, scale = 1/sqrt(D)
    unless the caller overrides it).
R5  Algorithms 1 and 2 write p = Log(qk - LSE): read p = exp(s - LSE), the safe
    softmax of Sec. 2.2, so that a row's masses sum to 1.
R6  Sum(p) in the second pass sums both axes of the B x B tile: one scalar
    W_sum_attn[p, q] per block pair (the W_sum_attn definition).
R7  The sparse-attention equation multiplies scores by M, which would still give
    masked entries weight exp(0): read the bias form of Sec. 4.1 with c -> inf,
    so masked keys are excluded.
R8  Global top-(1-s)(L/B)^2 vs row-wise uniform selection (Sec. 4.3): selection
    is per query-block row with the same count k_h for every video row of a
    head; text query rows keep every key block (text sink).
R9  TOPK count: k_h = clamp(ceil(keep_bp * NKB / 10000), max(1, #text key
    blocks), NKB); forced text blocks count inside k_h.
R10 Text sink: a block is a text block if its token range overlaps the text
    range; text key blocks are always kept; text query rows keep all blocks.
R11 COVERAGE mode (the per-head coverage target): k_h is the smallest uniform
    per-row count whose head Recall reaches tau_h, text query rows counted as
    fully kept.  It is head-adaptive and row-wise uniform.
R12 Ordering of candidate key blocks in a row: text blocks first, then mass
    descending, then key-block index ascending; -0.0 equals +0.0; NaN masses
    rank last.  Kept indices are emitted ascending.
R13 Cumulative masses for coverage and Recall are exact integers: each fp32
    mass m is quantised to q = min(round_half_even(m * 2^32), cap) with
    cap = floor(2^62 / (NQB * NKB)); NaN and m <= 0 give 0, +inf gives cap.
    Coverage holds when kept * 10000 >= total * tau_bp (exact).  Head Recall
    is reported as float32(double(kept) / double(total)); with total = 0 the
    Recall is 1.
R14 Head-adaptive hierarchical mode (Sec. 4.2): n = #heads with Recall
    strictly above the threshold at base sparsity s, capped at floor(H/2);
    the n highest-Recall heads move to sparsity (1+s)/2, the n lowest to
    (3s-1)/2 (clamped at 0); ties rank by lower head index.
R15 A query row that keeps no key has output 0 and LSE -inf.
R16 LSE is the natural logarithm.
"""

_Q32 = float(2 ** 32)


def _f64(x) -> np.ndarray:
    return np.asarray(x, dtype=np.float64)


# ---------------------------------------------------------------------------
# Sec. 2.2: scores, log-sum-exp, dense attention
# ---------------------------------------------------------------------------

def attention_scores(q, k, scale: float) -> np.ndarray:
    """s_ij = scale * sum_d q_id k_jd  (attention-weights equation, Sec. 2.2;
    reading R4).  q: [Lq, D], k: [Lk, D] -> [Lq, Lk] float64."""
    return float(scale) * (_f64(q) @ _f64(k).T)


def log_sum_exp(s) -> np.ndarray:
    """LSE(z) = max_j z_j + log sum_j exp(z_j - max_k z_k)  (LSE equation,
    Sec. 2.2; natural log, R16).  Rows with every entry -inf give -inf (R15)."""
    s = _f64(s)
    m = s.max(axis=-1)
    finite = np.isfinite(m)
    m_safe = np.where(finite, m, 0.0)
    with np.errstate(invalid="ignore"):
        tot = np.exp(s - m_safe[..., None]).sum(axis=-1)
    out = m_safe + np.log(np.where(finite, tot, 1.0))
    return np.where(finite, out, -np.inf)


def dense_attention(q, k, v, scale: float):
    """O = Softmax_safe(scale * Q K^T) V and the per-row LSE (Sec. 2.2).

    q: [Lq, D] query rows (any subset of rows), k, v: [Lk, D].
    Returns (o [Lq, D], lse [Lq]) in float64."""
    s = attention_scores(q, k, scale)
    lse = log_sum_exp(s)
    w = np.exp(s - lse[:, None])          # safe softmax: exp(z_j - LSE(z))
    return w @ _f64(v), lse


# ---------------------------------------------------------------------------
# Sec. 4.1: block attention mass W_sum_attn (Algorithms 1 and 2, second pass)
# ---------------------------------------------------------------------------

def block_mass_rows(q_rows, k, lse_rows, scale: float, block: int) -> np.ndarray:
    """Sum over the given query rows and over each key block q of
    exp(s_ij - LSE_i) (W_sum_attn definition, Sec. 4.1; R5, R6).

    ``lse_rows`` is whatever LSE the caller supplies: the fresh one of the
    first pass (Algorithm 1) or one cached from an earlier step (Algorithm 2).
    There is no renormalisation.  Returns [NKB] float64."""
    s = attention_scores(q_rows, k, scale)
    p = np.exp(s - _f64(lse_rows)[:, None])
    Lk = p.shape[1]
    nkb = (Lk + block - 1) // block
    out = np.zeros(nkb)
    col = p.sum(axis=0)
    for qb in range(nkb):
        out[qb] = col[qb * block:(qb + 1) * block].sum()
    return out


def block_mass(q, k, lse, scale: float, block: int,
               qblocks: Sequence[int] | None = None) -> np.ndarray:
    """W_sum_attn for one head: [NQB, NKB] float64 (or only the listed
    query-block rows, in the listed order).  q, k: [L, D]; lse: [L]."""
    L = q.shape[0]
    nqb = (L + block - 1) // block
    rows = range(nqb) if qblocks is None else qblocks
    return np.stack([block_mass_rows(q[p * block:(p + 1) * block], k,
                                     lse[p * block:(p + 1) * block], scale, block)
                     for p in rows])


# ---------------------------------------------------------------------------
# Sec. 4.1 (S*), Sec. 4.3 (text sink, row-wise) and Sec. 4.2: selection
# ---------------------------------------------------------------------------

def text_block_set(seqlen: int, block: int, text_start: int, text_len: int) -> set:
    """Blocks whose token range overlaps [text_start, text_start+text_len) (R10)."""
    if text_len <= 0:
        return set()
    return set(range(text_start // block, (text_start + text_len - 1) // block + 1))


def quantize_q32(m: float, cap: int) -> int:
    """Exact integer stand-in of a non-negative fp32 mass (R13)."""
    m = float(m)
    if math.isnan(m) or m <= 0.0:
        return 0
    x = m * _Q32
    if x >= cap:
        return cap
    return min(int(round(x)), cap)          # Python round(): half to even


def row_order(masses: Sequence[float], text_kblocks: set) -> list:
    """Candidate key blocks of one row in selection order (R12)."""
    def key(qi):
        m = float(masses[qi])
        nan = math.isnan(m)
        return (qi not in text_kblocks, nan, 0.0 if nan else -m, qi)
    return sorted(range(len(masses)), key=key)


def topk_count(keep_bp: int, nkb: int, n_text_k: int) -> int:
    """R9: k_h = clamp(ceil(keep_bp * NKB / 10000), max(1, #text), NKB)."""
    k = (keep_bp * nkb + 9999) // 10000
    return max(max(1, n_text_k), min(k, nkb))


def _head_recall_curve(Wh, text_q, text_k, cap):
    """kept(k) for k = 0..NKB and the total, all exact integers (R11, R13)."""
    nqb, nkb = Wh.shape
    kept = [0] * (nkb + 1)
    total = 0
    orders = []
    for p in range(nqb):
        qv = [quantize_q32(Wh[p, j], cap) for j in range(nkb)]
        row_total = sum(qv)
        total += row_total
        if p in text_q:
            orders.append(None)
            for kk in range(nkb + 1):
                kept[kk] += row_total
            continue
        order = row_order(Wh[p], text_k)
        orders.append(order)
        acc = 0
        kept[0] += 0
        for kk in range(1, nkb + 1):
            acc += qv[order[kk - 1]]
            kept[kk] += acc
    return kept, total, orders


def _recall_f32(kept: int, total: int) -> np.float32:
    if total == 0:
        return np.float32(1.0)
    return np.float32(float(kept) / float(total))


def select_blocks(W, seqlen: int, block: int, text_start: int, text_len: int,
                  mode: str, head_param_bp: Sequence[int],
                  base_sparsity_bp: int = 8000, recall_threshold_bp: int = 8000,
                  text_sink: bool = True):
    """Block selection for every (b, h, query block) row.

    W: float32 [B, H, NQB, NKB] block masses.  ``mode`` is "topk" (per-head
    keep fraction in basis points), "coverage" (per-head Recall target tau in
    basis points, R11) or "hierarchical" (Sec. 4.2, R14; head_param_bp unused).
    Returns a dict with row_ptr (int64 [B*H*NQB+1]), col_idx (int32),
    head_k (int32 [B, H]) and head_recall (float32 [B, H]).
    Row r = (b*H + h)*NQB + p; kept indices ascending (R12)."""
    W = np.asarray(W, dtype=np.float32)
    B, H, nqb, nkb = W.shape
    cap = (2 ** 62) // (nqb * nkb)
    tk = text_block_set(seqlen, block, text_start, text_len) if text_sink else set()
    tq = tk
    kmin = max(1, len(tk))
    head_k = np.zeros((B, H), dtype=np.int32)
    head_recall = np.zeros((B, H), dtype=np.float32)
    orders_all = {}
    for b in range(B):
        curves = []
        for h in range(H):
            kept, total, orders = _head_recall_curve(W[b, h], tq, tk, cap)
            orders_all[(b, h)] = orders
            curves.append((kept, total))
        if mode == "topk":
            ks = [topk_count(int(head_param_bp[h]), nkb, len(tk)) for h in range(H)]
        elif mode == "coverage":
            ks = []
            for h in range(H):
                kept, total = curves[h]
                tau = int(head_param_bp[h])
                k = kmin
                while kept[k] * 10000 < total * tau:
                    k += 1
                ks.append(k)
        elif mode == "hierarchical":
            ks = hierarchical_counts([curves[h] for h in range(H)], nkb, len(tk),
                                     base_sparsity_bp, recall_threshold_bp)
        else:
            raise ValueError(mode)
        for h in range(H):
            kept, total = curves[h]
            head_k[b, h] = ks[h]
            head_recall[b, h] = _recall_f32(kept[ks[h]], total)
    row_ptr = [0]
    cols = []
    for b in range(B):
        for h in range(H):
            for p in range(nqb):
                order = orders_all[(b, h)][p]
                if order is None:
                    row = list(range(nkb))
                else:
                    row = sorted(order[:int(head_k[b, h])])
                cols.extend(row)
                row_ptr.append(row_ptr[-1] + len(row))
    return {"row_ptr": np.asarray(row_ptr, dtype=np.int64),
            "col_idx": np.asarray(cols, dtype=np.int32),
            "head_k": head_k, "head_recall": head_recall}


def hierarchical_counts(curves, nkb: int, n_text_k: int, base_sparsity_bp: int,
                        recall_threshold_bp: int) -> list:
    """Head-adaptive hierarchical sparsity (Sec. 4.2; R14).

    At base sparsity s every head keeps k(s) blocks per row; heads are ranked by
    their Recall there; n = #heads whose Recall exceeds the threshold (capped at
    floor(H/2)); the top-n heads move to sparsity (1+s)/2 and the bottom-n heads
    to (3s-1)/2, clamped at 0."""
    H = len(curves)
    keep0 = 10000 - base_sparsity_bp
    k0 = topk_count(keep0, nkb, n_text_k)
    rec = []
    for h, (kept, total) in enumerate(curves):
        # Recall > threshold, exactly: kept*10000 > total*thr (total 0 -> Recall 1)
        rec.append((kept[k0], total))
    def above(h):
        kept, total = rec[h]
        if total == 0:
            return 10000 > recall_threshold_bp
        return kept * 10000 > total * recall_threshold_bp
    from fractions import Fraction
    def r(h):
        kept, total = rec[h]
        return Fraction(1) if total == 0 else Fraction(kept, total)
    ranked = sorted(range(H), key=lambda h: (-r(h), h))
    n = min(sum(1 for h in range(H) if above(h)), H // 2)
    s = base_sparsity_bp
    s_hi = (10000 + s) // 2                       # (1+s)/2 in basis points
    s_lo = max(0, (3 * s - 10000) // 2)           # (3s-1)/2, clamped at 0
    ks = [k0] * H
    for h in ranked[:n]:
        ks[h] = topk_count(10000 - s_hi, nkb, n_text_k)
    for h in ranked[H - n:] if n > 0 else []:
        ks[h] = topk_count(10000 - s_lo, nkb, n_text_k)
    return ks


# ---------------------------------------------------------------------------
# Sec. 4.1: blockified sparse attention (bias form with c -> infinity, R7)
# ---------------------------------------------------------------------------

def key_mask_from_blocks(kept_blocks: Sequence[int], seqlen_k: int, block: int) -> np.ndarray:
    """Expand the kept key blocks of one query-block row to a token mask."""
    m = np.zeros(seqlen_k, dtype=bool)
    for c in kept_blocks:
        m[c * block:(c + 1) * block] = True
    return m


def masked_attention(q_rows, k, v, key_mask, scale: float):
    """Softmax_safe(scale * q K^T - inf * (1 - M)) V for query rows that share
    one key mask (one query-block row of M_S expanded, Sec. 4.1; R7, R15).

    With every key kept this performs exactly the operations of
    ``dense_attention`` and returns bit-identical results."""
    s = attention_scores(q_rows, k, scale)
    s = np.where(np.asarray(key_mask, dtype=bool)[None, :], s, -np.inf)
    lse = log_sum_exp(s)
    lse_safe = np.where(np.isfinite(lse), lse, 0.0)
    w = np.where(np.isfinite(lse)[:, None], np.exp(s - lse_safe[:, None]), 0.0)
    return w @ _f64(v), lse


def biased_attention(q_rows, k, v, key_mask, scale: float, c: float):
    """The bias form of Sec. 4.1 with a finite constant c (used only to pin R7)."""
    s = attention_scores(q_rows, k, scale) - c * (1.0 - np.asarray(key_mask, np.float64))[None, :]
    lse = log_sum_exp(s)
    return np.exp(s - lse[:, None]) @ _f64(v), lse


def block_sparse_attention(q, k, v, row_ptr, col_idx, scale: float, block: int,
                           qblocks: Sequence[int] | None = None):
    """Masked attention for one head from a CSR block list (rows = query
    blocks of this head).  Returns (o [L, D] or rows of the listed blocks,
    lse) in float64."""
    L = q.shape[0]
    nqb = (L + block - 1) // block
    rows = range(nqb) if qblocks is None else qblocks
    outs, lses = [], []
    for p in rows:
        kept = [int(c) for c in col_idx[row_ptr[p]:row_ptr[p + 1]]]
        mask = key_mask_from_blocks(kept, k.shape[0], block)
        o, l = masked_attention(q[p * block:(p + 1) * block], k, v, mask, scale)
        outs.append(o)
        lses.append(l)
    return np.concatenate(outs), np.concatenate(lses)


# ---------------------------------------------------------------------------
# Sec. 2.3: Recall
# ---------------------------------------------------------------------------

def recall(W_head, kept_rows: Sequence[Sequence[int]]) -> float:
    """Kept attention mass over total attention mass for one head, from the
    block masses (Recall equation, Sec. 2.3), in float64."""
    W_head = _f64(W_head)
    kept = sum(W_head[p, list(c)].sum() for p, c in enumerate(kept_rows))
    return float(kept / W_head.sum())
