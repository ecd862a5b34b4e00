"""Pins for the fp64 oracle: checks against what the paper and mathematics fix.

None of these re-types the oracle's own formula.  They use a hand-derived
worked example (tests/golden), closed forms, invariants, brute force over
every subset on tiny inputs, and special cases that reduce to simpler
definitions.  Each test names the oracle function and passage it pins.
"""
import itertools
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle
from workloads import TINY, make_qkv, random_block_masses

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "worked_example.json")


def _frac(s):
    return float(Fraction(s))


def _ln(s):
    assert s.startswith("ln ")
    return math.log(float(s[3:]))


@pytest.fixture(scope="module")
def worked():
    with open(GOLDEN) as f:
        g = json.load(f)
    a = np.array(g["a"], dtype=np.float64)
    q = np.log(a)
    k = np.eye(4)
    v = np.array(g["v"], dtype=np.float64)
    return g, q, k, v


# --- worked example (hand-derived, tests/golden/worked_example.json) -------

def test_worked_dense_and_lse(worked):
    g, q, k, v = worked
    o, lse = oracle.dense_attention(q, k, v, 1.0)
    exp_o = np.array([[_frac(x) for x in r] for r in g["dense_out"]])
    exp_l = np.array([_ln(x) for x in g["lse"]])
    np.testing.assert_allclose(o, exp_o, rtol=0, atol=1e-13)
    np.testing.assert_allclose(lse, exp_l, rtol=0, atol=1e-14)


def test_worked_block_mass(worked):
    g, q, k, v = worked
    _, lse = oracle.dense_attention(q, k, v, 1.0)
    W = oracle.block_mass(q, k, lse, 1.0, 2)
    exp_w = np.array([[_frac(x) for x in r] for r in g["block_mass"]])
    np.testing.assert_allclose(W, exp_w, rtol=0, atol=1e-14)


def test_worked_selection_and_sparse(worked):
    g, q, k, v = worked
    _, lse = oracle.dense_attention(q, k, v, 1.0)
    W = oracle.block_mass(q, k, lse, 1.0, 2).astype(np.float32)[None, None]
    nt = g["no_text"]
    sel = oracle.select_blocks(W, 4, 2, 0, 0, "topk", [nt["topk_keep_bp"]])
    assert int(sel["head_k"][0, 0]) == nt["k"]
    rows = [sel["col_idx"][sel["row_ptr"][p]:sel["row_ptr"][p + 1]].tolist() for p in range(2)]
    assert rows == nt["kept"]
    assert float(sel["head_recall"][0, 0]) == _frac(nt["recall"])
    for case in nt["coverage"]:
        s2 = oracle.select_blocks(W, 4, 2, 0, 0, "coverage", [case["tau_bp"]])
        assert int(s2["head_k"][0, 0]) == case["k"], case
    o, l = oracle.block_sparse_attention(q, k, v, sel["row_ptr"], sel["col_idx"], 1.0, 2)
    np.testing.assert_allclose(o, [[_frac(x) for x in r] for r in nt["sparse_out"]], atol=1e-13)
    np.testing.assert_allclose(l, [_ln(x) for x in nt["sparse_lse"]], atol=1e-14)
    ts = g["text_sink"]
    s3 = oracle.select_blocks(W, 4, 2, ts["text_start"], ts["text_len"], "topk",
                              [ts["topk_keep_bp"]])
    rows = [s3["col_idx"][s3["row_ptr"][p]:s3["row_ptr"][p + 1]].tolist() for p in range(2)]
    assert rows == ts["kept"]
    assert int(s3["head_k"][0, 0]) == ts["k"]
    assert float(s3["head_recall"][0, 0]) == _frac(ts["recall"])


# --- invariants and closed forms on structured inputs ----------------------

@pytest.fixture(scope="module")
def tiny_head():
    q, k, v = make_qkv(TINY.replace(seqlen=512, text_len=64, frames=4, patches=112), heads=range(1))
    return (q[0, 0].float().numpy().astype(np.float64), k[0, 0].float().numpy().astype(np.float64),
            v[0, 0].float().numpy().astype(np.float64))


def test_lse_equals_unshifted_log_sum(tiny_head):
    """P3: LSE_i = log(sum_j exp(s_ij)) computed with no max shift (scores here
    are far from fp64 overflow), term by term in a Python loop."""
    q, k, v = tiny_head
    _, lse = oracle.dense_attention(q, k, v, 0.125)
    for i in (0, 1, 63, 64, 300, 511):
        tot = 0.0
        for j in range(k.shape[0]):
            tot += math.exp(0.125 * math.fsum(q[i] * k[j]))
        assert abs(lse[i] - math.log(tot)) <= 1e-12 * abs(lse[i])


def test_block_mass_rows_sum_to_block_rows(tiny_head):
    """P2: with the fresh LSE every query row's probabilities sum to one, so a
    block row of W_sum_attn sums to the number of valid rows in the block
    (including a ragged last block)."""
    q, k, v = tiny_head
    for L in (512, 500):
        _, lse = oracle.dense_attention(q[:L], k[:L], v[:L], 0.125)
        W = oracle.block_mass(q[:L], k[:L], lse, 0.125, 64)
        nrows = [min(64, L - 64 * p) for p in range(W.shape[0])]
        np.testing.assert_allclose(W.sum(1), nrows, rtol=1e-12, atol=0)
        assert W.shape == (math.ceil(L / 64),) * 2


def test_output_is_convex_combination(tiny_head):
    """P8: every output coordinate lies between the min and max of V over the
    attended keys (dense and masked)."""
    q, k, v = tiny_head
    o, _ = oracle.dense_attention(q, k, v, 0.125)
    assert np.all(o <= v.max(0) + 1e-12) and np.all(o >= v.min(0) - 1e-12)
    mask = oracle.key_mask_from_blocks([1, 5], k.shape[0], 64)
    om, _ = oracle.masked_attention(q[:64], k, v, mask, 0.125)
    assert np.all(om <= v[mask].max(0) + 1e-12) and np.all(om >= v[mask].min(0) - 1e-12)


def test_zero_query_closed_form(tiny_head):
    """P6: Q = 0 gives uniform attention: o_i = mean_j v_j, LSE_i = log L and
    W[p, q] = |p| |q| / L."""
    _, k, v = tiny_head
    L = 320
    q = np.zeros((L, k.shape[1]))
    o, lse = oracle.dense_attention(q, k[:L], v[:L], 0.125)
    np.testing.assert_allclose(o, np.broadcast_to(v[:L].mean(0), o.shape), atol=1e-13)
    np.testing.assert_allclose(lse, math.log(L), rtol=0, atol=1e-13)
    W = oracle.block_mass(q, k[:L], lse, 0.125, 128)
    sizes = [128, 128, 64]
    exp_w = np.array([[a * b / L for b in sizes] for a in sizes])
    np.testing.assert_allclose(W, exp_w, rtol=1e-12)


def test_dominant_key_gives_one_hot():
    """P6: one key aligned with every query and far above the others makes
    the output that key's value row (up to exp(-huge))."""
    rng = np.random.default_rng(0)
    L, D = 200, 8
    q = np.zeros((L, D)); q[:, 0] = 10.0
    k = rng.standard_normal((L, D)) * 0.1
    k[37] = 0; k[37, 0] = 10.0
    v = rng.standard_normal((L, D))
    o, lse = oracle.dense_attention(q, k, v, 1.0)
    np.testing.assert_allclose(o, np.broadcast_to(v[37], o.shape), atol=1e-30 + 1e-12)
    np.testing.assert_allclose(lse, 100.0, atol=1e-12)


def test_all_blocks_kept_is_dense_exactly(tiny_head):
    """P1: selecting every block reproduces dense attention bit for bit."""
    q, k, v = tiny_head
    o, lse = oracle.dense_attention(q, k, v, 0.125)
    nb = 8
    row_ptr = np.arange(nb + 1) * nb
    col_idx = np.tile(np.arange(nb), nb)
    om, lm = oracle.block_sparse_attention(q, k, v, row_ptr, col_idx, 0.125, 64)
    assert np.array_equal(o, om) and np.array_equal(lse, lm)


def test_single_block_sequence_sparse_is_dense(tiny_head):
    """P6: with L = block there is one block; selection must keep it and the
    sparse result is the dense one."""
    q, k, v = tiny_head
    q, k, v = q[:64], k[:64], v[:64]
    o, lse = oracle.dense_attention(q, k, v, 0.125)
    W = oracle.block_mass(q, k, lse, 0.125, 64).astype(np.float32)[None, None]
    sel = oracle.select_blocks(W, 64, 64, 0, 0, "topk", [1])
    assert sel["col_idx"].tolist() == [0]
    om, lm = oracle.block_sparse_attention(q, k, v, sel["row_ptr"], sel["col_idx"], 0.125, 64)
    assert np.array_equal(o, om) and np.array_equal(lse, lm)


def test_bias_form_matches_block_skipping(tiny_head):
    """P9 (reading R7): the bias form -c(1-M) of Sec. 4.1 with a large finite c
    agrees with excluding the masked keys."""
    q, k, v = tiny_head
    mask = oracle.key_mask_from_blocks([0, 2, 7], k.shape[0], 64)
    o1, l1 = oracle.masked_attention(q[64:128], k, v, mask, 0.125)
    o2, l2 = oracle.biased_attention(q[64:128], k, v, mask, 0.125, c=1e4)
    assert np.max(np.abs(o1 - o2)) < 1e-300 or np.allclose(o1, o2, rtol=0, atol=1e-300)
    np.testing.assert_allclose(l1, l2, rtol=0, atol=1e-300)


def test_masked_attention_is_renormalised_dense_restricted(tiny_head):
    """Masked attention equals the dense weights restricted to kept keys and
    renormalised by their kept mass (a consequence of the safe softmax)."""
    q, k, v = tiny_head
    s = oracle.attention_scores(q[:64], k, 0.125)
    mask = oracle.key_mask_from_blocks([3, 4], k.shape[0], 64)
    p = np.exp(s - s.max(1, keepdims=True)) * mask[None, :]
    expect = (p / p.sum(1, keepdims=True)) @ v
    o, _ = oracle.masked_attention(q[:64], k, v, mask, 0.125)
    np.testing.assert_allclose(o, expect, rtol=1e-12, atol=1e-12)


def test_cached_lse_equals_fresh_when_unchanged(tiny_head):
    """P10: block mass from a cached LSE (Algorithm 2) equals the fused search
    (Algorithm 1) when the cache holds the same LSE, and scales by
    exp(LSE_fresh - LSE_cached) row by row otherwise."""
    q, k, v = tiny_head
    _, lse = oracle.dense_attention(q, k, v, 0.125)
    W1 = oracle.block_mass(q, k, lse, 0.125, 64)
    W2 = oracle.block_mass(q, k, lse.copy(), 0.125, 64)
    assert np.array_equal(W1, W2)
    shift = np.zeros_like(lse); shift[:64] = 0.5      # stale LSE on block row 0
    W3 = oracle.block_mass(q, k, lse + shift, 0.125, 64)
    np.testing.assert_allclose(W3[0], W1[0] * math.exp(-0.5), rtol=1e-12)
    assert np.array_equal(W3[1:], W1[1:])


def test_key_block_permutation_equivariance(tiny_head):
    """P11: permuting key blocks (with their values) permutes the columns of
    W_sum_attn and leaves the output unchanged."""
    q, k, v = tiny_head
    perm = [3, 0, 7, 1, 6, 2, 5, 4]
    tok = np.concatenate([np.arange(c * 64, (c + 1) * 64) for c in perm])
    o, lse = oracle.dense_attention(q, k, v, 0.125)
    op, lsep = oracle.dense_attention(q, k[tok], v[tok], 0.125)
    np.testing.assert_allclose(op, o, rtol=1e-12, atol=1e-12)
    W = oracle.block_mass(q, k, lse, 0.125, 64)
    Wp = oracle.block_mass(q, k[tok], lsep, 0.125, 64)
    np.testing.assert_allclose(Wp, W[:, perm], rtol=1e-12)


# --- selection: brute force, optimality, coverage minimality ----------------

def _brute_topk_rows(W, k, text):
    """Independent brute force: forced text blocks, then the remaining blocks
    by (mass descending, index ascending), via Python's sort of tuples."""
    rows = []
    for p in range(W.shape[0]):
        forced = [c for c in range(W.shape[1]) if c in text]
        rest = sorted((c for c in range(W.shape[1]) if c not in text),
                      key=lambda c: (-float(W[p, c]), c))
        rows.append(sorted(forced + rest[:k - len(forced)]) if p not in text else list(range(W.shape[1])))
    return rows


@pytest.mark.parametrize("seed,ties", [(0, False), (1, True), (2, True)])
@pytest.mark.parametrize("text", [(0, 0), (0, 64), (448, 64), (100, 40)])
def test_selection_matches_brute_force_sort(seed, ties, text):
    """P4: TOPK selection == brute-force sort on small inputs, including many
    exact ties (lowest index wins) and text placed first, last or unaligned."""
    nb = 8
    W = random_block_masses((1, 3, nb, nb), seed, ties=ties).numpy()
    tset = oracle.text_block_set(512, 64, *text)
    # Counts worked out by hand for NB = 8: ceil(keep * 8 / 10000) is 0, 1, 1,
    # 3, 4, 8, 8 for these keep fractions, raised to at least one block and to
    # at least the forced text blocks (two for the unaligned range 100..139).
    kmin = 2 if text == (100, 40) else 1
    expect_k = dict(zip((0, 1, 1250, 3000, 5000, 9999, 10000),
                        [max(kmin, x) for x in (0, 1, 1, 3, 4, 8, 8)]))
    for keep, k in expect_k.items():
        sel = oracle.select_blocks(W, 512, 64, text[0], text[1], "topk", [keep] * 3)
        for h in range(3):
            assert sel["head_k"][0, h] == k
            got = [sel["col_idx"][sel["row_ptr"][h * nb + p]:sel["row_ptr"][h * nb + p + 1]].tolist()
                   for p in range(nb)]
            assert got == _brute_topk_rows(W[0, h], k, tset)


def test_topk_row_is_optimal_over_all_subsets():
    """P5: the per-row top-k keeps at least as much mass as every other k-subset
    that contains the forced text blocks (Eq. for S*: top-k of W_sum_attn is
    the argmax of the kept mass)."""
    nb = 9
    W = random_block_masses((1, 1, nb, nb), 5).numpy().astype(np.float64)
    text = {0}
    for keep in (2000, 4000, 6000):
        sel = oracle.select_blocks(W.astype(np.float32), nb * 32, 32, 0, 32, "topk", [keep])
        k = int(sel["head_k"][0, 0])
        for p in range(1, nb):
            kept = sel["col_idx"][sel["row_ptr"][p]:sel["row_ptr"][p + 1]].tolist()
            best = max(sum(W[0, 0, p, list(s)]) for s in itertools.combinations(range(nb), k)
                       if text <= set(s))
            assert sum(W[0, 0, p, kept]) == pytest.approx(best, rel=1e-12)


def test_coverage_k_is_minimal_and_recall_monotone():
    """P7: Recall(k) is non-decreasing, Recall(NKB) == 1 exactly, and the
    COVERAGE count is the smallest k whose Recall reaches tau (checked with
    exact rational arithmetic on dyadic masses, so the integer stand-in of the
    masses is exact)."""
    nb = 10
    rng = np.random.default_rng(7)
    W = (rng.integers(0, 64, size=(1, 2, nb, nb)) / 16.0).astype(np.float32)
    text = {0}
    for tau in (0, 1, 5000, 8000, 9000, 9900, 10000):
        sel = oracle.select_blocks(W, nb * 16, 16, 0, 16, "coverage", [tau, tau])
        for h in range(2):
            Wh = W[0, h].astype(np.float64)
            total = Fraction(Wh.sum())
            def rec(k):
                kept = Fraction(0)
                for p in range(nb):
                    rows = _brute_topk_rows(Wh, k, text)
                    kept += sum(Fraction(Wh[p, c]) for c in rows[p])
                return kept / total
            curve = [rec(k) for k in range(1, nb + 1)]
            assert all(a <= b for a, b in zip(curve, curve[1:]))
            assert curve[-1] == 1
            k = int(sel["head_k"][0, h])
            assert curve[k - 1] >= Fraction(tau, 10000)
            if k > 1:
                assert curve[k - 2] < Fraction(tau, 10000)
            assert float(sel["head_recall"][0, h]) == pytest.approx(float(curve[k - 1]), rel=1e-7)


def test_selection_nan_and_negative_zero():
    """R12: -0.0 ties with +0.0 (lowest index wins); NaN ranks last and
    contributes nothing to Recall."""
    W = np.array([[[[0.0, -0.0, np.nan, 0.5], [np.nan, np.nan, 1.0, -0.0],
                    [-0.0, 0.0, 0.0, 0.0], [2.0, np.nan, 2.0, 1.0]]]], dtype=np.float32)
    sel = oracle.select_blocks(W, 4, 1, 0, 0, "topk", [5000])
    rows = [sel["col_idx"][sel["row_ptr"][p]:sel["row_ptr"][p + 1]].tolist() for p in range(4)]
    assert rows == [[0, 3], [2, 3], [0, 1], [0, 2]]


def test_q32_quantisation():
    """R13 edge cases of the exact-integer stand-in."""
    cap = 2 ** 62 // 100
    assert oracle.quantize_q32(0.0, cap) == 0
    assert oracle.quantize_q32(-0.0, cap) == 0
    assert oracle.quantize_q32(float("nan"), cap) == 0
    assert oracle.quantize_q32(-3.0, cap) == 0
    assert oracle.quantize_q32(float("inf"), cap) == cap
    assert oracle.quantize_q32(1.0, cap) == 2 ** 32
    assert oracle.quantize_q32(2.0 ** -33, cap) == 0          # half rounds to even (0)
    assert oracle.quantize_q32(3 * 2.0 ** -33, cap) == 2      # 1.5 -> 2
    assert oracle.quantize_q32(1e30, cap) == cap


def test_hierarchical_mode_levels():
    """R14 (Sec. 4.2): with base sparsity 0.8 the n heads above Recall 0.8 move
    to sparsity 0.9 and the n lowest to 0.7, keeping the mean count when k
    divides evenly; n is capped at floor(H/2)."""
    nb = 20
    H = 5
    W = np.zeros((1, H, nb, nb), dtype=np.float32)
    # head h concentrates its mass on the diagonal with strength decreasing in h
    for h in range(H):
        for p in range(nb):
            W[0, h, p] = 1.0
            W[0, h, p, p] = 1.0 + 400.0 / (h + 1) ** 3
    sel = oracle.select_blocks(W, nb * 16, 16, 0, 0, "hierarchical", [0] * H,
                               base_sparsity_bp=8000, recall_threshold_bp=8000)
    # base k = 4 of 20; Recall at k=4 per head: strong diagonal heads exceed 0.8
    k0 = 4
    recs = []
    for h in range(H):
        r = (W[0, h].astype(np.float64).max(1) + 3).sum() / W[0, h].astype(np.float64).sum()
        recs.append(r)
    n = min(sum(r > 0.8 for r in recs), H // 2)
    ranked = sorted(range(H), key=lambda h: (-recs[h], h))
    expect = [k0] * H
    for h in ranked[:n]:
        expect[h] = 2          # sparsity 0.9 -> keep 10% of 20
    for h in ranked[H - n:] if n else []:
        expect[h] = 6          # sparsity 0.7 -> keep 30% of 20
    assert sel["head_k"][0].tolist() == expect
    assert n >= 1


# --- hand-derived values for the remaining oracle functions ----------------

def test_recall_worked_example(worked):
    """Recall equation (Sec. 2.3): kept mass over total mass, from the block
    masses of the worked example.  Without text sink the top-1 rows keep
    W[0,1] and W[1,0]: (5/4 + 5/4) / 4 = 5/8; with the text sink block row 0
    is a text row kept whole: (2 + 5/4) / 4 = 13/16.  Keeping everything gives
    1 and keeping nothing 0."""
    g, q, k, v = worked
    _, lse = oracle.dense_attention(q, k, v, 1.0)
    W = oracle.block_mass(q, k, lse, 1.0, 2)
    assert oracle.recall(W, [[1], [0]]) == pytest.approx(_frac(g["no_text"]["recall"]), abs=1e-15)
    assert oracle.recall(W, [[0, 1], [0]]) == pytest.approx(_frac(g["text_sink"]["recall"]), abs=1e-15)
    assert oracle.recall(W, [[0, 1], [0, 1]]) == pytest.approx(1.0, abs=1e-15)
    assert oracle.recall(W, [[], []]) == 0.0
    # a row listed out of order counts the same blocks
    assert oracle.recall(W, [[1, 0], [0]]) == pytest.approx(13 / 16, abs=1e-15)


@pytest.mark.parametrize("rng_,block,expect", [
    ((100, 40), 64, {1, 2}),        # tokens 100..139: blocks [64,128) and [128,192)
    ((63, 2), 64, {0, 1}),          # tokens 63, 64 straddle the first boundary
    ((64, 64), 64, {1}),            # exactly block 1
    ((127, 1), 64, {1}),            # the last token of block 1
    ((128, 1), 64, {2}),            # the first token of block 2
    ((0, 1), 64, {0}),
    ((0, 256), 128, {0, 1}),        # the long-video text range at block 128
    ((0, 256), 64, {0, 1, 2, 3}),   # ... and at block 64
    ((1000, 300), 128, {7, 8, 9, 10}),   # tokens 1000..1299: blocks 7 (896..1023) to 10 (1280..1407)
    ((500, 0), 64, set()),          # no text
])
def test_text_block_set_hand_derived(rng_, block, expect):
    """Text sink (Sec. 4.3, reading R10): a block is a text block when its
    token range overlaps the text range; expected sets worked out by hand
    from the token ranges, including unaligned starts and ends."""
    assert oracle.text_block_set(4096, block, *rng_) == expect


def test_topk_count_fixed_values():
    """Reading R9 at the long-video shape (NB = 862 key blocks of 128, two
    text blocks): keep 5/10/20/50% give 44/87/173/431 blocks per video row
    (ceil of 43.1, 86.2, 172.4 and 431.0); at block 64 (NB = 1,724, four text
    blocks) keep 10% gives 173.  The clamps: nothing kept still keeps the text
    blocks (or one block without text), everything kept is NB."""
    assert [oracle.topk_count(b, 862, 2) for b in (500, 1000, 2000, 5000)] == [44, 87, 173, 431]
    assert oracle.topk_count(1000, 1724, 4) == 173
    assert oracle.topk_count(0, 862, 2) == 2
    assert oracle.topk_count(0, 10, 0) == 1
    assert oracle.topk_count(1, 862, 0) == 1            # ceil(0.0862)
    assert oracle.topk_count(10000, 862, 2) == 862
    assert oracle.topk_count(9999, 862, 2) == 862       # ceil(861.9138)
    assert oracle.topk_count(100, 3, 5) == 5            # the text blocks win over the fraction


def _two_block_heads(strengths, nb=10):
    """Head h: every row p keeps mass a_h on blocks p and p+1 (mod nb) and 1
    elsewhere, so its Recall at k = 1, 2, 3 ... is known by hand."""
    W = np.ones((1, len(strengths), nb, nb), dtype=np.float32)
    for h, a in enumerate(strengths):
        for p in range(nb):
            W[0, h, p, p] = a
            W[0, h, p, (p + 1) % nb] = a
    return W


def test_hierarchical_cap_clamp_and_strict_threshold():
    """Sec. 4.2 head-adaptive sparsity (reading R14), values worked out by
    hand on heads whose Recall is known in closed form: with strengths a_h on
    two blocks per row and 1 on the other eight, the Recall at k = 2 is
    2a/(2a + 8).

    * a = 100, 50, 20, 10 (Recall 0.96, 0.93, 0.83, 0.71 at base sparsity 0.8,
      k = 2): all four exceed 0.5, so n = 4 is capped at floor(4/2) = 2; the
      top two move to sparsity 0.9 (k = 1), the bottom two to 0.7 (k = 3).
    * the same heads at base sparsity 0.2 (k = 8): (3s-1)/2 = -0.2 is clamped
      to 0 (k = 10, every block), (1+s)/2 = 0.6 keeps 40% (k = 4).
    * three heads (cap floor(3/2) = 1): only the top and bottom head move.
    * "exceeds" is strict: a = 12 gives Recall exactly 24/32 = 0.75 at k = 2,
      which does not exceed a threshold of 0.75 (n = 1 from a = 100 alone)."""
    nb = 10
    W = _two_block_heads([100, 50, 20, 10], nb)
    sel = oracle.select_blocks(W, nb * 16, 16, 0, 0, "hierarchical", None,
                               base_sparsity_bp=8000, recall_threshold_bp=5000)
    assert sel["head_k"][0].tolist() == [1, 1, 3, 3]
    sel = oracle.select_blocks(W, nb * 16, 16, 0, 0, "hierarchical", None,
                               base_sparsity_bp=2000, recall_threshold_bp=5000)
    assert sel["head_k"][0].tolist() == [4, 4, 10, 10]
    W3 = _two_block_heads([20, 100, 10], nb)
    sel = oracle.select_blocks(W3, nb * 16, 16, 0, 0, "hierarchical", None,
                               base_sparsity_bp=8000, recall_threshold_bp=5000)
    assert sel["head_k"][0].tolist() == [2, 1, 3]
    Ws = _two_block_heads([100, 12, 12, 12], nb)
    sel = oracle.select_blocks(Ws, nb * 16, 16, 0, 0, "hierarchical", None,
                               base_sparsity_bp=8000, recall_threshold_bp=7500)
    # n = 1: head 0 -> k = 1; the lowest Recall ties (0.75 each) go to the
    # highest head index last in the ranking, so head 3 -> k = 3
    assert sel["head_k"][0].tolist() == [1, 2, 2, 3]
    assert float(sel["head_recall"][0, 1]) == 0.75
