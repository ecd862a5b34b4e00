"""The benchmarked chain at the long-video shape (B=1, H=24, L=110,336, d=128,
block 128, and block 64, the paper's default, where NB = 1,724), in the
launch configuration the benchmark times: dense attention
+ LSE, then the search with the fresh LSE (coverage 0.9 per head, text sink,
caller workspace), then block-sparse attention with the text range given
(text query blocks first, queued tail).

The oracle gets only the seeded inputs, never a GPU result.  At this size it
can afford sampled query blocks: their LSE and block masses from Q and K, and
from those the check that every sampled row of the GPU's index lists is a
valid selection (text blocks kept, text query rows complete, the head's count
on video rows, and any block that differs from the oracle's top-k within
rounding of the k-th mass).  The sparse kernel is checked on a seeded pattern
shaped like the coverage pattern (complete text rows, short video rows whose
length varies by head) in the same launch configuration."""
import numpy as np
import pytest
import torch

import oracle
import paper_2502_21079_amd as ad
from workloads import LONG, make_qkv, random_block_lists, text_blocks
from _helpers import check_lse, check_mass, check_out, csr_rows, f64, sample_blocks

pytestmark = pytest.mark.gpu

HEADS = (0, 11, 23)


@pytest.fixture(scope="module")
def inputs():
    return make_qkv(LONG, device="cuda")


@pytest.fixture(scope="module", params=[128, 64], ids=["b128", "b64"])
def wl(request):
    return LONG if request.param == 128 else LONG.replace(block=64)


@pytest.fixture(scope="module")
def searched(inputs, wl):
    w = wl
    B, H, L, D = w.batch, w.heads, w.seqlen, w.head_dim
    q, k, v = inputs
    tau = [w.coverage_bp] * H
    _, lse = ad.dense_attn_lse(q, k, v)
    wsb = ad.block_search_workspace((B, H, L, D), w.block, w.text_start, w.text_len, "coverage", tau)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    res = ad.block_search(q, k, lse, block=w.block, text_start=w.text_start, text_len=w.text_len,
                          mode="coverage", head_param_bp=tau, workspace=ws)
    torch.cuda.synchronize()
    return res


def _oracle_masses(w, q, k, v, h, p):
    """Oracle LSE of query block p of head h (all keys), then its block masses."""
    rows = np.arange(p * w.block, min((p + 1) * w.block, w.seqlen))
    idx = torch.as_tensor(rows, device=q.device)
    qr = f64(q[0, h, idx])
    _, l_ref = oracle.dense_attention(qr, f64(k[0, h]), f64(v[0, h]), w.scale)
    return oracle.block_mass_rows(qr, f64(k[0, h]), l_ref, w.scale, w.block)


def test_chain_masses_and_selection_sampled(inputs, searched, wl):
    w = wl
    q, k, v = inputs
    res = searched
    nb = w.nblocks
    tk = set(text_blocks(w.seqlen, w.block, w.text_start, w.text_len))
    rp, ci = csr_rows(res.row_ptr, res.col_idx)
    gk = res.head_k.cpu().numpy()
    gr = res.head_recall.cpu().numpy()
    assert np.all(gr >= w.coverage_bp / 10000), "a head's Recall is below its target"
    for h in HEADS:
        kh = int(gk[0, h])
        assert len(tk) <= kh <= nb
        for p in sample_blocks(nb, 3, seed=900 + h, always=(0, 2)):
            ref = _oracle_masses(w, q, k, v, h, p)
            check_mass(res.block_mass[0, h, p], ref, f"h{h} p{p}")
            r = h * nb + p
            got = ci[rp[r]:rp[r + 1]]
            assert np.all(np.diff(got) > 0), f"h{h} p{p}: not strictly ascending"
            if p in tk:
                assert np.array_equal(got, np.arange(nb)), f"h{h} p{p}: text row not complete"
                continue
            assert len(got) == kh, f"h{h} p{p}: {len(got)} blocks, head count {kh}"
            assert tk <= set(got.tolist()), f"h{h} p{p}: text blocks missing"
            order = oracle.row_order(ref, tk)
            exp = set(order[:kh])
            others = np.array([ref[c] for c in range(nb) if c not in tk])
            kth = np.sort(others)[::-1][kh - len(tk) - 1]
            for c in set(got.tolist()) ^ exp:
                assert abs(ref[c] - kth) <= 1e-3 * kth, (h, p, c)


@pytest.fixture(scope="module")
def coverage_shaped_pattern(wl):
    """Seeded lists shaped like the coverage-0.9 pattern at this shape: text
    query blocks keep every block, video query blocks keep the text blocks
    plus a per-head number of others (15 to 60 blocks of 128 per row, twice
    as many blocks of 64)."""
    w = wl
    nb = w.nblocks
    tb = text_blocks(w.seqlen, w.block, w.text_start, w.text_len)
    f = 128 // w.block
    counts = np.random.default_rng(31).integers(15 * f, 60 * f + 1, size=w.heads)
    rows = []
    for h in range(w.heads):
        rp_h, ci_h = random_block_lists(nb, nb, int(counts[h]), seed=3100 + h, always=tb)
        for p in range(nb):
            rows.append(list(range(nb)) if p in tb else ci_h[rp_h[p]:rp_h[p + 1]].tolist())
    row_ptr = np.zeros(len(rows) + 1, dtype=np.int64)
    row_ptr[1:] = np.cumsum([len(r) for r in rows])
    col_idx = np.concatenate([np.asarray(r, dtype=np.int32) for r in rows])
    return row_ptr, col_idx


def test_sparse_coverage_shaped_as_benchmarked(inputs, coverage_shaped_pattern, wl):
    w = wl
    q, k, v = inputs
    nb = w.nblocks
    rpn, cin = coverage_shaped_pattern
    rp = torch.as_tensor(rpn.astype(np.int32), device="cuda")
    ci = torch.as_tensor(cin, device="cuda")
    out, lse = ad.block_sparse_attn(q, k, v, rp, ci, block=w.block, text_start=w.text_start,
                                    text_len=w.text_len)
    torch.cuda.synchronize()
    for h in HEADS:
        blocks = sample_blocks(nb, 4, seed=950 + h, always=(0, 1, 2, 3, 4))
        o_ref, l_ref = oracle.block_sparse_attention(f64(q[0, h]), f64(k[0, h]), f64(v[0, h]),
                                                     rpn[h * nb:(h + 1) * nb + 1], cin, w.scale,
                                                     w.block, qblocks=blocks)
        rows = np.concatenate([np.arange(p * w.block, min((p + 1) * w.block, w.seqlen))
                               for p in blocks])
        idx = torch.as_tensor(rows, device="cuda")
        check_out(out[0, h, idx], o_ref, f"h{h}")
        check_lse(lse[0, h, idx], l_ref, f"h{h}")
