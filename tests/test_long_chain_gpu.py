"""The benchmarked chain at the long-video shape (B=1, H=24, L=110,336, d=128,
block 128), in the launch configuration the benchmark times: dense attention
+ LSE, then the search with the fresh LSE (coverage 0.9 per head, text sink,
caller workspace), then block-sparse attention on the CSR it emitted.

Every stage is checked against the oracle on what the oracle can afford at
this size: the masses of sampled query blocks (given the GPU's fp32 LSE), the
complete selection of three heads (coverage is decided per head, so a head's
rows depend on its own masses only; the oracle selects from the GPU's fp32
masses, so indices, counts and Recall must be bit-exact), and the sparse
output of sampled query blocks of those heads (text query blocks included)
on the GPU's index lists."""
import numpy as np
import pytest
import torch

import oracle
import paper_2502_21079_amd as ad
from workloads import LONG, make_qkv
from _helpers import check_lse, check_mass, check_out, csr_rows, f64, sample_blocks

pytestmark = pytest.mark.gpu

HEADS = (0, 11, 23)


@pytest.fixture(scope="module")
def chain():
    w = LONG
    B, H, L, D = w.batch, w.heads, w.seqlen, w.head_dim
    tau = [w.coverage_bp] * H
    q, k, v = make_qkv(w, device="cuda")
    _, lse = ad.dense_attn_lse(q, k, v)
    wsb = ad.block_search_workspace((B, H, L, D), w.block, w.text_start, w.text_len, "coverage", tau)
    ws = torch.empty(wsb, dtype=torch.uint8, device="cuda")
    res = ad.block_search(q, k, lse, block=w.block, text_start=w.text_start, text_len=w.text_len,
                          mode="coverage", head_param_bp=tau, workspace=ws)
    out, lse_m = ad.block_sparse_attn(q, k, v, res.row_ptr, res.col_idx, block=w.block,
                                      text_start=w.text_start, text_len=w.text_len)
    torch.cuda.synchronize()
    return w, q, k, v, lse, res, out, lse_m


def test_chain_masses_sampled(chain):
    w, q, k, _, lse, res, _, _ = chain
    nb = w.nblocks
    for h in HEADS:
        for p in sample_blocks(nb, 2, seed=900 + h, always=(0, 2)):
            rows = np.arange(p * w.block, min((p + 1) * w.block, w.seqlen))
            idx = torch.as_tensor(rows, device="cuda")
            ref = oracle.block_mass_rows(f64(q[0, h, idx]), f64(k[0, h]), f64(lse[0, h, idx]),
                                         w.scale, w.block)
            check_mass(res.block_mass[0, h, p], ref, f"h{h} p{p}")


def test_chain_selection_bit_exact(chain):
    w, _, _, _, _, res, _, _ = chain
    nb = w.nblocks
    rp, ci = csr_rows(res.row_ptr, res.col_idx)
    W = res.block_mass.cpu().numpy()
    for h in HEADS:
        sel = oracle.select_blocks(W[:, h:h + 1], w.seqlen, w.block, w.text_start, w.text_len,
                                   "coverage", [w.coverage_bp])
        lo, hi = rp[h * nb], rp[(h + 1) * nb]
        assert np.array_equal(rp[h * nb:(h + 1) * nb + 1] - lo, sel["row_ptr"]), f"h{h}: row lengths"
        assert np.array_equal(ci[lo:hi], sel["col_idx"]), f"h{h}: indices"
        assert int(res.head_k[0, h]) == int(sel["head_k"][0, 0]), f"h{h}: count"
        assert res.head_recall[0, h].cpu().numpy() == sel["head_recall"][0, 0], f"h{h}: Recall"
        assert float(sel["head_recall"][0, 0]) >= w.coverage_bp / 10000


def test_chain_sparse_output_sampled(chain):
    w, q, k, v, _, res, out, lse_m = chain
    nb = w.nblocks
    rp, ci = csr_rows(res.row_ptr, res.col_idx)
    for h in HEADS:
        blocks = sample_blocks(nb, 4, seed=950 + h, always=(0, 1, 2))
        o_ref, l_ref = oracle.block_sparse_attention(f64(q[0, h]), f64(k[0, h]), f64(v[0, h]),
                                                     rp[h * nb:(h + 1) * nb + 1], ci, w.scale,
                                                     w.block, qblocks=blocks)
        rows = np.concatenate([np.arange(p * w.block, min((p + 1) * w.block, w.seqlen))
                               for p in blocks])
        idx = torch.as_tensor(rows, device="cuda")
        check_out(out[0, h, idx], o_ref, f"h{h}")
        check_lse(lse_m[0, h, idx], l_ref, f"h{h}")
