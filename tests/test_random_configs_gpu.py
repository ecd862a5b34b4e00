"""Seeded random problem shapes through every entry point, against the oracle.

Each case draws batch, heads, head dim, block size, sequence length (1 to
2,300 tokens, ragged), the text range (absent, first, last or inside) and a
selection mode, then checks on the same seeded inputs:
- dense attention and LSE (Sec. 2.2) against the oracle on every row;
- the two-pass search's masses from the fresh LSE (Sec. 4.1) against the
  oracle's, and its selection bit for bit against the oracle's selection of
  the same fp32 masses (Sec. 4.1-4.3);
- block-sparse attention (Sec. 4.1) on that pattern against the oracle;
- the fused online search equal to the two calls bit for bit, and the
  single-pass search's output and LSE equal to the dense kernel's and its
  masses against the oracle (Algorithm 1).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2502_21079_amd as ad
from workloads import TINY, make_qkv
from _helpers import check_lse, check_mass, check_out, csr_rows, f64

pytestmark = pytest.mark.gpu

N_CASES = 48


def _case(seed):
    g = np.random.default_rng(1000 + seed)
    D = int(g.choice([64, 128]))
    block = int(g.choice([64, 128]))
    L = int(g.integers(1, 2301))
    B, H = int(g.integers(1, 3)), int(g.integers(1, 4))
    where = str(g.choice(["none", "first", "last", "inside"]))
    tl = 0 if where == "none" else int(g.integers(1, max(2, min(L, 300))))
    tl = min(tl, L)
    ts = {"none": 0, "first": 0, "last": L - tl, "inside": int(g.integers(0, L - tl + 1))}[where]
    mode = str(g.choice(["topk", "coverage", "hierarchical"]))
    params = None if mode == "hierarchical" else [int(x) for x in g.integers(0, 10001, size=H)]
    video = L - tl
    frames = 4
    w = TINY.replace(name=f"random{seed}", batch=B, heads=H, head_dim=D, block=block, seqlen=L,
                     text_len=tl, text_first=(where != "last"), frames=frames,
                     patches=max(1, -(-video // frames)), seed=50 + seed)
    return w, ts, mode, params


@pytest.mark.parametrize("seed", range(N_CASES))
def test_random_config_against_oracle(seed):
    w, ts, mode, params = _case(seed)
    B, H, L, D, blk = w.batch, w.heads, w.seqlen, w.head_dim, w.block
    print(f"[random] seed {seed}: B{B} H{H} d{D} L{L} block {blk} text [{ts}, {ts + w.text_len}) {mode}",
          flush=True)
    # The generator lays the text tokens first or last; for text inside the
    # sequence the problem names another range as text (what the kernels
    # treat as text is the range they are given).
    q, k, v = make_qkv(w, device="cuda")
    kw = dict(block=blk, text_start=ts, text_len=w.text_len, mode=mode, head_param_bp=params,
              base_sparsity_bp=9000)
    out, lse = ad.dense_attn_lse(q, k, v)
    res = ad.block_search(q, k, lse, **kw)
    sp_out, sp_lse = ad.block_sparse_attn(q, k, v, res.row_ptr, res.col_idx, block=blk, text_start=ts,
                                          text_len=w.text_len)
    fo, fl, fr = ad.fused_online_search(q, k, v, **kw)
    so, sl, sr = ad.single_pass_online_search(q, k, v, **kw)
    torch.cuda.synchronize()

    nb = w.nblocks
    W = np.zeros((B, H, nb, nb))
    for b in range(B):
        for h in range(H):
            qh, kh, vh = f64(q[b, h]), f64(k[b, h]), f64(v[b, h])
            o_ref, l_ref = oracle.dense_attention(qh, kh, vh, w.scale)
            check_out(out[b, h], o_ref, f"dense b{b} h{h}")
            check_lse(lse[b, h], l_ref, f"dense lse b{b} h{h}")
            W[b, h] = oracle.block_mass(qh, kh, l_ref, w.scale, blk)
            check_mass(res.block_mass[b, h], W[b, h], f"masses b{b} h{h}")
            check_mass(sr.block_mass[b, h], W[b, h], f"single-pass masses b{b} h{h}")
    sel = oracle.select_blocks(res.block_mass.cpu().numpy(), L, blk, ts, w.text_len, mode,
                               params if params is not None else [0] * H, base_sparsity_bp=9000)
    rp, ci = csr_rows(res.row_ptr, res.col_idx)
    assert np.array_equal(rp, sel["row_ptr"]) and np.array_equal(ci, sel["col_idx"])
    assert np.array_equal(res.head_k.cpu().numpy(), sel["head_k"])
    for b in range(B):
        for h in range(H):
            r0 = (b * H + h) * nb
            o_sp, l_sp = oracle.block_sparse_attention(f64(q[b, h]), f64(k[b, h]), f64(v[b, h]),
                                                       sel["row_ptr"][r0:r0 + nb + 1], sel["col_idx"],
                                                       w.scale, blk)
            check_out(sp_out[b, h], o_sp, f"sparse b{b} h{h}")
            check_lse(sp_lse[b, h], l_sp, f"sparse lse b{b} h{h}")
    # Algorithm 1 in one launch: bit for bit the two calls; the single pass:
    # the dense output and LSE bit for bit, its masses checked above
    assert torch.equal(fo, out) and torch.equal(fl, lse) and torch.equal(fr.block_mass, res.block_mass)
    assert torch.equal(fr.row_ptr, res.row_ptr) and torch.equal(fr.col_idx[:res.nnz()], res.col_idx[:res.nnz()])
    assert torch.equal(so, out) and torch.equal(sl, lse)
