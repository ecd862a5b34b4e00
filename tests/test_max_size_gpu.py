"""GPU parity at the largest problems the library accepts, against the oracle
on sampled rows.

- Block-sparse attention (Sec. 4.1) at the largest head, d = 64 and 128:
  L * D just under 2^30 elements, so a head's K and V each come within 28 KB
  of 2^31 bytes and every in-kernel byte offset sits near the top of its
  32-bit range.  Rows keep the text blocks, their own block, one block spread
  over the whole sequence and the ragged last block.
- Dense attention + LSE, the block masses, the selection and block-sparse
  attention on the selected pattern (Sec. 2.2, 4.1, 4.3) at the most key
  blocks a search takes (8,192), at block 128 (L just over one million
  tokens) and block 64 (the block-64 kernel's map of one row's key blocks is
  then full), the last block ragged; the single-pass search at the same
  sizes (34 GB and 17 GB of per-row block masses): its output and LSE equal
  to the dense kernel's, its masses against the oracle.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2502_21079_amd as ad
from workloads import Workload, make_qkv, text_blocks
from _helpers import check_lse, check_mass, check_out, f64

pytestmark = pytest.mark.gpu

# 256 text tokens + 32 frames (the last one a few tokens short).  d = 128:
# 65,536 blocks of 128, the last one 20 rows; d = 64: 131,071 blocks, the
# last one 40 rows.
MAX_HEAD = {
    128: Workload("max_head_L8388500_H1_d128_b128", 1, 1, 128, 8388500, 256, 32, 262133, 128, seed=21),
    64: Workload("max_head_L16777000_H1_d64_b128", 1, 1, 64, 16777000, 256, 32, 524274, 128, seed=23),
}
# 8,192 key blocks: block 128 (256 text tokens + 32 frames of 32,758 patches,
# the last block 52 rows) and block 64 (32 frames of 16,375 patches, the last
# block 26 rows).
MAX_BLOCKS = {
    128: Workload("max_blocks_L1048500_H1_d128_b128", 1, 1, 128, 1048500, 256, 32, 32758, 128, seed=22),
    64: Workload("max_blocks_L524250_H1_d128_b64", 1, 1, 128, 524250, 256, 32, 16375, 64, seed=24),
}


def _rows(p, block, L):
    return np.arange(p * block, min((p + 1) * block, L))


def _key_rows(kept, block, L):
    return np.concatenate([_rows(int(c), block, L) for c in kept])


def _spread_pattern(nb, n_text):
    """Every row keeps the text blocks, block p itself, block (7919 p + 13) mod
    nb and the last block; text rows keep the text blocks, the next block and
    the last.  Indices ascending, duplicates removed."""
    p = np.arange(nb, dtype=np.int64)
    cand = np.stack([np.zeros(nb, np.int64), np.ones(nb, np.int64), np.maximum(p, n_text),
                     (7919 * p + 13) % nb, np.full(nb, nb - 1)], axis=1)
    cand[:n_text, 3] = n_text           # text rows: the first video block instead
    cand.sort(axis=1)
    keep = np.ones_like(cand, dtype=bool)
    keep[:, 1:] = cand[:, 1:] != cand[:, :-1]
    counts = keep.sum(axis=1)
    row_ptr = np.zeros(nb + 1, np.int64)
    row_ptr[1:] = np.cumsum(counts)
    return row_ptr.astype(np.int32), cand[keep].astype(np.int32)


@pytest.mark.parametrize("D", [128, 64])
def test_sparse_at_largest_head(D):
    w = MAX_HEAD[D]
    L, blk = w.seqlen, w.block
    assert L * D < 2 ** 30 and L * D * 2 > 2 ** 31 - 28 * 1024
    nb = w.nblocks
    assert (nb, L - (nb - 1) * blk) == ({128: (65536, 20), 64: (131071, 40)}[D])
    print(f"[max] {w.name}: inputs", flush=True)
    q, k, v = make_qkv(w, device="cuda")
    tb = text_blocks(L, blk, w.text_start, w.text_len)
    rp, ci = _spread_pattern(nb, len(tb))
    print(f"[max] {w.name}: block-sparse attention, {len(ci)} entries", flush=True)
    out, lse = ad.block_sparse_attn(q, k, v, torch.from_numpy(rp).cuda(), torch.from_numpy(ci).cuda(),
                                    block=blk, text_start=w.text_start, text_len=w.text_len)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(lse).all()) and bool(torch.isfinite(out).all())
    for p in (0, 1, 2, 3, nb // 2, nb - 3, nb - 2, nb - 1):
        kept = ci[rp[p]:rp[p + 1]]
        qr, kr = _rows(p, blk, L), _key_rows(kept, blk, L)
        qi, ki = torch.as_tensor(qr, device="cuda"), torch.as_tensor(kr, device="cuda")
        # masked attention of the row over its kept keys: the mask of the
        # gathered key rows keeps all of them
        o_ref, l_ref = oracle.masked_attention(f64(q[0, 0, qi]), f64(k[0, 0, ki]), f64(v[0, 0, ki]),
                                               np.ones(len(kr), bool), w.scale)
        check_out(out[0, 0, qi], o_ref, f"query block {p}")
        check_lse(lse[0, 0, qi], l_ref, f"query block {p}")


@pytest.mark.parametrize("block", [128, 64])
def test_dense_search_sparse_at_most_blocks(block):
    w = MAX_BLOCKS[block]
    L, blk = w.seqlen, w.block
    nb = w.nblocks
    assert nb == 8192 and L - (nb - 1) * blk == {128: 52, 64: 26}[block]
    print(f"[max] {w.name}: inputs", flush=True)
    q, k, v = make_qkv(w, device="cuda")
    print(f"[max] {w.name}: dense attention + LSE", flush=True)
    out, lse = ad.dense_attn_lse(q, k, v)
    print(f"[max] {w.name}: search, TOPK 0.5%", flush=True)
    res = ad.block_search(q, k, lse, block=blk, text_start=w.text_start, text_len=w.text_len,
                          mode="topk", head_param_bp=[50])
    torch.cuda.synchronize()
    tb = text_blocks(L, blk, w.text_start, w.text_len)
    kk = oracle.topk_count(50, nb, len(tb))
    assert kk == 41 and int(res.head_k[0, 0]) == kk
    print(f"[max] {w.name}: single-pass search", flush=True)
    o1, l1, r1 = ad.single_pass_online_search(q, k, v, block=blk, text_start=w.text_start,
                                              text_len=w.text_len, mode="topk", head_param_bp=[50])
    torch.cuda.synchronize()
    assert torch.equal(o1, out) and torch.equal(l1, lse)
    sp_sums = r1.block_mass[0, 0].double().sum(-1).cpu().numpy()
    sp_mass = r1.block_mass[0, 0].cpu()              # checked against the oracle below
    del o1, l1, r1
    torch.cuda.empty_cache()
    print(f"[max] {w.name}: block-sparse attention on the selected pattern", flush=True)
    sp_out, sp_lse = ad.block_sparse_attn(q, k, v, res.row_ptr, res.col_idx, block=blk,
                                          text_start=w.text_start, text_len=w.text_len)
    torch.cuda.synchronize()

    # each row of masses from the fresh LSE sums to the row's query count
    sums = res.block_mass[0, 0].double().sum(-1).cpu().numpy()
    expect = np.full(nb, float(blk))
    expect[-1] = L - (nb - 1) * blk
    np.testing.assert_allclose(sums, expect, rtol=1e-3)
    np.testing.assert_allclose(sp_sums, expect, rtol=1e-3)

    # dense output, LSE and masses of sampled query blocks against the oracle,
    # and block-sparse attention of those blocks over the keys they keep
    print(f"[max] {w.name}: oracle on sampled query blocks", flush=True)
    kh, vh = f64(k[0, 0]), f64(v[0, 0])
    rpn = res.row_ptr.cpu().numpy().astype(np.int64)
    ci = res.col_idx[: int(rpn[-1])].cpu().numpy()
    for p in (0, len(tb), len(tb) + 1, 4000, 4001, nb - 2, nb - 1):
        qr = _rows(p, blk, L)
        qi = torch.as_tensor(qr, device="cuda")
        qh = f64(q[0, 0, qi])
        o_ref, l_ref = oracle.dense_attention(qh, kh, vh, w.scale)
        check_out(out[0, 0, qi], o_ref, f"dense, query block {p}")
        check_lse(lse[0, 0, qi], l_ref, f"dense, query block {p}")
        m_ref = oracle.block_mass_rows(qh, kh, l_ref, w.scale, blk)
        check_mass(res.block_mass[0, 0, p], m_ref, f"masses, query block {p}")
        check_mass(sp_mass[p], m_ref, f"single-pass masses, query block {p}")
        kr = _key_rows(ci[rpn[p]:rpn[p + 1]], blk, L)
        o_ref, l_ref = oracle.masked_attention(qh, kh[kr], vh[kr], np.ones(len(kr), bool), w.scale)
        check_out(sp_out[0, 0, qi], o_ref, f"sparse, query block {p}")
        check_lse(sp_lse[0, 0, qi], l_ref, f"sparse, query block {p}")
    del kh, vh

    # selection from the GPU's own masses: bit-exact on sampled rows (TOPK
    # rows are independent given the count)
    assert rpn[0] == 0 and np.all(np.diff(rpn) == np.where(np.isin(np.arange(nb), tb), nb, kk))
    rng = np.random.default_rng(5)
    sample = sorted(set(tb) | {2, nb - 2, nb - 1} | set(rng.choice(nb, 40, replace=False).tolist()))
    for p in sample:
        got = ci[rpn[p]:rpn[p + 1]]
        if p in tb:
            assert np.array_equal(got, np.arange(nb)), p
            continue
        row = res.block_mass[0, 0, p].cpu().numpy()
        exp = sorted(oracle.row_order(row, set(tb))[:kk])
        assert np.array_equal(got, np.asarray(exp)), p
