"""GPU parity at the largest problems the library accepts, against the oracle
on sampled rows.

- Block-sparse attention (Sec. 4.1) at the largest head: L * D just under
  2^30 elements, so a head's K and V reach 2^31 bytes less 27 KB and every
  in-kernel byte offset sits near the top of its 32-bit range.  Rows keep the
  text blocks, their own block, one block spread over the whole sequence and
  the ragged last block (20 rows).
- Dense attention + LSE, the block masses and the selection (Sec. 2.2, 4.1,
  4.3) at the most key blocks a search takes (8,192 at block 128, L just
  over one million tokens, the last block ragged).
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2502_21079_amd as ad
from workloads import Workload, make_qkv, text_blocks
from _helpers import check_lse, check_mass, check_out, f64

pytestmark = pytest.mark.gpu

# 256 text tokens + 32 frames of 262,133 patches (the last frame 12 tokens
# short): 65,536 blocks of 128, the last one 20 rows.
MAX_HEAD = Workload("max_head_L8388500_H1_d128_b128", 1, 1, 128, 8388500, 256, 32, 262133, 128,
                    seed=21)
# 256 text tokens + 32 frames of 32,758 patches: 8,192 blocks of 128, the last
# one 52 rows.
MAX_BLOCKS = Workload("max_blocks_L1048500_H1_d128_b128", 1, 1, 128, 1048500, 256, 32, 32758, 128,
                      seed=22)


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


def test_sparse_at_largest_head():
    w = MAX_HEAD
    L, blk = w.seqlen, w.block
    assert L * w.head_dim < 2 ** 30 and L * w.head_dim * 2 > 2 ** 31 - 32768
    nb = w.nblocks
    assert nb == 65536 and L - (nb - 1) * blk == 20
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


def test_dense_mass_and_selection_at_most_blocks():
    w = MAX_BLOCKS
    L, blk = w.seqlen, w.block
    nb = w.nblocks
    assert nb == 8192 and L - (nb - 1) * blk == 52
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

    # each row of masses from the fresh LSE sums to the row's query count
    sums = res.block_mass[0, 0].double().sum(-1).cpu().numpy()
    expect = np.full(nb, float(blk))
    expect[-1] = L - (nb - 1) * blk
    np.testing.assert_allclose(sums, expect, rtol=1e-3)

    # dense output, LSE and masses of sampled query blocks against the oracle
    print(f"[max] {w.name}: oracle on sampled query blocks", flush=True)
    kh, vh = f64(k[0, 0]), f64(v[0, 0])
    for p in (0, 2, 4000, nb - 2, nb - 1):
        qr = _rows(p, blk, L)
        qi = torch.as_tensor(qr, device="cuda")
        qh = f64(q[0, 0, qi])
        o_ref, l_ref = oracle.dense_attention(qh, kh, vh, w.scale)
        check_out(out[0, 0, qi], o_ref, f"dense, query block {p}")
        check_lse(lse[0, 0, qi], l_ref, f"dense, query block {p}")
        m_ref = oracle.block_mass_rows(qh, kh, l_ref, w.scale, blk)
        check_mass(res.block_mass[0, 0, p], m_ref, f"masses, query block {p}")
    del kh, vh

    # selection from the GPU's own masses: bit-exact on sampled rows (TOPK
    # rows are independent given the count)
    rpn = res.row_ptr.cpu().numpy().astype(np.int64)
    assert rpn[0] == 0 and np.all(np.diff(rpn) == np.where(np.isin(np.arange(nb), tb), nb, kk))
    ci = res.col_idx[: int(rpn[-1])].cpu().numpy()
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
