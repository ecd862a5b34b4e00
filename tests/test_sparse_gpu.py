"""GPU parity of adaspa_block_sparse_attn (Sec. 4.1 blockified sparse
attention) against the fp64 oracle, on seeded block patterns."""
import numpy as np
import pytest
import torch

import oracle
import paper_2502_21079_amd as ad
from workloads import LONG, MODERATE, TINY, make_qkv, random_block_lists, text_blocks
from _helpers import check_lse, check_out, f64, sample_blocks

pytestmark = pytest.mark.gpu


def _all_blocks(B, H, nb):
    row_ptr = torch.arange(B * H * nb + 1, dtype=torch.int32) * nb
    col_idx = torch.arange(nb, dtype=torch.int32).repeat(B * H * nb)
    return row_ptr.cuda(), col_idx.cuda()


@pytest.mark.parametrize("D,block,L", [(64, 64, 2048), (128, 128, 1000), (128, 64, 777), (64, 128, 4096)])
def test_all_blocks_equals_dense_bitwise(D, block, L):
    """P1 on the GPU: keeping every block reproduces the dense kernel bit for bit."""
    w = TINY.replace(head_dim=D, block=block, seqlen=L, patches=(L - 64 + 3) // 4)
    q, k, v = make_qkv(w, device="cuda")
    od, ld = ad.dense_attn_lse(q, k, v)
    rp, ci = _all_blocks(1, w.heads, w.nblocks)
    os_, ls = ad.block_sparse_attn(q, k, v, rp, ci, block=block)
    torch.cuda.synchronize()
    assert torch.equal(od, os_) and torch.equal(ld, ls)


def _pattern(nrows, nb, k, seed, always):
    return random_block_lists(nrows, nb, k, seed, always=always)


@pytest.mark.parametrize("D,block,L,k", [(64, 64, 2048, 6), (128, 128, 1000, 3), (128, 64, 777, 4),
                                         (64, 128, 2048, 1)])
def test_sparse_matches_oracle(D, block, L, k):
    w = TINY.replace(head_dim=D, block=block, seqlen=L, patches=(L - 64 + 3) // 4)
    q, k_, v = make_qkv(w, device="cuda")
    nb = w.nblocks
    tb = text_blocks(L, block, 0, 64)
    rp, ci = _pattern(w.heads * nb, nb, k, seed=L + k, always=tb)
    out, lse = ad.block_sparse_attn(q, k_, v, rp.cuda(), ci.cuda(), block=block)
    torch.cuda.synchronize()
    rpn, cin = rp.numpy(), ci.numpy()
    for h in range(w.heads):
        o_ref, l_ref = oracle.block_sparse_attention(f64(q[0, h]), f64(k_[0, h]), f64(v[0, h]),
                                                     rpn[h * nb:(h + 1) * nb + 1], cin, w.scale, block)
        check_out(out[0, h], o_ref, f"h{h}")
        check_lse(lse[0, h], l_ref)


def test_sparse_long_sampled():
    """The 110K-token shape at about 20% density, sampled query blocks."""
    w = LONG
    q, k, v = make_qkv(w, device="cuda")
    nb = w.nblocks
    kk = oracle.topk_count(2000, nb, 2)
    rp, ci = _pattern(w.heads * nb, nb, kk, seed=5, always=[0, 1])
    out, lse = ad.block_sparse_attn(q, k, v, rp.cuda(), ci.cuda(), block=w.block)
    torch.cuda.synchronize()
    rpn, cin = rp.numpy(), ci.numpy()
    for h in (0, 13, 23):
        blocks = sample_blocks(nb, 3, seed=400 + h, always=(0, 2))
        o_ref, l_ref = oracle.block_sparse_attention(f64(q[0, h]), f64(k[0, h]), f64(v[0, h]),
                                                     rpn[h * nb:(h + 1) * nb + 1], cin, w.scale,
                                                     w.block, qblocks=blocks)
        rows = np.concatenate([np.arange(p * 128, min((p + 1) * 128, w.seqlen)) for p in blocks])
        idx = torch.as_tensor(rows, device="cuda")
        check_out(out[0, h, idx], o_ref, f"h{h}")
        check_lse(lse[0, h, idx], l_ref)


def test_empty_rows_and_skipped_indices():
    """A row with no kept block gives zeros and LSE -inf; entries outside
    [0, NB) are skipped by the kernel's own bounds check."""
    w = TINY.replace(seqlen=512, patches=112)
    q, k, v = make_qkv(w, device="cuda")
    nb = 8
    rows = []
    for r in range(w.heads * nb):
        rows.append([] if r % 3 == 0 else [r % nb])
    rows[1] = [-1, 2, 99]           # out-of-range entries around a valid one
    row_ptr = torch.tensor([0] + list(np.cumsum([len(x) for x in rows])), dtype=torch.int32)
    col_idx = torch.tensor([c for x in rows for c in x], dtype=torch.int32)
    out, lse = ad.block_sparse_attn(q, k, v, row_ptr.cuda(), col_idx.cuda(), block=64)
    torch.cuda.synchronize()
    for r, kept in enumerate(rows):
        h, p = divmod(r, nb)
        valid = [c for c in kept if 0 <= c < nb]
        mask = oracle.key_mask_from_blocks(valid, 512, 64)
        o_ref, l_ref = oracle.masked_attention(f64(q[0, h, p * 64:(p + 1) * 64]), f64(k[0, h]),
                                               f64(v[0, h]), mask, w.scale)
        check_out(out[0, h, p * 64:(p + 1) * 64], o_ref, f"row {r}")
        check_lse(lse[0, h, p * 64:(p + 1) * 64], l_ref)
        if not valid:
            assert torch.all(out[0, h, p * 64:(p + 1) * 64] == 0)


def test_sparse_deterministic():
    w = TINY.replace(head_dim=128, block=128)
    q, k, v = make_qkv(w, device="cuda")
    rp, ci = _pattern(w.heads * w.nblocks, w.nblocks, 5, seed=1, always=[0])
    rp, ci = rp.cuda(), ci.cuda()
    o1, l1 = ad.block_sparse_attn(q, k, v, rp, ci, block=128)
    o2, l2 = ad.block_sparse_attn(q, k, v, rp, ci, block=128)
    torch.cuda.synchronize()
    assert torch.equal(o1, o2) and torch.equal(l1, l2)


@pytest.mark.parametrize("block", [64, 128])
@pytest.mark.parametrize("text", [(0, 128), (512, 200), (1664, 384), (0, 0)])
def test_text_first_order_covers_every_row(text, block):
    """The work order that starts text query blocks first is a bijection:
    every (head, query block) row is computed, for text at the start, in the
    middle (unaligned), at the end and absent, with more heads than XCDs."""
    t0, tl = text
    w = TINY.replace(heads=9, block=block)
    q, k, v = make_qkv(w, device="cuda")
    nb = w.nblocks
    tb = text_blocks(w.seqlen, w.block, t0, tl) if tl > 0 else []
    # text query blocks keep every block (as the selection emits them); others keep 3
    lists = []
    g = np.random.default_rng(7)
    for r in range(w.heads * nb):
        p = r % nb
        if p in tb:
            lists.append(list(range(nb)))
        else:
            lists.append(sorted(set(tb) | set(g.choice(nb, 3, replace=False).tolist())))
    rp = torch.tensor([0] + list(np.cumsum([len(x) for x in lists])), dtype=torch.int32)
    ci = torch.tensor([c for x in lists for c in x], dtype=torch.int32)
    out, lse = ad.block_sparse_attn(q, k, v, rp.cuda(), ci.cuda(), block=w.block, text_start=t0,
                                    text_len=tl)
    torch.cuda.synchronize()
    rpn, cin = rp.numpy(), ci.numpy()
    for h in range(w.heads):
        o_ref, l_ref = oracle.block_sparse_attention(f64(q[0, h]), f64(k[0, h]), f64(v[0, h]),
                                                     rpn[h * nb:(h + 1) * nb + 1], cin, w.scale, w.block)
        check_out(out[0, h], o_ref, f"h{h}")
        check_lse(lse[0, h], l_ref)


def test_unordered_rows_take_the_masked_path():
    """Block 64 pairs two query blocks and merges their lists, which needs
    ascending lists; a row given out of order (or with a repeat) is done tile
    by tile instead, with the same result."""
    w = TINY.replace(seqlen=640, patches=144)
    q, k, v = make_qkv(w, device="cuda")
    nb = w.nblocks
    g = np.random.default_rng(11)
    lists = [sorted(g.choice(nb, 3, replace=False).tolist()) for _ in range(w.heads * nb)]
    lists[2] = [7, 1, 4]               # descending / unordered
    lists[5] = [3, 3]                  # repeat: counted twice, like the per-row kernel
    rp = torch.tensor([0] + list(np.cumsum([len(x) for x in lists])), dtype=torch.int32)
    ci = torch.tensor([c for x in lists for c in x], dtype=torch.int32)
    out, lse = ad.block_sparse_attn(q, k, v, rp.cuda(), ci.cuda(), block=64)
    torch.cuda.synchronize()
    for r, kept in enumerate(lists):
        if r == 5:
            continue                   # a repeated block is not a valid pattern
        h, p = divmod(r, nb)
        mask = oracle.key_mask_from_blocks(kept, w.seqlen, 64)
        o_ref, l_ref = oracle.masked_attention(f64(q[0, h, p * 64:(p + 1) * 64]), f64(k[0, h]),
                                               f64(v[0, h]), mask, w.scale)
        check_out(out[0, h, p * 64:(p + 1) * 64], o_ref, f"row {r}")
        check_lse(lse[0, h, p * 64:(p + 1) * 64], l_ref)


@pytest.mark.parametrize("block", [64, 128])
def test_sparse_work_queue_matches_static_split(block):
    """The queued last tenth of the query blocks only changes which CU runs a
    block: outputs and LSE are bitwise those of the static split, with a
    text range and an item count that do not divide by the eight queues,
    on back-to-back calls that reuse one workspace (each call clears it)."""
    L = 128 * 61 + 40
    w = TINY.replace(head_dim=128, heads=3, block=block, seqlen=L, text_len=200,
                     patches=(L - 200 + 3) // 4)
    q, k, v = make_qkv(w, device="cuda")
    nb = w.nblocks
    tb = text_blocks(L, block, 0, 200)
    rp, ci = _pattern(w.heads * nb, nb, 9, seed=77, always=tb)
    rp, ci = rp.cuda(), ci.cuda()
    txt = dict(text_start=0, text_len=200)
    o0, l0 = ad.block_sparse_attn(q, k, v, rp, ci, block=block, balance=False, **txt)
    ws = torch.empty(ad.block_sparse_attn_workspace(q.shape, block), dtype=torch.uint8, device="cuda")
    for _ in range(3):
        o1, l1 = ad.block_sparse_attn(q, k, v, rp, ci, block=block, workspace=ws, **txt)
        torch.cuda.synchronize()
        assert torch.equal(o0, o1) and torch.equal(l0, l1)


def test_sparse_moderate_sampled():
    """The moderate shape (48 heads, L = 17,920, d = 64, block 128) at about
    20% density with the text sink, sampled query blocks of every sixth head
    (text blocks and the last block always included)."""
    w = MODERATE
    q, k, v = make_qkv(w, device="cuda")
    nb = w.nblocks
    tb = text_blocks(w.seqlen, w.block, w.text_start, w.text_len)
    kk = oracle.topk_count(2000, nb, len(tb))
    rp, ci = _pattern(w.heads * nb, nb, kk, seed=17, always=tb)
    out, lse = ad.block_sparse_attn(q, k, v, rp.cuda(), ci.cuda(), block=w.block,
                                    text_start=w.text_start, text_len=w.text_len)
    torch.cuda.synchronize()
    rpn, cin = rp.numpy(), ci.numpy()
    for h in range(0, w.heads, 6):
        blocks = sample_blocks(nb, 4, seed=600 + h, always=tuple(tb))
        o_ref, l_ref = oracle.block_sparse_attention(f64(q[0, h]), f64(k[0, h]), f64(v[0, h]),
                                                     rpn[h * nb:(h + 1) * nb + 1], cin, w.scale,
                                                     w.block, qblocks=blocks)
        rows = np.concatenate([np.arange(p * w.block, min((p + 1) * w.block, w.seqlen)) for p in blocks])
        idx = torch.as_tensor(rows, device="cuda")
        check_out(out[0, h, idx], o_ref, f"h{h}")
        check_lse(lse[0, h, idx], l_ref)


@pytest.mark.parametrize("bad", [float("nan"), float("inf")])
def test_nonfinite_key_in_a_block_only_the_partner_keeps(bad):
    """Block 64 pairs two query blocks over the union of their lists.  A
    non-finite key in a block that only one of the two keeps must not reach
    the other: its rows match the oracle, which never looks at that block;
    the rows that keep it are non-finite, as in the oracle."""
    w = TINY                                   # 32 blocks of 64
    q, k, v = make_qkv(w, device="cuda")
    nb = w.nblocks
    k[0, :, 20 * 64 + 7, :] = bad              # a key of block 20, both heads
    lists = [[0, 3 * (p % 5) + 1] if p % 2 else sorted({0, 3 * (p % 5) + 1, 9}) for p in range(nb)]
    lists[2] = [0, 5, 20]                      # pair (2, 3): only block 2 keeps block 20
    lists[3] = [0, 5, 9]
    lists[10] = [0, 12]                        # pair (10, 11): only block 11 keeps block 20
    lists[11] = [0, 12, 20, 21]
    all_lists = lists * w.heads
    rp = torch.tensor([0] + list(np.cumsum([len(x) for x in all_lists])), dtype=torch.int32)
    ci = torch.tensor([c for x in all_lists for c in x], dtype=torch.int32)
    out, lse = ad.block_sparse_attn(q, k, v, rp.cuda(), ci.cuda(), block=64)
    torch.cuda.synchronize()
    for h in range(w.heads):
        qh, kh, vh = f64(q[0, h]), f64(k[0, h]), f64(v[0, h])
        for p, kept in enumerate(lists):
            rows = slice(p * 64, (p + 1) * 64)
            if 20 in kept:
                assert not torch.isfinite(out[0, h, rows].float()).all(), (h, p)
                continue
            mask = oracle.key_mask_from_blocks(kept, w.seqlen, 64)
            o_ref, l_ref = oracle.masked_attention(qh[rows], kh, vh, mask, w.scale)
            check_out(out[0, h, rows], o_ref, f"h{h} p{p}")
            check_lse(lse[0, h, rows], l_ref, f"h{h} p{p}")
