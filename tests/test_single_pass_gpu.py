"""The single-pass online search (Algorithm 1 with one pass over Q K^T: the
attention pass adds its own exponentials per key block, and the masses of the
fresh LSE follow from those sums once each row's LSE is known) against the
oracle.

Its attention output and LSE come from the same instructions as the dense
kernel's, so they must equal adaspa_dense_attn_lse's bit for bit.  Its block
masses are the same fp32 sums as the two-pass search's in another order, so
they are checked against the oracle's (within 1e-3 relative, every row at
small sizes, sampled query blocks at larger ones) and against the two-pass
search's (within the bf16 rounding of the weights behind its LSE).  The selection must equal the oracle's selection of the same fp32
masses bit for bit.  Shapes cover both block sizes and head dimensions,
ragged lengths (a last block of 128 that holds one full tile and no ragged
tile, a ragged tile after an odd and after an even number of full tiles),
two batch elements, the softmax extremes and degenerate lengths."""
import numpy as np
import pytest
import torch

import oracle
import paper_2502_21079_amd as ad
from workloads import EXTREME_KINDS, LONG, MODERATE, TINY, make_extreme_qkv, make_qkv
from _helpers import MASS_ABS_FLOOR, check_mass, f64, sample_blocks

pytestmark = pytest.mark.gpu

SHAPES = [
    TINY,                                                                          # d 64, block 64, L 2048
    TINY.replace(head_dim=128, block=128, seqlen=1000, patches=234),              # 15 tiles + ragged tile
    TINY.replace(head_dim=128, block=128, seqlen=960, patches=224),               # 15 tiles, last block = 1 tile
    TINY.replace(head_dim=64, block=128, seqlen=1050, patches=247),               # 16 tiles + ragged tile
    TINY.replace(head_dim=128, block=64, seqlen=777, frames=5, patches=178),      # ragged block 64
    TINY.replace(head_dim=64, block=128, seqlen=300, patches=59),                 # one tile of 256 rows + 44
    TINY.replace(batch=2, heads=3, head_dim=128, block=64, seqlen=1000, patches=234),
    MODERATE.replace(heads=3),                                                     # d 64, block 128, NB 140
    LONG.replace(name="slice_L17456_H2_d128_b64", heads=2, frames=5, seqlen=256 + 5 * 3440,
                 block=64),                                                        # NB 273
]


def _params(mode, H):
    if mode == "coverage":
        return [9000 - 500 * (h % 3) for h in range(H)]
    if mode == "topk":
        return [1000 + 1500 * (h % 3) for h in range(H)]
    return None


def _compare_selection(res, sel):
    rp = res.row_ptr.cpu().numpy().astype(np.int64)
    ci = res.col_idx[: int(rp[-1])].cpu().numpy()
    assert np.array_equal(rp, sel["row_ptr"]), "row_ptr differs"
    assert np.array_equal(ci, sel["col_idx"]), "col_idx differs"
    assert np.array_equal(res.head_k.cpu().numpy(), sel["head_k"])
    assert np.array_equal(res.head_recall.cpu().numpy(), sel["head_recall"])


def _oracle_masses(q, k, v, b, h, scale, block, blocks):
    """Oracle masses of the listed query blocks (rows of W) of head (b, h),
    from the oracle's own fp64 LSE of those rows."""
    L = q.shape[2]
    kh, vh = f64(k[b, h]), f64(v[b, h])
    out = []
    for p in blocks:
        qr = f64(q[b, h, p * block:min((p + 1) * block, L)])
        _, l_ref = oracle.dense_attention(qr, kh, vh, scale)
        out.append(oracle.block_mass_rows(qr, kh, l_ref, scale, block))
    return np.stack(out)


def _check_against_two_pass(res, q, k, lse, w, mode, params):
    """The two-pass search from the stored LSE: the same sums in another fp32
    order, normalised by the LSE of the rounded weights instead of the
    unrounded row sum.  Those two row sums differ by at most the weights'
    bf16 rounding, 2^-9 of the sum, so the masses agree within that plus
    fp32 noise."""
    two = ad.block_search(q, k, lse, block=w.block, text_start=w.text_start, text_len=w.text_len,
                          mode=mode, head_param_bp=params, base_sparsity_bp=9000)
    torch.cuda.synchronize()
    a, b = f64(res.block_mass), f64(two.block_mass)
    rel = np.abs(a - b) / (np.abs(b) + MASS_ABS_FLOOR)
    assert rel.max() <= 2 ** -9 + 2e-4, f"single pass against two-pass masses: max rel {rel.max():.3e}"


@pytest.mark.parametrize("case", range(len(SHAPES)))
@pytest.mark.parametrize("mode", ["coverage", "topk", "hierarchical"])
def test_single_pass_against_oracle(case, mode):
    w = SHAPES[case]
    print(f"[single] {w.name} B{w.batch} H{w.heads} d{w.head_dim} L{w.seqlen} b{w.block} {mode}", flush=True)
    q, k, v = make_qkv(w, device="cuda")
    B, H, L = w.batch, w.heads, w.seqlen
    params = _params(mode, H)
    out, lse, res = ad.single_pass_online_search(q, k, v, block=w.block, text_start=w.text_start,
                                                 text_len=w.text_len, mode=mode, head_param_bp=params,
                                                 base_sparsity_bp=9000)
    od, ld = ad.dense_attn_lse(q, k, v)
    torch.cuda.synchronize()
    assert torch.equal(out, od) and torch.equal(lse, ld)
    nb = w.nblocks
    for b in range(B):
        for h in range(H):
            blocks = list(range(nb)) if L <= 2048 else sample_blocks(nb, 4, seed=L + 31 * h, always=(0, 1))
            ref = _oracle_masses(q, k, v, b, h, w.scale, w.block, blocks)
            check_mass(res.block_mass[b, h, blocks], ref, f"{w.name} b{b} h{h}")
    sums = res.block_mass.double().sum(-1).cpu().numpy()
    rows = np.minimum(w.block, L - np.arange(nb) * w.block).astype(np.float64)
    np.testing.assert_allclose(sums, np.broadcast_to(rows, sums.shape), rtol=1e-3)
    sel = oracle.select_blocks(res.block_mass.cpu().numpy(), L, w.block, w.text_start, w.text_len, mode,
                               params if params is not None else [0] * H, base_sparsity_bp=9000)
    _compare_selection(res, sel)
    _check_against_two_pass(res, q, k, lse, w, mode, params)


@pytest.mark.parametrize("kind", EXTREME_KINDS)
@pytest.mark.parametrize("D,block,L", [(64, 64, 1000), (128, 128, 777), (128, 128, 1000)])
def test_single_pass_extreme_scores(kind, D, block, L):
    """Scores far below the fp32 exponent range, row maxima that rise on every
    tile (the reference moves inside a key block) and large random jumps (rows
    redone on the exact path): masses against the oracle, output and LSE equal
    to the dense kernel's."""
    (q, k, v), scale = make_extreme_qkv(kind, heads=2, seqlen=L, head_dim=D, device="cuda")
    out, lse, res = ad.single_pass_online_search(q, k, v, block=block, text_start=0, text_len=0,
                                                 mode="topk", head_param_bp=[2000, 2000], scale=scale)
    od, ld = ad.dense_attn_lse(q, k, v, scale=scale)
    torch.cuda.synchronize()
    assert torch.equal(out, od) and torch.equal(lse, ld)
    nb = (L + block - 1) // block
    for h in range(2):
        ref = _oracle_masses(q, k, v, 0, h, scale, block, range(nb))
        check_mass(res.block_mass[0, h], ref, f"{kind} h{h}")


@pytest.mark.parametrize("D,block,L", [(64, 64, 1), (128, 64, 64), (128, 128, 130), (64, 128, 64)])
def test_single_pass_degenerate_lengths(D, block, L):
    w = TINY.replace(head_dim=D, block=block, seqlen=L, text_len=0, patches=max(1, L))
    q, k, v = make_qkv(w, device="cuda")
    out, lse, res = ad.single_pass_online_search(q, k, v, block=block, text_start=0, text_len=0,
                                                 mode="coverage", head_param_bp=[9000] * w.heads)
    od, ld = ad.dense_attn_lse(q, k, v)
    torch.cuda.synchronize()
    assert torch.equal(out, od) and torch.equal(lse, ld)
    nb = w.nblocks
    for h in range(w.heads):
        ref = _oracle_masses(q, k, v, 0, h, w.scale, block, range(nb))
        check_mass(res.block_mass[0, h], ref, f"L{L} h{h}")


@pytest.mark.parametrize("block", [128, 64])
def test_single_pass_long_sampled(block):
    """The 110K-token shape (three heads): sampled query blocks against the
    oracle, every mass row summing to its query count, the selection equal
    to the oracle's of the same masses on every row."""
    w = LONG.replace(block=block)
    q, k, v = make_qkv(w, device="cuda", heads=range(3))
    H, L, nb = 3, w.seqlen, w.nblocks
    tau = [9000] * H
    out, lse, res = ad.single_pass_online_search(q, k, v, block=block, text_start=0, text_len=w.text_len,
                                                 mode="coverage", head_param_bp=tau)
    od, ld = ad.dense_attn_lse(q, k, v)
    torch.cuda.synchronize()
    assert torch.equal(out, od) and torch.equal(lse, ld)
    sums = res.block_mass[0].double().sum(-1).cpu().numpy()
    np.testing.assert_allclose(sums, float(block), rtol=1e-3)
    for h in range(H):
        blocks = sample_blocks(nb, 3, seed=700 + h, always=(0, nb - 1))
        ref = _oracle_masses(q, k, v, 0, h, w.scale, block, blocks)
        check_mass(res.block_mass[0, h, blocks], ref, f"110K b{block} h{h}")
    sel = oracle.select_blocks(res.block_mass.cpu().numpy(), L, block, 0, w.text_len, "coverage", tau)
    _compare_selection(res, sel)


def test_single_pass_without_lse_output():
    """The LSE output is optional: the masses come from the kernel's own row
    sums either way, so every output is the same bit for bit."""
    w = TINY.replace(head_dim=128, block=128, seqlen=1000, patches=234)
    q, k, v = make_qkv(w, device="cuda")
    kw = dict(block=w.block, text_start=w.text_start, text_len=w.text_len, mode="coverage",
              head_param_bp=[9000] * w.heads)
    o1, l1, r1 = ad.single_pass_online_search(q, k, v, **kw)
    o2, l2, r2 = ad.single_pass_online_search(q, k, v, want_lse=False, **kw)
    torch.cuda.synchronize()
    assert l2 is None and torch.equal(o1, o2)
    assert torch.equal(r1.block_mass, r2.block_mass) and torch.equal(r1.row_ptr, r2.row_ptr)
    n = r1.nnz()
    assert torch.equal(r1.col_idx[:n], r2.col_idx[:n]) and torch.equal(r1.head_recall, r2.head_recall)


@pytest.mark.parametrize("mode", ["coverage", "hierarchical"])
def test_single_pass_in_head_groups(mode):
    """A workspace between the least and the full size runs the (batch, head)
    pairs in groups: one pair at a time, four at a time (the last group
    partial) and all at once give the same outputs bit for bit, also where
    the selection ranks heads against each other (hierarchical).  A
    workspace on another device is refused."""
    w = TINY.replace(batch=2, heads=3, head_dim=128, block=64, seqlen=1000, patches=234)
    q, k, v = make_qkv(w, device="cuda")
    H = w.heads
    params = None if mode == "hierarchical" else [9000, 8000, 7000]
    kw = dict(block=w.block, text_start=w.text_start, text_len=w.text_len, mode=mode, head_param_bp=params,
              base_sparsity_bp=9000)
    shape = tuple(q.shape)
    full = ad.single_pass_online_search_workspace(shape, w.block, w.text_start, w.text_len, mode, params,
                                                  base_sparsity_bp=9000)
    least = ad.single_pass_online_search_min_workspace(shape, w.block, w.text_start, w.text_len, mode, params,
                                                       base_sparsity_bp=9000)
    # the search's workspace, then g pairs' per-row masses and row LSEs, each
    # rounded up to 256 bytes
    L, nb = w.seqlen, w.nblocks
    rnd = lambda x: (x + 255) // 256 * 256
    base = least - rnd(nb * L * 4) - rnd(L * 4)
    assert full == base + rnd(6 * nb * L * 4) + rnd(6 * L * 4)
    four = base + rnd(4 * nb * L * 4) + rnd(4 * L * 4)
    outs = []
    for size in (least, four, full):
        # a workspace of any dtype counts in bytes: the middle one as int32
        ws = (torch.empty(-(-size // 4), dtype=torch.int32, device="cuda") if size not in (least, full)
              else torch.empty(size, dtype=torch.uint8, device="cuda"))
        outs.append(ad.single_pass_online_search(q, k, v, workspace=ws, **kw))
    torch.cuda.synchronize()
    (o0, l0, r0) = outs[-1]
    for o, l, r in outs[:-1]:
        assert torch.equal(o, o0) and torch.equal(l, l0)
        assert torch.equal(r.block_mass, r0.block_mass) and torch.equal(r.row_ptr, r0.row_ptr)
        n = r0.nnz()
        assert torch.equal(r.col_idx[:n], r0.col_idx[:n])
        assert torch.equal(r.head_k, r0.head_k) and torch.equal(r.head_recall, r0.head_recall)
    with pytest.raises(ad.AdaspaError):
        ad.single_pass_online_search(q, k, v, workspace=torch.empty(full, dtype=torch.uint8), **kw)
