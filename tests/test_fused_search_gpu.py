"""The fused online search (Algorithm 1 in one launch: dense attention and
LSE of 256 query rows, then the block masses of the same rows from that
fresh LSE, then the selection) against the two separate calls it fuses, and
against the oracle.

The fused kernel runs both passes with the same rows per wave and lane as
the separate kernels and the same arithmetic, so its outputs must equal
theirs bit for bit: O, LSE, block masses, the CSR lists, head counts and
Recall.  Shapes cover both block sizes and head dimensions, ragged lengths
(the last 256-row tile and the last query block partly past L), two batch
elements and the block-64 slice with 273 key blocks."""
import numpy as np
import pytest
import torch

import oracle
import paper_2502_21079_amd as ad
from workloads import LONG, MODERATE, TINY, make_qkv
from _helpers import check_lse, check_mass, check_out, f64

pytestmark = pytest.mark.gpu


def _separate(q, k, v, **kw):
    out, lse = ad.dense_attn_lse(q, k, v, scale=kw.get("scale"))
    res = ad.block_search(q, k, lse, **kw)
    return out, lse, res


def _assert_same(a, b):
    (o1, l1, r1), (o2, l2, r2) = a, b
    torch.cuda.synchronize()
    assert torch.equal(o1, o2), "out"
    assert torch.equal(l1, l2), "lse"
    assert torch.equal(r1.block_mass, r2.block_mass), "block_mass"
    assert torch.equal(r1.row_ptr, r2.row_ptr), "row_ptr"
    n = r1.nnz()
    assert n == r2.nnz()
    assert torch.equal(r1.col_idx[:n], r2.col_idx[:n]), "col_idx"
    assert torch.equal(r1.head_k, r2.head_k) and torch.equal(r1.head_recall, r2.head_recall)


SHAPES = [
    TINY,                                                                          # d 64, block 64, L 2048
    TINY.replace(head_dim=128, block=128, seqlen=1000, patches=234),              # ragged, 4 tiles of 256
    TINY.replace(head_dim=128, block=64, seqlen=777, frames=5, patches=178),      # ragged block 64, last tile 9 rows
    TINY.replace(head_dim=64, block=128, seqlen=300, patches=59),                 # one tile and 44 rows
    TINY.replace(batch=2, heads=3, head_dim=128, block=64, seqlen=1000, patches=234),
    MODERATE.replace(heads=4),                                                     # d 64, block 128, NB 140
    LONG.replace(name="slice_L17456_H2_d128_b64", heads=2, frames=5, seqlen=256 + 5 * 3440,
                 block=64),                                                        # NB 273
]


@pytest.mark.parametrize("case", range(len(SHAPES)))
@pytest.mark.parametrize("mode", ["coverage", "topk", "hierarchical"])
def test_fused_equals_separate_calls(case, mode):
    w = SHAPES[case]
    print(f"[fused] {w.name} B{w.batch} H{w.heads} d{w.head_dim} L{w.seqlen} b{w.block} {mode}", flush=True)
    q, k, v = make_qkv(w, device="cuda")
    H = q.shape[1]
    params = None if mode == "hierarchical" else ([9000] * H if mode == "coverage" else [2000] * H)
    kw = dict(block=w.block, text_start=w.text_start, text_len=w.text_len, mode=mode,
              head_param_bp=params, base_sparsity_bp=8000, recall_threshold_bp=8000)
    _assert_same(ad.fused_online_search(q, k, v, **kw), _separate(q, k, v, **kw))


def test_fused_without_lse_output():
    """lse may be skipped: the masses still come from the fresh LSE."""
    w = SHAPES[2]
    q, k, v = make_qkv(w, device="cuda")
    kw = dict(block=w.block, text_start=w.text_start, text_len=w.text_len, mode="coverage",
              head_param_bp=[9000] * w.heads)
    out, lse, res = ad.fused_online_search(q, k, v, want_lse=False, **kw)
    assert lse is None
    o2, _, r2 = _separate(q, k, v, **kw)
    torch.cuda.synchronize()
    assert torch.equal(out, o2) and torch.equal(res.block_mass, r2.block_mass)


@pytest.mark.parametrize("block", [128, 64])
def test_fused_long_shape(block):
    """The 110K-token workload (24 heads, d 128, coverage 0.9) at both block
    sizes: 862 or 1,724 key blocks."""
    w = LONG if block == 128 else LONG.replace(block=64)
    print(f"[fused] 110K block {block}", flush=True)
    q, k, v = make_qkv(w, device="cuda")
    kw = dict(block=w.block, text_start=w.text_start, text_len=w.text_len, mode="coverage",
              head_param_bp=[w.coverage_bp] * w.heads)
    _assert_same(ad.fused_online_search(q, k, v, **kw), _separate(q, k, v, **kw))


def test_fused_against_oracle():
    """Algorithm 1 end to end on the tiny workload: dense output and LSE, and
    the masses of the fresh LSE, against the oracle; every row's masses sum
    to its 64 query rows' probability mass of 1 each."""
    w = TINY
    q, k, v = make_qkv(w, device="cuda")
    out, lse, res = ad.fused_online_search(q, k, v, block=w.block, text_start=w.text_start,
                                           text_len=w.text_len, mode="coverage",
                                           head_param_bp=[w.coverage_bp] * w.heads)
    torch.cuda.synchronize()
    for h in range(w.heads):
        qh, kh, vh = f64(q[0, h]), f64(k[0, h]), f64(v[0, h])
        o_ref, l_ref = oracle.dense_attention(qh, kh, vh, w.scale)
        check_out(out[0, h], o_ref, f"h{h}")
        check_lse(lse[0, h], l_ref, f"h{h}")
        check_mass(res.block_mass[0, h], oracle.block_mass(qh, kh, l_ref, w.scale, w.block), f"h{h}")
    np.testing.assert_allclose(res.block_mass.double().sum(-1).cpu().numpy(), 64.0, rtol=1e-3)


@pytest.mark.parametrize("kind", ["negative", "rising", "spiky"])
@pytest.mark.parametrize("D,block,L", [(64, 64, 1000), (128, 128, 777), (128, 64, 777)])
def test_fused_extreme_scores_equal_separate_calls(kind, D, block, L):
    """Scores that stress the online softmax (rows below the fp32 exponent
    range, maxima rising on every tile, large jumps that send waves to the
    exact-path redo): the fused kernel's first pass takes the same paths as
    the dense kernel, and its second pass uses the resulting LSE from
    registers, so all outputs still equal the two calls bit for bit."""
    from workloads import make_extreme_qkv
    (q, k, v), scale = make_extreme_qkv(kind, heads=2, seqlen=L, head_dim=D, device="cuda")
    kw = dict(block=block, text_start=0, text_len=0, mode="topk", head_param_bp=[5000, 5000],
              scale=scale)
    _assert_same(ad.fused_online_search(q, k, v, **kw), _separate(q, k, v, **kw))


@pytest.mark.parametrize("D,block,L", [(128, 64, 1), (64, 128, 1), (64, 64, 64), (128, 128, 130),
                                       (128, 64, 130)])
def test_degenerate_lengths(D, block, L):
    """Lengths of one token, exactly one block, and one block plus two rows:
    the mass pass (no full key tile, or one, and a ragged last tile) against
    the oracle given the same fp32 LSE, and the fused search equal to the two
    calls bit for bit."""
    T = min(64, L)
    w = TINY.replace(head_dim=D, block=block, seqlen=L, text_len=T, frames=4,
                     patches=max(1, (L - T + 3) // 4))
    q, k, v = make_qkv(w, device="cuda")
    H = w.heads
    lse_ref = torch.empty(1, H, L, dtype=torch.float32)
    for h in range(H):
        _, l_ref = oracle.dense_attention(f64(q[0, h]), f64(k[0, h]), f64(v[0, h]), w.scale)
        lse_ref[0, h] = torch.from_numpy(l_ref.astype(np.float32))
    res = ad.block_search(q, k, lse_ref.cuda(), block=block, text_start=0, text_len=T, mode="topk",
                          head_param_bp=[5000] * H)
    torch.cuda.synchronize()
    for h in range(H):
        ref = oracle.block_mass(f64(q[0, h]), f64(k[0, h]), f64(lse_ref[0, h]), w.scale, block)
        check_mass(res.block_mass[0, h], ref, f"L{L} h{h}")
    kw = dict(block=block, text_start=0, text_len=T, mode="coverage", head_param_bp=[9000] * H)
    _assert_same(ad.fused_online_search(q, k, v, **kw), _separate(q, k, v, **kw))
