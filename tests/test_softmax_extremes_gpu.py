"""GPU parity under score ranges that stress the online softmax's lazy
reference (Sec. 2.2 online softmax; the reference moves on a rare path): rows
whose scaled scores all lie far below the fp32 exponent range, row maxima that
rise on every key tile, and large random jumps.  Dense, block-sparse and the
all-blocks identity, each against the fp64 oracle on the same inputs."""
import numpy as np
import pytest
import torch

import oracle
import paper_2502_21079_amd as ad
from workloads import EXTREME_KINDS, make_extreme_qkv, random_block_lists
from _helpers import check_lse, check_mass, check_out, f64

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("kind", EXTREME_KINDS)
@pytest.mark.parametrize("D,L", [(64, 1000), (128, 777)])
def test_dense_extreme_scores(kind, D, L):
    (q, k, v), scale = make_extreme_qkv(kind, heads=2, seqlen=L, head_dim=D, device="cuda")
    out, lse = ad.dense_attn_lse(q, k, v, scale=scale)
    torch.cuda.synchronize()
    for h in range(2):
        o_ref, l_ref = oracle.dense_attention(f64(q[0, h]), f64(k[0, h]), f64(v[0, h]), scale)
        assert np.all(np.isfinite(l_ref))
        check_out(out[0, h], o_ref, f"{kind} D{D} h{h}")
        check_lse(lse[0, h], l_ref, f"{kind} lse h{h}")


@pytest.mark.parametrize("kind", EXTREME_KINDS)
@pytest.mark.parametrize("D,block,L,kb", [(64, 64, 1000, 5), (128, 128, 777, 3), (128, 64, 777, 4),
                                           (64, 128, 1000, 8)])
def test_sparse_extreme_scores(kind, D, block, L, kb):
    (q, k, v), scale = make_extreme_qkv(kind, heads=2, seqlen=L, head_dim=D, device="cuda")
    nb = (L + block - 1) // block
    rp, ci = random_block_lists(2 * nb, nb, kb, seed=L + kb, always=[0])
    out, lse = ad.block_sparse_attn(q, k, v, rp.cuda(), ci.cuda(), block=block, scale=scale,
                                    text_start=0, text_len=0)
    torch.cuda.synchronize()
    rpn, cin = rp.numpy(), ci.numpy()
    for h in range(2):
        o_ref, l_ref = oracle.block_sparse_attention(f64(q[0, h]), f64(k[0, h]), f64(v[0, h]),
                                                     rpn[h * nb:(h + 1) * nb + 1], cin, scale, block)
        check_out(out[0, h], o_ref, f"{kind} b{block} h{h}")
        check_lse(lse[0, h], l_ref, f"{kind} lse h{h}")


@pytest.mark.parametrize("kind", EXTREME_KINDS)
@pytest.mark.parametrize("block", [64, 128])
@pytest.mark.parametrize("L", [900, 1000])
def test_all_blocks_equals_dense_extreme(kind, block, L):
    """Keeping every block equals dense bit for bit, also where waves redo
    their rows on the exact path; at L = 1000 the last block of 128 holds a
    full tile that both kernels take through the pipeline."""
    (q, k, v), scale = make_extreme_qkv(kind, heads=2, seqlen=L, head_dim=64, device="cuda")
    nb = (L + block - 1) // block
    od, ld = ad.dense_attn_lse(q, k, v, scale=scale)
    rp = (torch.arange(2 * nb + 1, dtype=torch.int32) * nb).cuda()
    ci = torch.arange(nb, dtype=torch.int32).repeat(2 * nb).cuda()
    os_, ls = ad.block_sparse_attn(q, k, v, rp, ci, block=block, scale=scale, text_start=0, text_len=0)
    torch.cuda.synchronize()
    assert torch.equal(od, os_) and torch.equal(ld, ls)


@pytest.mark.parametrize("kind", EXTREME_KINDS)
@pytest.mark.parametrize("D,block,L", [(64, 64, 1000), (128, 128, 777)])
def test_mass_extreme_scores(kind, D, block, L):
    """The mass pass with the oracle's fp32 LSE on both sides: exp(s - LSE)
    summed per block stays exact where the scores span hundreds of units."""
    (q, k, v), scale = make_extreme_qkv(kind, heads=2, seqlen=L, head_dim=D, device="cuda")
    lse = torch.empty(1, 2, L, dtype=torch.float32)
    for h in range(2):
        _, l_ref = oracle.dense_attention(f64(q[0, h]), f64(k[0, h]), f64(v[0, h]), scale)
        lse[0, h] = torch.from_numpy(l_ref.astype(np.float32))
    lse = lse.cuda()
    res = ad.block_search(q, k, lse, block=block, text_start=0, text_len=0, mode="topk",
                          head_param_bp=[5000, 5000], scale=scale)
    torch.cuda.synchronize()
    for h in range(2):
        ref = oracle.block_mass(f64(q[0, h]), f64(k[0, h]), f64(lse[0, h]), scale, block)
        check_mass(res.block_mass[0, h], ref, f"{kind} h{h}")


BIG_V = 2.0 ** 72


@pytest.mark.parametrize("kind", ["rising", "spiky"])
@pytest.mark.parametrize("block", [64, 128])
def test_large_values_take_the_exact_path(kind, block):
    """Large |V|.  The lazy softmax reference lets a tile's probabilities grow
    to about 2^58 before the row sums move it; times V entries near 2^74 the
    products overflow fp32 in the output accumulator while the row sums stay
    in range.  Those rows must be redone on the exact path.  V is the N(0, 1)
    draw scaled by 2^72 (exact in bf16); outputs divided by 2^72 are checked
    against the oracle on the unscaled V, for dense, block-sparse and the
    all-blocks identity."""
    L, D = 1000, 64
    (q, k, v0), scale = make_extreme_qkv(kind, heads=2, seqlen=L, head_dim=D, device="cuda")
    v = (v0.float() * BIG_V).to(torch.bfloat16)
    assert torch.equal(v.float() / BIG_V, v0.float())
    nb = (L + block - 1) // block
    od, ld = ad.dense_attn_lse(q, k, v, scale=scale)
    rp, ci = random_block_lists(2 * nb, nb, 5, seed=91 + block, always=[0])
    os_, ls = ad.block_sparse_attn(q, k, v, rp.cuda(), ci.cuda(), block=block, scale=scale,
                                   text_start=0, text_len=0)
    rpa = (torch.arange(2 * nb + 1, dtype=torch.int32) * nb).cuda()
    cia = torch.arange(nb, dtype=torch.int32).repeat(2 * nb).cuda()
    oa, la = ad.block_sparse_attn(q, k, v, rpa, cia, block=block, scale=scale, text_start=0,
                                  text_len=0)
    torch.cuda.synchronize()
    assert torch.equal(od, oa) and torch.equal(ld, la)
    rpn, cin = rp.numpy(), ci.numpy()
    for h in range(2):
        qh, kh, vh = f64(q[0, h]), f64(k[0, h]), f64(v0[0, h])
        o_ref, l_ref = oracle.dense_attention(qh, kh, vh, scale)
        check_out(od[0, h].float() / BIG_V, o_ref, f"{kind} dense h{h}")
        check_lse(ld[0, h], l_ref, f"{kind} dense lse h{h}")
        o_sp, l_sp = oracle.block_sparse_attention(qh, kh, vh, rpn[h * nb:(h + 1) * nb + 1], cin,
                                                   scale, block)
        check_out(os_[0, h].float() / BIG_V, o_sp, f"{kind} b{block} sparse h{h}")
        check_lse(ls[0, h], l_sp, f"{kind} b{block} sparse lse h{h}")
