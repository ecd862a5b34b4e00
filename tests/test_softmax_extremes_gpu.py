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
from _helpers import check_lse, check_out, f64

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
@pytest.mark.parametrize("D,block,L,kb", [(64, 64, 1000, 5), (128, 128, 777, 3), (128, 64, 777, 4)])
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
def test_all_blocks_equals_dense_extreme(kind, block):
    (q, k, v), scale = make_extreme_qkv(kind, heads=2, seqlen=900, head_dim=64, device="cuda")
    nb = (900 + block - 1) // block
    od, ld = ad.dense_attn_lse(q, k, v, scale=scale)
    rp = (torch.arange(2 * nb + 1, dtype=torch.int32) * nb).cuda()
    ci = torch.arange(nb, dtype=torch.int32).repeat(2 * nb).cuda()
    os_, ls = ad.block_sparse_attn(q, k, v, rp, ci, block=block, scale=scale, text_start=0, text_len=0)
    torch.cuda.synchronize()
    assert torch.equal(od, os_) and torch.equal(ld, ls)
