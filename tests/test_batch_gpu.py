"""GPU parity with two batch elements: every call indexes (b*H + h) for the
tensors and (b*H + h)*NB + p for the block rows (Sec. 4.1 definitions per
batch element and head).  Mass pass and block-sparse attention against the
fp64 oracle, each batch element with its own seeded inputs and pattern."""
import numpy as np
import pytest
import torch

import oracle
import paper_2502_21079_amd as ad
from workloads import TINY, make_qkv, random_block_lists, text_blocks
from _helpers import check_lse, check_mass, check_out, f64

pytestmark = pytest.mark.gpu


def _w(D, block, L):
    return TINY.replace(batch=2, heads=3, head_dim=D, block=block, seqlen=L, text_len=64,
                        patches=(L - 64 + 3) // 4)


@pytest.mark.parametrize("D,block,L", [(64, 64, 1000), (128, 128, 1000)])
def test_mass_two_batch_elements(D, block, L):
    """Masses with the oracle's fp32 LSE on both sides, per (b, h)."""
    w = _w(D, block, L)
    q, k, v = make_qkv(w, device="cuda")
    lse = torch.empty(2, 3, L, dtype=torch.float32)
    for b in range(2):
        for h in range(3):
            _, l_ref = oracle.dense_attention(f64(q[b, h]), f64(k[b, h]), f64(v[b, h]), w.scale)
            lse[b, h] = torch.from_numpy(l_ref.astype(np.float32))
    lse = lse.cuda()
    res = ad.block_search(q, k, lse, block=block, text_start=0, text_len=64, mode="topk",
                          head_param_bp=[2000] * 3)
    torch.cuda.synchronize()
    for b in range(2):
        for h in range(3):
            ref = oracle.block_mass(f64(q[b, h]), f64(k[b, h]), f64(lse[b, h]), w.scale, block)
            check_mass(res.block_mass[b, h], ref, f"b{b} h{h}")


@pytest.mark.parametrize("D,block,L", [(64, 64, 1000), (128, 64, 777), (128, 128, 1000), (64, 128, 777)])
def test_sparse_two_batch_elements(D, block, L):
    w = _w(D, block, L)
    q, k, v = make_qkv(w, device="cuda")
    nb = w.nblocks
    rp, ci = random_block_lists(2 * 3 * nb, nb, 4, seed=L + D, always=text_blocks(L, block, 0, 64))
    out, lse = ad.block_sparse_attn(q, k, v, rp.cuda(), ci.cuda(), block=block, text_start=0, text_len=64)
    torch.cuda.synchronize()
    rpn, cin = rp.numpy(), ci.numpy()
    for b in range(2):
        for h in range(3):
            r0 = (b * 3 + h) * nb
            o_ref, l_ref = oracle.block_sparse_attention(f64(q[b, h]), f64(k[b, h]), f64(v[b, h]),
                                                         rpn[r0:r0 + nb + 1], cin, w.scale, block)
            check_out(out[b, h], o_ref, f"b{b} h{h}")
            check_lse(lse[b, h], l_ref, f"b{b} h{h}")
