"""The allocation-free entry point of block-sparse attention against the
entry point it is a variant of (adaspa_block_sparse_attn with a caller
workspace): bitwise the same outputs and LSE, on two calls in a row, the
second on a smaller problem, for both block sizes.  Nothing is allocated
for the call: outputs are allocated before it."""
import numpy as np
import pytest
import torch

import paper_2502_21079_amd as ad
from workloads import TINY, make_qkv, random_block_lists, text_blocks

pytestmark = pytest.mark.gpu


def _case(block, L, heads, seed):
    w = TINY.replace(head_dim=128, heads=heads, block=block, seqlen=L, text_len=256,
                     patches=(L - 256 + 3) // 4)
    q, k, v = make_qkv(w, device="cuda")
    nb = w.nblocks
    tb = text_blocks(L, block, 0, 256)
    rp, ci = random_block_lists(heads * nb, nb, max(len(tb), nb // 5), seed=seed, always=tb)
    return w, q, k, v, rp.cuda(), ci.cuda()


@pytest.mark.parametrize("block", [64, 128])
def test_noalloc_matches_workspace_entry_point(block):
    for L, heads, seed in ((128 * 97 + 40, 5, 1), (128 * 23 + 8, 3, 2)):   # second call smaller
        w, q, k, v, rp, ci = _case(block, L, heads, seed)
        txt = dict(text_start=w.text_start, text_len=w.text_len)
        ws = torch.empty(ad.block_sparse_attn_workspace(q.shape, block), dtype=torch.uint8,
                         device="cuda")
        o_ref, l_ref = ad.block_sparse_attn(q, k, v, rp, ci, block=block, workspace=ws, **txt)
        out = torch.empty_like(q)
        lse = torch.empty(q.shape[:3], dtype=torch.float32, device="cuda")
        torch.cuda.synchronize()
        o_na, l_na = ad.block_sparse_attn_noalloc(q, k, v, rp, ci, block=block, out=out, lse=lse,
                                                  **txt)
        torch.cuda.synchronize()
        assert o_na.data_ptr() == out.data_ptr() and l_na.data_ptr() == lse.data_ptr()
        assert torch.equal(o_ref, o_na), (block, L)
        assert torch.equal(l_ref, l_na), (block, L)
        assert np.isfinite(l_na.cpu().numpy()).all()
