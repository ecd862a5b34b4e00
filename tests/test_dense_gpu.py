"""GPU parity of adaspa_dense_attn_lse against the fp64 oracle (Sec. 2.2)."""
import numpy as np
import pytest
import torch

import paper_2502_21079_amd as ad
from workloads import LONG, MODERATE, TINY, make_qkv
from _helpers import check_lse, check_out, oracle_rows, sample_blocks

pytestmark = pytest.mark.gpu


def _run(w, heads=None):
    q, k, v = make_qkv(w, device="cuda", heads=heads)
    out, lse = ad.dense_attn_lse(q, k, v)
    torch.cuda.synchronize()
    return q, k, v, out, lse


def test_dense_tiny_full():
    w = TINY
    q, k, v, out, lse = _run(w)
    rows = np.arange(w.seqlen)
    for h in range(w.heads):
        o_ref, l_ref = oracle_rows(q, k, v, (0, h), rows, w.scale)
        check_out(out[0, h], o_ref, f"out h{h}")
        check_lse(lse[0, h], l_ref, f"lse h{h}")


@pytest.mark.parametrize("D,L,text_first", [(128, 1000, False), (64, 777, True), (128, 130, True),
                                            (64, 64, True), (128, 1, True), (128, 2049, True)])
def test_dense_ragged_and_degenerate(D, L, text_first):
    w = TINY.replace(head_dim=D, seqlen=L, text_len=min(64, L), frames=4,
                     patches=max(1, (L - min(64, L) + 3) // 4), text_first=text_first)
    q, k, v, out, lse = _run(w)
    rows = np.arange(L)
    for h in range(w.heads):
        o_ref, l_ref = oracle_rows(q, k, v, (0, h), rows, w.scale)
        check_out(out[0, h], o_ref, f"D{D} L{L} h{h}")
        check_lse(lse[0, h], l_ref)


def test_dense_moderate_sampled():
    w = MODERATE
    q, k, v, out, lse = _run(w)
    nb = w.nblocks
    for h in range(0, w.heads, 3):
        blocks = sample_blocks(nb, 3, seed=100 + h, always=(0, 1, 2))
        rows = np.concatenate([np.arange(p * w.block, min((p + 1) * w.block, w.seqlen)) for p in blocks])
        o_ref, l_ref = oracle_rows(q, k, v, (0, h), rows, w.scale)
        idx = torch.as_tensor(rows, device="cuda")
        check_out(out[0, h, idx], o_ref, f"h{h}")
        check_lse(lse[0, h, idx], l_ref)


def test_dense_long_sampled():
    w = LONG
    q, k, v, out, lse = _run(w)
    nb = w.nblocks
    for h in range(0, w.heads, 4):
        blocks = sample_blocks(nb, 3, seed=200 + h, always=(0, 1))
        rows = np.concatenate([np.arange(p * w.block, min((p + 1) * w.block, w.seqlen)) for p in blocks])
        o_ref, l_ref = oracle_rows(q, k, v, (0, h), rows, w.scale)
        idx = torch.as_tensor(rows, device="cuda")
        check_out(out[0, h, idx], o_ref, f"h{h}")
        check_lse(lse[0, h, idx], l_ref)


def test_dense_deterministic_and_lse_optional():
    q, k, v = make_qkv(TINY.replace(head_dim=128), device="cuda")
    o1, l1 = ad.dense_attn_lse(q, k, v)
    o2, l2 = ad.dense_attn_lse(q, k, v)
    o3, l3 = ad.dense_attn_lse(q, k, v, want_lse=False)
    torch.cuda.synchronize()
    assert l3 is None
    assert torch.equal(o1, o2) and torch.equal(l1, l2) and torch.equal(o1, o3)


def test_dense_work_queue_matches_static_split():
    """The per-XCD work queues only change which CU computes a tile: the
    output and LSE are bitwise those of the static split, for a tile count
    that does not divide by the eight queues, and on back-to-back calls that
    reuse one workspace (the counters are cleared by each call)."""
    w = TINY.replace(head_dim=128, heads=3, seqlen=1900, patches=459)
    q, k, v = make_qkv(w, device="cuda")
    o0, l0 = ad.dense_attn_lse(q, k, v, balance=False)
    ws = torch.empty(ad.dense_attn_workspace(q.shape), dtype=torch.uint8, device="cuda")
    for _ in range(3):
        o1, l1 = ad.dense_attn_lse(q, k, v, workspace=ws)
        torch.cuda.synchronize()
        assert torch.equal(o0, o1) and torch.equal(l0, l1)


def test_dense_batch_and_custom_scale():
    w = TINY.replace(batch=2, seqlen=512, text_len=64, patches=112)
    q, k, v = make_qkv(w, device="cuda")
    out, lse = ad.dense_attn_lse(q, k, v, scale=0.05)
    torch.cuda.synchronize()
    rows = np.arange(512)
    for b in range(2):
        for h in range(2):
            o_ref, l_ref = oracle_rows(q, k, v, (b, h), rows, 0.05)
            check_out(out[b, h], o_ref)
            check_lse(lse[b, h], l_ref)
