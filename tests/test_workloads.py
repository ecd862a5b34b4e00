"""The seeded input generator (the input recipe shared by the tests and the
benchmark): token layout of the Sec. 2.1 sequence-length equation, the
frame/patch structure of the video tokens, determinism, per-head draws and
the optional per-head weight of the shared part.  CPU only."""
import torch

from workloads import LONG, MODERATE, TINY, make_qkv, text_blocks


def test_token_layout_of_the_named_workloads():
    for w in (TINY, MODERATE, LONG):
        assert w.seqlen == w.text_len + w.video_len
        assert w.text_start == 0 and w.text_first
        full, part = divmod(w.video_len, w.patches)
        assert full + (part > 0) == w.frames            # the last frame may be partial
    assert LONG.seqlen == 110336 and LONG.nblocks == 862 and LONG.video_len == 32 * 3440
    assert MODERATE.video_len == 13 * 1358 + 10
    assert text_blocks(LONG.seqlen, 128, 0, 256) == [0, 1]


def test_draws_are_deterministic_and_per_head():
    w = TINY.replace(heads=3)
    a = make_qkv(w)
    b = make_qkv(w)
    one = make_qkv(w, heads=range(1, 2))
    for x, y, z in zip(a, b, one):
        assert x.dtype == torch.bfloat16 and x.shape == (1, 3, w.seqlen, w.head_dim)
        assert torch.equal(x, y)
        assert torch.equal(x[:, 1:2], z)
    other = make_qkv(w.replace(seed=w.seed + 1))
    assert not torch.equal(a[0], other[0])


def test_text_tokens_are_plain_noise_and_video_tokens_share_frames():
    """Text rows carry no shared part; video tokens of one frame share U[f],
    so their mean Q.K score is well above that of text tokens."""
    w = TINY
    q, k, _ = make_qkv(w, fp32=True)
    t, v0 = w.text_len, w.text_len
    qt, kt = q[0, 0, :t], k[0, 0, :t]
    qv, kv = q[0, 0, v0:v0 + w.patches], k[0, 0, v0:v0 + w.patches]   # frame 0
    text_score = (qt @ kt.T).mean().item()
    frame_score = (qv @ kv.T).mean().item()
    assert abs(text_score) < 2.0
    assert frame_score > 0.5 * (0.8 ** 2) * w.head_dim


def test_head_structure_weights_the_shared_part_only():
    w = TINY.replace(heads=2)
    base = make_qkv(w, fp32=True)
    assert all(torch.equal(x, y) for x, y in zip(base, make_qkv(w.replace(head_structure=()), fp32=True)))
    zero = make_qkv(w.replace(head_structure=(0.0,)), fp32=True)
    two = make_qkv(w.replace(head_structure=(2.0, 1.0)), fp32=True)
    t = w.text_len
    for b_, z_, t_ in zip(base, zero, two):
        assert torch.equal(b_[..., :t, :], z_[..., :t, :])         # text tokens untouched
        shared = b_[0, :, t:] - z_[0, :, t:]
        torch.testing.assert_close(t_[0, 0, t:] - z_[0, 0, t:], 2.0 * shared[0], rtol=0, atol=1e-5)
        assert torch.equal(t_[0, 1], b_[0, 1])                      # weight 1: the default draw


def test_frame_table_must_hold_every_video_token():
    """A workload whose frames cannot hold its video tokens is refused when it
    is made, on the host: make_qkv indexes the frame table by v // patches,
    and on a GPU an index past the table is a memory fault, not an error
    (L = 777 with 64 text tokens and 178 patches needs a fifth frame)."""
    import pytest
    with pytest.raises(ValueError, match="frames"):
        TINY.replace(head_dim=128, block=64, seqlen=777, patches=178)
    ok = TINY.replace(head_dim=128, block=64, seqlen=777, frames=5, patches=178)
    assert (ok.video_len - 1) // ok.patches == ok.frames - 1
    with pytest.raises(ValueError, match="text_len"):
        TINY.replace(seqlen=32)
