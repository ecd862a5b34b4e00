"""CPU checks of the C-ABI library: it loads, exports every symbol the header
declares, and rejects invalid arguments synchronously (before any GPU work).

Only validation paths and pure host helpers are called here: no kernel runs.
"""
import ctypes
import os
import re

import pytest
import torch

import paper_2502_21079_amd as ad

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "adaspa.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(adaspa_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    return ad.load_library()


def test_header_declares_the_binding_symbols():
    assert _declared_functions() == sorted(ad.EXPORTED_SYMBOLS)


def test_library_exports_every_declared_symbol(lib):
    for name in _declared_functions():
        assert hasattr(lib, name), name
        assert getattr(lib, name) is not None


def test_status_strings(lib):
    for code in range(6):
        assert lib.adaspa_status_string(code)
    assert lib.adaspa_status_string(0) == b"ok"


def _prob(**kw):
    base = dict(batch=1, heads=2, seqlen=2048, head_dim=64, block=64, text_start=0,
                text_len=64, softmax_scale=0.0)
    base.update(kw)
    return ad._Problem(*[base[f] for f, _ in ad._Problem._fields_])


def _sel(mode=0, flags=1, params=(2000, 2000)):
    arr = (ctypes.c_int32 * len(params))(*params)
    return ad._Select(mode, flags, ctypes.cast(arr, ctypes.POINTER(ctypes.c_int32))), arr


FAKE = ctypes.c_void_p(0x10000)     # aligned, never dereferenced: validation fails first


@pytest.mark.parametrize("kw,status", [
    (dict(head_dim=96), 2), (dict(head_dim=256), 2), (dict(block=32), 2), (dict(block=256), 2),
    (dict(seqlen=0), 1), (dict(batch=0), 1), (dict(heads=0), 1),
    (dict(text_start=2000, text_len=100), 1), (dict(text_len=-1), 1),
    (dict(softmax_scale=float("nan")), 1), (dict(softmax_scale=float("inf")), 1),
])
def test_dense_rejects_bad_problems(lib, kw, status):
    p = _prob(**kw)
    assert lib.adaspa_dense_attn_lse(ctypes.byref(p), FAKE, FAKE, FAKE, FAKE, None, None, 0, None) == status
    assert lib.adaspa_dense_attn_workspace(ctypes.byref(p)) == 0


def test_dense_rejects_null_and_misaligned(lib):
    p = _prob()
    assert lib.adaspa_dense_attn_lse(None, FAKE, FAKE, FAKE, FAKE, None, None, 0, None) == 1
    assert lib.adaspa_dense_attn_lse(ctypes.byref(p), None, FAKE, FAKE, FAKE, None, None, 0, None) == 1
    assert lib.adaspa_dense_attn_lse(ctypes.byref(p), ctypes.c_void_p(0x10008), FAKE, FAKE, FAKE,
                                     None, None, 0, None) == 1
    assert lib.adaspa_dense_attn_lse(ctypes.byref(p), FAKE, FAKE, FAKE, FAKE,
                                     ctypes.c_void_p(0x10002), None, 0, None) == 1


def test_dense_workspace_checks(lib):
    """The work-queue workspace is optional; when given it must be large
    enough and 16-byte aligned (checked before anything is enqueued)."""
    p = _prob()
    need = lib.adaspa_dense_attn_workspace(ctypes.byref(p))
    assert need >= 36 and need % 16 == 0
    assert lib.adaspa_dense_attn_lse(ctypes.byref(p), FAKE, FAKE, FAKE, FAKE, None, FAKE,
                                     need - 1, None) == 4
    assert lib.adaspa_dense_attn_lse(ctypes.byref(p), FAKE, FAKE, FAKE, FAKE, None,
                                     ctypes.c_void_p(0x10004), need, None) == 4


def test_capacity_and_workspace(lib):
    p = _prob()
    s, _a = _sel(mode=0, params=(2000, 5000))
    nb = 32
    # one text block -> text row keeps 32; video rows keep ceil(0.2*32)=7 / 16
    expect = (nb + (nb - 1) * 7) + (nb + (nb - 1) * 16)
    assert lib.adaspa_block_search_capacity(ctypes.byref(p), ctypes.byref(s)) == expect
    s2, _b = _sel(mode=1, params=(9000, 9000))
    assert lib.adaspa_block_search_capacity(ctypes.byref(p), ctypes.byref(s2)) == 2 * nb * nb
    ws = lib.adaspa_block_search_workspace(ctypes.byref(p), ctypes.byref(s2))
    assert ws >= 2 * nb * nb * 12 and ws % 256 == 0
    bad, _c = _sel(mode=1, params=(9000, 10001))
    assert lib.adaspa_block_search_workspace(ctypes.byref(p), ctypes.byref(bad)) == 0
    assert lib.adaspa_block_search_capacity(ctypes.byref(p), ctypes.byref(bad)) == -1
    bad2, _d = _sel(mode=7)
    assert lib.adaspa_block_search_capacity(ctypes.byref(p), ctypes.byref(bad2)) == -1


def test_hierarchical_capacity_and_validation(lib):
    import oracle
    p = _prob(seqlen=110336, heads=3, head_dim=128, block=128, text_len=256)
    for base in (0, 5000, 8000, 9000, 10000):
        s = ad._Select(2, 1, None, base, 8000)
        s_hi, s_lo = (10000 + base) // 2, max(0, (3 * base - 10000) // 2)
        kmax = max(oracle.topk_count(10000 - x, 862, 2) for x in (base, s_hi, s_lo))
        assert lib.adaspa_block_search_capacity(ctypes.byref(p), ctypes.byref(s)) == 3 * (2 * 862 + 860 * kmax)
        assert lib.adaspa_block_search_workspace(ctypes.byref(p), ctypes.byref(s)) > 0
    for bad in ((-1, 8000), (10001, 8000), (8000, -1), (8000, 10001)):
        s = ad._Select(2, 1, None, *bad)
        assert lib.adaspa_block_search_capacity(ctypes.byref(p), ctypes.byref(s)) == -1


def test_block_count_limit(lib):
    s, _a = _sel(mode=0, params=(1000,))
    ok = _prob(seqlen=8192 * 64, heads=1, block=64, text_len=256)
    assert lib.adaspa_block_search_capacity(ctypes.byref(ok), ctypes.byref(s)) > 0
    too_many = _prob(seqlen=8192 * 64 + 1, heads=1, block=64, text_len=256)
    assert lib.adaspa_block_search_capacity(ctypes.byref(too_many), ctypes.byref(s)) == -1


def test_capacity_matches_oracle_counts(lib):
    import oracle
    for keep in (0, 1, 500, 1000, 2000, 5000, 10000):
        p = _prob(seqlen=110336, heads=1, head_dim=128, block=128, text_len=256)
        s, _a = _sel(mode=0, params=(keep,))
        k = oracle.topk_count(keep, 862, 2)
        assert lib.adaspa_block_search_capacity(ctypes.byref(p), ctypes.byref(s)) == 2 * 862 + 860 * k


def test_search_rejects_bad_arguments(lib):
    p = _prob()
    s, _a = _sel()
    ws = lib.adaspa_block_search_workspace(ctypes.byref(p), ctypes.byref(s))
    cap = lib.adaspa_block_search_capacity(ctypes.byref(p), ctypes.byref(s))
    args = lambda **o: [o.get("prob", ctypes.byref(p)), FAKE, FAKE, FAKE, o.get("sel", ctypes.byref(s)),
                        FAKE, FAKE, FAKE, o.get("cap", cap), None, None, o.get("ws", FAKE),
                        o.get("wsb", ws), None]
    assert lib.adaspa_block_search(*args(cap=cap - 1)) == 3
    assert lib.adaspa_block_search(*args(wsb=ws - 1)) == 4
    assert lib.adaspa_block_search(*args(ws=None)) == 4
    assert lib.adaspa_block_search(*args(ws=ctypes.c_void_p(0x10010))) == 4
    assert lib.adaspa_block_search(*args(sel=None)) == 1
    s_bad, _b = _sel(flags=8)
    assert lib.adaspa_block_search(*args(sel=ctypes.byref(s_bad))) == 1
    big = _prob(heads=600)
    arr = (ctypes.c_int32 * 600)(*([1000] * 600))
    s_big = ad._Select(0, 1, ctypes.cast(arr, ctypes.POINTER(ctypes.c_int32)))
    assert lib.adaspa_block_search(ctypes.byref(big), FAKE, FAKE, FAKE, ctypes.byref(s_big), FAKE,
                                   FAKE, FAKE, 10 ** 9, None, None, FAKE, 10 ** 12, None) == 2


def test_sparse_rejects_bad_arguments(lib):
    p = _prob()
    assert lib.adaspa_block_sparse_attn(ctypes.byref(p), FAKE, FAKE, FAKE, None, FAKE, 10, FAKE,
                                        None, None, 0, None) == 1
    assert lib.adaspa_block_sparse_attn(ctypes.byref(p), FAKE, FAKE, FAKE, FAKE, FAKE, -1, FAKE,
                                        None, None, 0, None) == 1
    assert lib.adaspa_block_sparse_attn(ctypes.byref(p), FAKE, FAKE, FAKE, FAKE,
                                        ctypes.c_void_p(0x10001), 10, FAKE, None, None, 0, None) == 1
    assert lib.adaspa_block_sparse_attn(ctypes.byref(_prob(head_dim=80)), FAKE, FAKE, FAKE, FAKE,
                                        FAKE, 10, FAKE, None, None, 0, None) == 2


def test_sparse_block64_block_limit(lib):
    """Block 64 pairs query blocks through a map of at most 8192 key blocks:
    longer sequences are refused before anything is enqueued (block 128 is not
    limited there)."""
    big64 = _prob(seqlen=8193 * 64, block=64)
    assert lib.adaspa_block_sparse_attn(ctypes.byref(big64), FAKE, FAKE, FAKE, FAKE, FAKE, 10, FAKE,
                                        None, None, 0, None) == 2
    # at the limit the call gets past that check to the (misaligned) workspace
    edge64 = _prob(seqlen=8192 * 64, block=64)
    assert lib.adaspa_block_sparse_attn(ctypes.byref(edge64), FAKE, FAKE, FAKE, FAKE, FAKE, 10, FAKE,
                                        None, ctypes.c_void_p(0x10004), 256, None) == 4
    big128 = _prob(seqlen=8193 * 128, block=128)
    assert lib.adaspa_block_sparse_attn(ctypes.byref(big128), FAKE, FAKE, FAKE, FAKE, FAKE, 10, FAKE,
                                        None, ctypes.c_void_p(0x10004), 256, None) == 4


def test_sparse_workspace_checks(lib):
    """As for dense attention: the work-queue workspace is optional, and when
    given it must be large enough and 16-byte aligned."""
    p = _prob()
    need = lib.adaspa_block_sparse_attn_workspace(ctypes.byref(p))
    assert need >= 36 and need % 16 == 0
    assert lib.adaspa_block_sparse_attn_workspace(ctypes.byref(_prob(head_dim=80))) == 0
    assert lib.adaspa_block_sparse_attn(ctypes.byref(p), FAKE, FAKE, FAKE, FAKE, FAKE, 10, FAKE,
                                        None, FAKE, need - 1, None) == 4
    assert lib.adaspa_block_sparse_attn(ctypes.byref(p), FAKE, FAKE, FAKE, FAKE, FAKE, 10, FAKE,
                                        None, ctypes.c_void_p(0x10004), need, None) == 4


def test_binding_raises_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(ad, "_lib", None)
    monkeypatch.setenv("ADASPA_LIB", str(tmp_path / "missing.so"))
    with pytest.raises(ad.AdaspaError):
        ad.load_library()


def test_binding_checks_per_head_parameter_count(lib):
    """The per-head modes read head_param_bp[0 .. H-1]: the binding refuses a
    list of another length before it reaches the library."""
    shape = (1, 24, 110336, 128)
    with pytest.raises(ad.AdaspaError, match="one entry per head"):
        ad.block_search_workspace(shape, 128, 0, 256, "topk", [9000])
    with pytest.raises(ad.AdaspaError, match="one entry per head"):
        ad.block_search_capacity(shape, 128, 0, 256, "coverage", [9000] * 25)
    assert ad.block_search_capacity(shape, 128, 0, 256, "topk", [2000] * 24) > 0
    # the hierarchical mode takes no per-head list
    assert ad.block_search_capacity(shape, 128, 0, 256, "hierarchical", None) > 0
    with pytest.raises(ad.AdaspaError, match="unknown selection mode"):
        ad.block_search_capacity(shape, 128, 0, 256, "top-k", [2000] * 24)


def test_sparse_noalloc_rejects_bad_arguments(lib):
    """The allocation-free entry point checks its arguments like the others,
    synchronously and before it touches a device."""
    f = lib.adaspa_block_sparse_attn_noalloc
    ok = _prob()
    assert f(None, FAKE, FAKE, FAKE, FAKE, FAKE, 10, FAKE, None, None) == 1
    assert f(ctypes.byref(_prob(head_dim=96)), FAKE, FAKE, FAKE, FAKE, FAKE, 10, FAKE, None, None) == 2
    assert f(ctypes.byref(ok), None, FAKE, FAKE, FAKE, FAKE, 10, FAKE, None, None) == 1
    assert f(ctypes.byref(ok), FAKE, FAKE, FAKE, FAKE, FAKE, -1, FAKE, None, None) == 1
    assert f(ctypes.byref(ok), ctypes.c_void_p(0x10008), FAKE, FAKE, FAKE, FAKE, 10, FAKE, None,
             None) == 1
    big = _prob(seqlen=64 * 8193, head_dim=64, block=64)
    assert f(ctypes.byref(big), FAKE, FAKE, FAKE, FAKE, FAKE, 10, FAKE, None, None) == 2


def test_fused_search_rejects_bad_arguments(lib):
    """The fused online search takes the arguments of dense attention and the
    search together and applies both sets of checks, plus one of its own:
    the masses are always computed (ADASPA_F_SCORES_GIVEN is refused)."""
    p = _prob()
    s, _a = _sel()
    ws = lib.adaspa_block_search_workspace(ctypes.byref(p), ctypes.byref(s))
    cap = lib.adaspa_block_search_capacity(ctypes.byref(p), ctypes.byref(s))

    def call(**o):
        return lib.adaspa_fused_online_search(
            o.get("prob", ctypes.byref(p)), o.get("q", FAKE), FAKE, o.get("v", FAKE), FAKE,
            o.get("lse", None), o.get("sel", ctypes.byref(s)), FAKE, FAKE, FAKE, o.get("cap", cap),
            None, None, o.get("ws", FAKE), o.get("wsb", ws), None)

    assert call(v=None) == 1
    assert call(q=ctypes.c_void_p(0x10008)) == 1
    assert call(lse=ctypes.c_void_p(0x10002)) == 1
    assert call(sel=None) == 1
    given, _b = _sel(flags=1 | 2)
    assert call(sel=ctypes.byref(given)) == 1
    assert call(cap=cap - 1) == 3
    assert call(wsb=ws - 1) == 4
    assert call(ws=None) == 4
    assert call(ws=ctypes.c_void_p(0x10010)) == 4
    assert call(prob=ctypes.byref(_prob(head_dim=96))) == 2
    assert call(prob=ctypes.byref(_prob(seqlen=0))) == 1


def test_single_pass_search_rejects_bad_arguments(lib):
    """The single-pass online search applies the fused search's checks; its
    full workspace adds B*H*NB*L floats of per-row block masses and B*H*L
    floats of row LSEs to the search's, the least it accepts those of one
    (batch, head) pair, and a smaller one is refused before anything is
    enqueued."""
    p = _prob()
    s, _a = _sel()
    ws_search = lib.adaspa_block_search_workspace(ctypes.byref(p), ctypes.byref(s))
    ws = lib.adaspa_single_pass_online_search_workspace(ctypes.byref(p), ctypes.byref(s))
    nb = 2048 // 64
    rnd = lambda x: (x + 255) // 256 * 256
    assert ws == ws_search + rnd(2 * nb * 2048 * 4) + rnd(2 * 2048 * 4)
    given, _b = _sel(flags=1 | 2)
    assert lib.adaspa_single_pass_online_search_workspace(ctypes.byref(p), ctypes.byref(given)) == 0
    assert lib.adaspa_single_pass_online_search_workspace(ctypes.byref(_prob(head_dim=96)),
                                                          ctypes.byref(s)) == 0
    # the least accepted: one (batch, head) pair's scratch
    least = lib.adaspa_single_pass_online_search_min_workspace(ctypes.byref(p), ctypes.byref(s))
    assert least == ws_search + rnd(nb * 2048 * 4) + rnd(2048 * 4) and least < ws
    assert lib.adaspa_single_pass_online_search_min_workspace(ctypes.byref(p), ctypes.byref(given)) == 0
    cap = lib.adaspa_block_search_capacity(ctypes.byref(p), ctypes.byref(s))

    def call(**o):
        return lib.adaspa_single_pass_online_search(
            o.get("prob", ctypes.byref(p)), o.get("q", FAKE), FAKE, o.get("v", FAKE), FAKE,
            o.get("lse", None), o.get("sel", ctypes.byref(s)), FAKE, FAKE, FAKE, o.get("cap", cap),
            None, None, o.get("ws", FAKE), o.get("wsb", ws), None)

    assert call(v=None) == 1
    assert call(q=ctypes.c_void_p(0x10008)) == 1
    assert call(lse=ctypes.c_void_p(0x10002)) == 1
    assert call(sel=None) == 1
    assert call(sel=ctypes.byref(given)) == 1
    assert call(cap=cap - 1) == 3
    assert call(wsb=least - 1) == 4           # (any size from `least` up would be used)
    assert call(wsb=ws_search) == 4
    assert call(ws=None) == 4
    assert call(ws=ctypes.c_void_p(0x10010)) == 4
    assert call(prob=ctypes.byref(_prob(head_dim=96))) == 2
    assert call(prob=ctypes.byref(_prob(seqlen=0))) == 1


def test_binding_checks_caller_outputs():
    """The binding refuses caller-provided outputs whose dtype, shape or
    layout differ from what the kernels write (the library sees pointers
    only): checked on the host, before any call."""
    import torch
    q = torch.empty(1, 2, 8, 64, dtype=torch.bfloat16)
    ad._check_outputs(q, torch.empty_like(q), torch.empty(1, 2, 8, dtype=torch.float32))
    ad._check_outputs(q, None, None)
    bad_out = [torch.empty(1, 2, 7, 64, dtype=torch.bfloat16), torch.empty(1, 2, 8, 64, dtype=torch.float32),
               torch.empty(1, 2, 64, 8, dtype=torch.bfloat16).transpose(2, 3)]
    for o in bad_out:
        with pytest.raises(ad.AdaspaError, match="out must"):
            ad._check_outputs(q, o, None)
    for l in [torch.empty(1, 2, 7, dtype=torch.float32), torch.empty(1, 2, 8, dtype=torch.bfloat16),
              torch.empty(2, 8, dtype=torch.float32)]:
        with pytest.raises(ad.AdaspaError, match="lse must"):
            ad._check_outputs(q, None, l)


def test_workspace_tensors_count_in_bytes():
    """A caller's workspace of any dtype counts in bytes; one on another
    device than the inputs, or not contiguous, is refused before any call."""
    cpu = torch.device("cpu")
    assert ad._workspace_bytes(torch.empty(10, dtype=torch.int32), cpu) == 40
    assert ad._workspace_bytes(torch.empty(7, dtype=torch.uint8), cpu) == 7
    with pytest.raises(ad.AdaspaError):
        ad._workspace_bytes(torch.empty(8, 2, dtype=torch.uint8).t(), cpu)
    with pytest.raises(ad.AdaspaError):
        ad._workspace_bytes(torch.empty(8, dtype=torch.uint8), torch.device("cuda", 0))
