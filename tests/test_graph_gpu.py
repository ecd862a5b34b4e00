"""The hot path under HIP graph capture.  Every call of the library only
validates its arguments and enqueues kernels (its work-queue counters are
cleared by a kernel, not a memset), so one denoising step of the search
schedule (dense attention + LSE, block search, block-sparse attention on the
new pattern; or the fused or single-pass online search, then block-sparse
attention) can be
captured once and replayed.  Between replays new seeded
inputs are written into the captured buffers and the same step runs eagerly
into separate buffers; every replay must equal the eager step bit for bit."""
import pytest
import torch

import paper_2502_21079_amd as ad
from workloads import MODERATE, TINY, make_qkv

pytestmark = pytest.mark.gpu

CASES = {
    "tiny_b64_d64": TINY,
    "slice_b128_d128": MODERATE.replace(name="slice_L17920_H4_d128_b128", heads=4, head_dim=128),
}


class Step:
    """One search step with every output and workspace allocated up front;
    ``way`` runs the dense pass and the masses as two calls, as the fused
    online search or as the single-pass online search."""

    def __init__(self, w, q, k, v, way="two_calls"):
        self.w, self.q, self.k, self.v = w, q, k, v
        self.way = way
        B, H, L, D = q.shape
        self.kw = dict(block=w.block, text_start=w.text_start, text_len=w.text_len)
        self.tau = [9000] * H
        self.out_d = torch.empty_like(q)
        self.lse = torch.empty(B, H, L, dtype=torch.float32, device=q.device)
        self.ws_d = torch.empty(ad.dense_attn_workspace(q.shape), dtype=torch.uint8, device=q.device)
        wsf = ad.single_pass_online_search_workspace if way == "single_pass" else ad.block_search_workspace
        self.ws_s = torch.empty(wsf(q.shape, w.block, w.text_start, w.text_len, "coverage", self.tau),
                                dtype=torch.uint8, device=q.device)
        self.ws_p = torch.empty(ad.block_sparse_attn_workspace(q.shape, w.block), dtype=torch.uint8,
                                device=q.device)
        self.out_s = torch.empty_like(q)
        self.lse_s = torch.empty_like(self.lse)
        self.res = None

    def __call__(self):
        if self.way != "two_calls":
            fn = ad.fused_online_search if self.way == "fused" else ad.single_pass_online_search
            _, _, self.res = fn(self.q, self.k, self.v, mode="coverage", head_param_bp=self.tau,
                                out=self.out_d, lse=self.lse, workspace=self.ws_s, result=self.res, **self.kw)
        else:
            ad.dense_attn_lse(self.q, self.k, self.v, out=self.out_d, lse=self.lse, workspace=self.ws_d)
            self.res = ad.block_search(self.q, self.k, self.lse, mode="coverage", head_param_bp=self.tau,
                                       workspace=self.ws_s, result=self.res, **self.kw)
        ad.block_sparse_attn(self.q, self.k, self.v, self.res.row_ptr, self.res.col_idx, out=self.out_s,
                             lse=self.lse_s, workspace=self.ws_p, **self.kw)

    def outputs(self):
        nnz = int(self.res.row_ptr[-1].item())
        return {"out": self.out_d, "lse": self.lse, "mass": self.res.block_mass,
                "row_ptr": self.res.row_ptr, "col_idx": self.res.col_idx[:nnz], "head_k": self.res.head_k,
                "recall": self.res.head_recall, "sparse_out": self.out_s, "sparse_lse": self.lse_s}


@pytest.mark.parametrize("way", ["two_calls", "fused", "single_pass"])
@pytest.mark.parametrize("case", sorted(CASES))
def test_step_graph_replays_equal_eager(case, way):
    w = CASES[case]
    q, k, v = (t.contiguous() for t in make_qkv(w, device="cuda"))
    cap = Step(w, q, k, v, way)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        cap()                                    # eager warm-up; also allocates the search result
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        cap()
    torch.cuda.synchronize()

    for seed in (11, 12, 13):
        qn, kn, vn = make_qkv(w.replace(seed=seed), device="cuda")
        q.copy_(qn)
        k.copy_(kn)
        v.copy_(vn)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = {name: t.clone() for name, t in cap.outputs().items()}
        ref = Step(w, qn.contiguous(), kn.contiguous(), vn.contiguous(), way)
        ref()
        torch.cuda.synchronize()
        want = ref.outputs()
        assert int(want["row_ptr"][-1].item()) > 0
        for name, t in want.items():
            assert got[name].shape == t.shape and torch.equal(got[name], t), (case, seed, name)
