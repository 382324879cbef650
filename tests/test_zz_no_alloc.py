"""pbg_score_edges_noalloc (no device allocation, static scratch) against
pbg_score_edges, through the C ABI: the same kernels on the same inputs, so
the scores must be bitwise equal, on two calls in a row (the second with a
smaller input, which must not see the first call's scratch contents), with
the linear operator (transposed matrices staged in the scratch) and without.
Out-of-range ids and oversized relation matrices are rejected."""

import numpy as np
import pytest
import torch

from tests.pbg_cases import GpuModel, make_problem

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("op,cmp,R", [("linear", "dot", 4), ("complex_diagonal", "dot", 5),
                                      ("linear", "cos", 1), ("translation", "cos", 1)])
def test_noalloc_scores_equal_allocating_entry_point(op, cmp, R):
    from paper_1903_12287_amd import pbg
    pb = make_problem(op, cmp, "ranking", n=300, R=R, d=24, m=2000, seed=41)
    gm = GpuModel(pb)
    try:
        for n in (2000, 333):
            src, dst = gm.src[:n].contiguous(), gm.dst[:n].contiguous()
            rel = None if gm.rel_ids is None else gm.rel_ids[:n].contiguous()
            want = torch.full((n,), float("nan"), dtype=torch.float32, device="cuda")
            got = torch.full((n,), float("nan"), dtype=torch.float32, device="cuda")
            pbg.pbg_score_edges(gm.ctx, 0, 0, src, rel, dst, want)
            pbg.pbg_score_edges_noalloc(gm.ctx, 0, 0, src, rel, dst, got)
            torch.cuda.synchronize()
            w, g = want.cpu().numpy(), got.cpu().numpy()
            assert np.all(np.isfinite(g))
            assert np.array_equal(w, g), (n, float(np.max(np.abs(w - g))))
        # an id out of range: rejected, the output untouched
        bad = gm.dst[:50].clone()
        bad[7] = pb.n
        out = torch.zeros(50, dtype=torch.float32, device="cuda")
        with pytest.raises(pbg.PbgError) as ei:
            pbg.pbg_score_edges_noalloc(gm.ctx, 0, 0, gm.src[:50].contiguous(),
                                        None if gm.rel_ids is None else gm.rel_ids[:50].contiguous(), bad, out)
        assert ei.value.status_name == "INVALID_ARG"
        assert not out.cpu().numpy().any()
        # the following valid call still works (the flag is cleared per call)
        pbg.pbg_score_edges_noalloc(gm.ctx, 0, 0, gm.src[:50].contiguous(),
                                    None if gm.rel_ids is None else gm.rel_ids[:50].contiguous(),
                                    gm.dst[:50].contiguous(), out)
        assert np.all(np.isfinite(out.cpu().numpy()))
    finally:
        gm.close()


def test_noalloc_rejects_relation_matrices_beyond_the_scratch():
    from paper_1903_12287_amd import pbg
    d = 64
    R = pbg.NOALLOC_MAX_REL_FLOATS // (d * d) + 1
    ctx = pbg.pbg_bucket_init(1000, 1, R, d, "linear", "dot", "ranking")
    try:
        emb = torch.zeros(1000, d, dtype=torch.float32, device="cuda")
        G = torch.zeros(1000, dtype=torch.float32, device="cuda")
        relp = torch.zeros(R, d * d, dtype=torch.float32, device="cuda")
        relG = torch.zeros_like(relp)
        pbg.pbg_bind_partition(ctx, 0, emb, G)
        pbg.pbg_bind_relations(ctx, relp, relG)
        idx = torch.zeros(4, dtype=torch.int32, device="cuda")
        out = torch.zeros(4, dtype=torch.float32, device="cuda")
        with pytest.raises(pbg.PbgError) as ei:
            pbg.pbg_score_edges_noalloc(ctx, 0, 0, idx, idx, idx, out)
        assert ei.value.status_name == "INVALID_ARG"
    finally:
        pbg.pbg_free(ctx)
