"""Training-pass parity, determinism, split calls and error paths on the GPU.

Tolerances: see test_gpu_parity.py.  A free-running pass over several steps
is compared at 1e-4 max abs.  These passes are small (a few hundred hinge
terms per step), where a ranking hinge within float32 rounding of its kink
is unlikely; the workload-shaped steps of test_gpu_configs run the hinge
census and follow the GPU's branch of every term inside the rounding band.
"""

import numpy as np
import pytest
import torch

from oracle import pbg_oracle as O
from paper_1903_12287_amd import synth
from tests.pbg_cases import GpuModel, make_problem, oracle_model

pytestmark = pytest.mark.gpu


def test_negatives_bit_exact():
    from paper_1903_12287_amd import pbg
    for (n, P, i, j, U, first, nch, seed) in [(10_000, 1, 0, 0, 100, 0, 50, 20190001),
                                              (121_216_723, 16, 3, 7, 1000, 9000, 8, 20190004),
                                              (41_652_230, 8, 5, 2, 1000, 123456, 4, 2**63 + 12345),
                                              (97, 2, 1, 0, 7, 3, 11, 0)]:
        ctx = pbg.pbg_bucket_init(n, P, 1, 8, "identity", "dot", "ranking")
        try:
            out = torch.empty(nch * 2 * U, dtype=torch.int32, device="cuda")
            pbg.pbg_sample_negatives(ctx, i, j, first, nch, U, seed, out)
            got = out.cpu().numpy().reshape(nch, 2, U)
        finally:
            pbg.pbg_free(ctx)
        rows_i, rows_j = O.partition_rows(n, P, i), O.partition_rows(n, P, j)
        for c in range(nch):
            want0 = O.uniform_negatives(seed, i * P + j, first + c, 0, U, rows_j)
            want1 = O.uniform_negatives(seed, i * P + j, first + c, 1, U, rows_i)
            assert np.array_equal(got[c, 0], want0)
            assert np.array_equal(got[c, 1], want1)


@pytest.mark.parametrize("op,cmp,loss,R,P,ij", [
    ("identity", "dot", "ranking", 1, 1, (0, 0)),
    ("translation", "cos", "ranking", 1, 1, (0, 0)),
    ("complex_diagonal", "dot", "softmax", 5, 1, (0, 0)),
    ("diagonal", "dot", "ranking", 7, 3, (1, 2)),
    ("linear", "dot", "logistic", 1, 2, (1, 1)),
    ("linear", "dot", "ranking", 5, 3, (2, 0)),
    ("linear", "cos", "softmax", 1, 2, (0, 1)),
    ("diagonal", "dot", "logistic", 4, 2, (0, 1)),
])
def test_multi_step_pass_matches_oracle(op, cmp, loss, R, P, ij):
    """Several steps with a short last chunk: per-step losses and the final state."""
    i, j = ij
    pb = make_problem(op, cmp, loss, n=150, P=P, R=R, d=24, m=437, C=16, U=10, S=3, i=i, j=j,
                      seed=7, sigma=0.2)
    gm = GpuModel(pb)
    try:
        gl = gm.train()
        from paper_1903_12287_amd import pbg
        steps = pbg.pbg_get_step_losses(gm.ctx)
        st = gm.state()
    finally:
        gm.close()
    om = oracle_model(pb)
    ol, osteps = O.train_bucket(om, i, j, pb.src, pb.rel_ids, pb.dst, pb.C, pb.U, pb.S, pb.lr,
                                pb.seed, return_steps=True)
    assert len(steps) == len(osteps) == 10      # 28 chunks in steps of 3
    for a, b in zip(steps, osteps):
        assert abs(a - b) <= 1e-4 * max(1.0, abs(b)), (a, b)
    for p in sorted({i, j}):
        err = float(np.max(np.abs(st["emb"][p] - om.emb[p])))
        assert err <= 1e-4, (p, err)
        gerr = float(np.max(np.abs(st["G"][p] - om.G[p]) / np.maximum(1.0, om.G[p])))
        assert gerr <= 1e-4, (p, gerr)
    if om.rel is not None:
        assert float(np.max(np.abs(st["rel"] - om.rel))) <= 1e-4


def test_tiny_social_full_pass():
    """The tiny social graph (10,000 nodes, 100,000 edges, d = 32, identity,
    dot, ranking 0.1, C = U = 100, S = 40, lr 0.1): one full pass."""
    w = synth.tiny_social()
    rng = synth.rng_for(w.seed + 1)
    emb = synth.init_embeddings(w.n, w.d, rng)
    from tests.pbg_cases import Problem
    pb = Problem(w.n, 1, 1, w.d, w.op, w.cmp, w.loss, w.margin, [emb], None, 0, 0,
                 w.src, None, w.dst, w.C, w.U, w.S, w.lr, w.seed)
    gm = GpuModel(pb)
    try:
        gl = gm.train()
        st = gm.state()
    finally:
        gm.close()
    om = oracle_model(pb)
    ol = O.train_bucket(om, 0, 0, w.src, None, w.dst, w.C, w.U, w.S, w.lr, w.seed)
    assert abs(gl - ol) <= 1e-4 * abs(ol), (gl, ol)
    err = float(np.max(np.abs(st["emb"][0] - om.emb[0])))
    assert err <= 1e-4, err


def test_bitwise_deterministic_and_split_calls():
    pb = make_problem("complex_diagonal", "dot", "softmax", n=120, R=6, d=20, m=300, C=16, U=8, S=2,
                      seed=9)
    states = []
    for split in (None, None, 96):
        gm = GpuModel(pb)
        try:
            if split is None:
                gm.train()
            else:
                # 96 edges = 6 chunks = 3 whole steps, then the rest from chunk 6
                gm.train(0, split, 0)
                gm.train(split, None, split // pb.C)
            states.append(gm.state())
        finally:
            gm.close()
    for s in states[1:]:
        assert np.array_equal(s["emb"][0], states[0]["emb"][0])
        assert np.array_equal(s["G"][0], states[0]["G"][0])
        assert np.array_equal(s["rel"], states[0]["rel"])


def test_out_of_range_ids_leave_parameters_untouched():
    from paper_1903_12287_amd import pbg
    pb = make_problem("diagonal", "dot", "ranking", n=50, R=3, m=64, seed=4)
    gm = GpuModel(pb)
    try:
        before = gm.state()
        bad_dst = gm.dst.clone()
        bad_dst[17] = 50
        with pytest.raises(pbg.PbgError) as ei:
            pbg.pbg_train_bucket(gm.ctx, 0, 0, gm.src, gm.rel_ids, bad_dst, 16, 8, 2, 0.1, 1)
        assert ei.value.status_name == "INVALID_ARG"
        # an id far past the table: the range check's verdict comes after the
        # sort keys are queued, whose key bits it overflows
        bad_src = gm.src.clone()
        bad_src[40] = 1 << 30
        with pytest.raises(pbg.PbgError) as ei:
            pbg.pbg_train_bucket(gm.ctx, 0, 0, bad_src, gm.rel_ids, gm.dst, 16, 8, 2, 0.1, 1)
        assert ei.value.status_name == "INVALID_ARG"
        bad_rel = gm.rel_ids.clone()
        bad_rel[3] = -1
        with pytest.raises(pbg.PbgError):
            pbg.pbg_train_bucket(gm.ctx, 0, 0, gm.src, bad_rel, gm.dst, 16, 8, 2, 0.1, 1)
        with pytest.raises(pbg.PbgError) as ei:
            pbg.pbg_train_bucket(gm.ctx, 0, 0, gm.src, None, gm.dst, 16, 8, 2, 0.1, 1)
        assert ei.value.status_name == "INVALID_ARG"
        after = gm.state()
        assert np.array_equal(before["emb"][0], after["emb"][0])
        assert np.array_equal(before["rel"], after["rel"])
        # an empty call is a no-op
        empty = torch.empty(0, dtype=torch.int32, device="cuda")
        assert pbg.pbg_train_bucket(gm.ctx, 0, 0, empty, empty, empty, 16, 8, 2, 0.1, 1) == 0.0
    finally:
        gm.close()


@pytest.mark.parametrize("op,cmp,loss,d,R", [("diagonal", "dot", "logistic", 200, 4),
                                             ("translation", "cos", "softmax", 160, 1)])
def test_long_call_crosses_sort_windows(op, cmp, loss, d, R):
    """One call of 70 steps: the sort keys of 32 steps are built and sorted
    together, so the second and third windows (slices 1..31 of each) run;
    d = 200 / 160 takes the row kernels with four floats a lane (gather,
    operator backward, segment update).  Per-step losses and the final state
    against the oracle at 1e-4 (smooth losses, no hinge kinks)."""
    C, U, S = 24, 16, 2
    m = 70 * S * C - 5                      # a short last chunk
    pb = make_problem(op, cmp, loss, n=400, R=R, d=d, m=m, C=C, U=U, S=S, seed=61, sigma=0.2)
    gm = GpuModel(pb)
    try:
        gl = gm.train()
        from paper_1903_12287_amd import pbg
        steps = pbg.pbg_get_step_losses(gm.ctx)
        st = gm.state()
    finally:
        gm.close()
    om = oracle_model(pb)
    ol, osteps = O.train_bucket(om, 0, 0, pb.src, pb.rel_ids, pb.dst, C, U, S, pb.lr, pb.seed, return_steps=True)
    assert len(steps) == len(osteps) == 70
    for a, b in zip(steps, osteps):
        assert abs(a - b) <= 1e-4 * max(1.0, abs(b)), (a, b)
    err = float(np.max(np.abs(st["emb"][0] - om.emb[0])))
    assert err <= 1e-4, err
    gerr = float(np.max(np.abs(st["G"][0] - om.G[0]) / np.maximum(1.0, om.G[0])))
    assert gerr <= 1e-4, gerr


@pytest.mark.parametrize("op,cmp,loss,R", [("translation", "cos", "ranking", 4),
                                           ("complex_diagonal", "cos", "softmax", 3),
                                           ("diagonal", "cos", "logistic", 6),
                                           ("diagonal", "dot", "logistic", 5),
                                           ("linear", "dot", "ranking", 4)])
def test_relation_grouped_chunks_match_oracle(op, cmp, loss, R):
    """Relation-grouped chunks (Sec. 4.3: batches sharing a relation type),
    edges sorted by relation: several steps of short and full chunks, cos with
    an operator and several relations included (each chunk's relation is
    applied to its source candidates)."""
    pb = make_problem(op, cmp, loss, n=150, R=R, d=24, m=437, C=16, U=10, S=3, seed=71, sigma=0.2,
                      chunking="by_relation")
    gm = GpuModel(pb)
    try:
        gl = gm.train()
        from paper_1903_12287_amd import pbg
        steps = pbg.pbg_get_step_losses(gm.ctx)
        st = gm.state()
    finally:
        gm.close()
    om = oracle_model(pb)
    ol, osteps = O.train_bucket(om, 0, 0, pb.src, pb.rel_ids, pb.dst, pb.C, pb.U, pb.S, pb.lr, pb.seed,
                                return_steps=True, chunking="by_relation")
    assert len(steps) == len(osteps)
    for a, b in zip(steps, osteps):
        assert abs(a - b) <= 1e-4 * max(1.0, abs(b)), (a, b)
    assert float(np.max(np.abs(st["emb"][0] - om.emb[0]))) <= 1e-4
    assert float(np.max(np.abs(st["rel"] - om.rel))) <= 1e-4


def test_relation_grouping_helper_and_errors():
    from paper_1903_12287_amd import pbg
    # pbg_group_by_relation is a stable sort by relation
    rng = np.random.default_rng(5)
    n, R = 100_003, 37
    src = torch.from_numpy(rng.integers(0, 1000, n).astype(np.int32)).cuda()
    dst = torch.from_numpy(rng.integers(0, 1000, n).astype(np.int32)).cuda()
    relh = rng.integers(0, R, n).astype(np.int32)
    rel = torch.from_numpy(relh).cuda()
    ctx = pbg.pbg_bucket_init(1000, 1, R, 8, "diagonal", "dot", "ranking")
    try:
        outs = [torch.empty(n, dtype=torch.int32, device="cuda") for _ in range(3)]
        pbg.pbg_group_by_relation(ctx, src, rel, dst, *outs)
        order = np.argsort(relh, kind="stable")
        assert np.array_equal(outs[0].cpu().numpy(), src.cpu().numpy()[order])
        assert np.array_equal(outs[1].cpu().numpy(), relh[order])
        assert np.array_equal(outs[2].cpu().numpy(), dst.cpu().numpy()[order])
        bad = rel.clone()
        bad[17] = R
        with pytest.raises(pbg.PbgError) as ei:
            pbg.pbg_group_by_relation(ctx, src, bad, dst, *outs)
        assert ei.value.status_name == "INVALID_ARG"
    finally:
        pbg.pbg_free(ctx)
    # cos + operator + several relations: consecutive chunks are refused, and
    # unsorted relations with relation-grouped chunks leave everything untouched
    pb = make_problem("translation", "cos", "ranking", n=60, R=3, m=80, seed=4)
    gm = GpuModel(pb)
    try:
        before = gm.state()
        with pytest.raises(pbg.PbgError) as ei:
            pbg.pbg_train_bucket(gm.ctx, 0, 0, gm.src, gm.rel_ids, gm.dst, 16, 8, 2, 0.1, 1)
        assert ei.value.status_name == "UNSUPPORTED"
        unsorted = gm.rel_ids.clone()
        unsorted[0], unsorted[1] = 2, 0
        with pytest.raises(pbg.PbgError) as ei:
            pbg.pbg_train_bucket(gm.ctx, 0, 0, gm.src, unsorted, gm.dst, 16, 8, 2, 0.1, 1, chunking="by_relation")
        assert ei.value.status_name == "INVALID_ARG"
        after = gm.state()
        assert np.array_equal(before["emb"][0], after["emb"][0]) and np.array_equal(before["rel"], after["rel"])
        ranks = torch.empty(2 * 4, dtype=torch.int32, device="cuda")
        with pytest.raises(pbg.PbgError) as ei:
            pbg.pbg_rank_eval(gm.ctx, gm.src[:4], gm.rel_ids[:4], gm.dst[:4], gm.src, gm.rel_ids, gm.dst, ranks)
        assert ei.value.status_name == "UNSUPPORTED"
    finally:
        gm.close()
    with pytest.raises(pbg.PbgError) as ei:
        pbg.pbg_bucket_init(100, 1, 3, 8, "linear", "cos", "ranking")
    assert ei.value.status_name == "UNSUPPORTED"


@pytest.mark.parametrize("op,cmp,loss,C,U", [("diagonal", "cos", "logistic", 300, 200),
                                             ("translation", "cos", "softmax", 260, 140),
                                             ("identity", "cos", "softmax", 520, 100)])
def test_shared_score_block_steps_match_oracle(op, cmp, loss, C, U):
    """Chunks of 260 to 520 edges with cos: the scores of side 1 against the
    chunk's own candidates come from side 0's full 128 x 128 tiles, transposed
    (Sec. 4.3: both sides' in-chunk negatives are the same products).  Several
    steps with a short last chunk, per-step losses and the final state against
    the oracle at 1e-4 (smooth losses)."""
    S = 2
    m = 3 * S * C - 37
    pb = make_problem(op, cmp, loss, n=3000, R=1, d=48, m=m, C=C, U=U, S=S, seed=83, sigma=0.2)
    gm = GpuModel(pb)
    try:
        gm.train()
        from paper_1903_12287_amd import pbg
        steps = pbg.pbg_get_step_losses(gm.ctx)
        st = gm.state()
    finally:
        gm.close()
    om = oracle_model(pb)
    ol, osteps = O.train_bucket(om, 0, 0, pb.src, pb.rel_ids, pb.dst, C, U, S, pb.lr, pb.seed, return_steps=True)
    assert len(steps) == len(osteps) == 3
    for a, b in zip(steps, osteps):
        assert abs(a - b) <= 1e-4 * max(1.0, abs(b)), (a, b)
    err = float(np.max(np.abs(st["emb"][0] - om.emb[0])))
    assert err <= 1e-4, err
    if "rel" in st:
        rerr = float(np.max(np.abs(st["rel"] - om.rel)))
        assert rerr <= 1e-4, rerr
