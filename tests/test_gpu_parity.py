"""HIP path vs the CPU oracle, through the C ABI (needs an MI355X).

Tolerances (fp32 kernels against the fp64 oracle):
  * losses: relative 1e-5 of the summed absolute loss terms;
  * scores: |gpu - oracle| <= 1e-5 * sum_k |g(x)_k y_k| (plain relative error is
    meaningless for a score near zero from cancellation);
  * embeddings, accumulators and relation parameters after one step from the
    same state: 1e-5 relative to the largest magnitude of the compared array
    plus 1e-6 absolute;
  * embeddings after a whole pass of several steps: 1e-4 max abs.
"""

import numpy as np
import pytest
import torch

from oracle import pbg_oracle as O
from tests.pbg_cases import GpuModel, make_problem, oracle_model, teacher_forced_step

pytestmark = pytest.mark.gpu

COMBOS = [
    ("identity", "dot", "ranking"),
    ("identity", "dot", "logistic"),
    ("identity", "dot", "softmax"),
    ("identity", "cos", "ranking"),
    ("translation", "dot", "ranking"),
    ("translation", "cos", "ranking"),
    ("translation", "cos", "softmax"),
    ("diagonal", "dot", "ranking"),
    ("diagonal", "dot", "logistic"),
    ("diagonal", "cos", "logistic"),
    ("complex_diagonal", "dot", "softmax"),
    ("complex_diagonal", "dot", "ranking"),
    ("complex_diagonal", "cos", "softmax"),
    ("linear", "dot", "logistic"),
    ("linear", "dot", "ranking"),
    ("linear", "dot", "softmax"),
    ("linear", "cos", "ranking"),
    ("linear", "cos", "logistic"),
    ("linear", "cos", "softmax"),
]


def _R_for(op, cmp):
    # cos with an operator takes one relation (several are UNSUPPORTED)
    return 1 if (cmp == "cos" and op != "identity") else 3


@pytest.mark.parametrize("op,cmp,loss", [("linear", "dot", "ranking"), ("linear", "dot", "logistic")])
def test_linear_single_relation_one_step(op, cmp, loss):
    """The linear operator with one relation (contractions over the whole
    step) next to the several-relation path the combinations above take."""
    pb = make_problem(op, cmp, loss, R=1, m=95, C=20, U=12, S=8, seed=31)
    gm = GpuModel(pb)
    try:
        gl = gm.train()
        st = gm.state()
    finally:
        gm.close()
    om = oracle_model(pb)
    ol = O.train_bucket(om, pb.i, pb.j, pb.src, pb.rel_ids, pb.dst, pb.C, pb.U, pb.S, pb.lr, pb.seed)
    assert abs(gl - ol) <= 1e-5 * max(1.0, abs(ol)), (gl, ol)
    for key, ref in (("G", om.G[0]), ("emb", om.emb[0])):
        ok, err = _close(st[key][0], ref)
        assert ok, (key, err)
    ok, err = _close(st["rel"], om.rel)
    assert ok, ("rel", err)


@pytest.mark.parametrize("op,cmp,loss,d,C,U", [("translation", "dot", "logistic", 24, 20, 12),
                                               ("complex_diagonal", "dot", "ranking", 20, 20, 12),
                                               ("diagonal", "dot", "softmax", 19, 13, 9),
                                               ("complex_diagonal", "cos", "ranking", 36, 20, 12),
                                               ("diagonal", "cos", "softmax", 130, 37, 29)])
def test_single_relation_sums_match_oracle(op, cmp, loss, d, C, U):
    """One relation: each block of the operator backward adds its rows of the
    parameter gradient (edges, and with cos the uniform source candidates),
    then fixed pieces per chunk are added; ragged chunks and blocks with idle
    waves included.  Relation parameters, embeddings and Adagrad state."""
    pb = make_problem(op, cmp, loss, R=1, d=d, m=95, C=C, U=U, S=3, seed=37)
    gm = GpuModel(pb)
    try:
        gl = gm.train()
        st = gm.state()
    finally:
        gm.close()
    om = oracle_model(pb)
    ol = O.train_bucket(om, pb.i, pb.j, pb.src, pb.rel_ids, pb.dst, pb.C, pb.U, pb.S, pb.lr, pb.seed)
    assert abs(gl - ol) <= 1e-5 * max(1.0, abs(ol)), (gl, ol)
    for key, ref in (("G", om.G[0]), ("emb", om.emb[0])):
        ok, err = _close(st[key][0], ref)
        assert ok, (key, err)
    ok, err = _close(st["rel"], om.rel)
    assert ok, ("rel", err)
    ok, err = _close(st["relG"], om.relG)
    assert ok, ("relG", err)


def _close(gpu, ref, rel=1e-5, abs_=1e-6):
    scale = max(1.0, float(np.max(np.abs(ref)))) if ref.size else 1.0
    err = float(np.max(np.abs(gpu - ref))) if ref.size else 0.0
    return err <= rel * scale + abs_, err


@pytest.mark.parametrize("op,cmp,loss", COMBOS)
def test_one_step_matches_oracle(op, cmp, loss):
    """A single step (all chunks of the call in one step) from the same state."""
    pb = make_problem(op, cmp, loss, R=_R_for(op, cmp), m=95, C=20, U=12, S=8, seed=3)
    gm = GpuModel(pb)
    try:
        gl = gm.train()
        st = gm.state()
    finally:
        gm.close()
    om = oracle_model(pb)
    ol = O.train_bucket(om, pb.i, pb.j, pb.src, pb.rel_ids, pb.dst, pb.C, pb.U, pb.S, pb.lr, pb.seed)
    assert abs(gl - ol) <= 1e-5 * max(1.0, abs(ol)), (gl, ol)
    ok, err = _close(st["G"][0], om.G[0])
    assert ok, ("G", err)
    ok, err = _close(st["emb"][0], om.emb[0])
    assert ok, ("emb", err)
    if om.rel is not None:
        ok, err = _close(st["rel"], om.rel)
        assert ok, ("rel", err)
        ok, err = _close(st["relG"], om.relG)
        assert ok, ("relG", err)


@pytest.mark.parametrize("op,cmp,loss,C,U", [
    ("translation", "cos", "ranking", 1, 12),
    ("complex_diagonal", "dot", "softmax", 1, 9),
    ("diagonal", "dot", "logistic", 1, 1),
    ("identity", "dot", "ranking", 2, 0),
])
def test_unbatched_and_minimal_chunks_match_oracle(op, cmp, loss, C, U):
    """One-edge chunks (every edge against its own uniform draws: the
    unbatched negatives of Sec. 4.3) and the smallest chunk_size + num_uniform
    = 2, over several steps."""
    pb = make_problem(op, cmp, loss, R=_R_for(op, cmp), m=37, C=C, U=U, S=8, seed=29)
    gm = GpuModel(pb)
    try:
        gl = gm.train()
        st = gm.state()
    finally:
        gm.close()
    om = oracle_model(pb)
    ol = O.train_bucket(om, pb.i, pb.j, pb.src, pb.rel_ids, pb.dst, pb.C, pb.U, pb.S, pb.lr, pb.seed)
    assert abs(gl - ol) <= 1e-5 * max(1.0, abs(ol)), (gl, ol)
    for key, ref in (("G", om.G[0]), ("emb", om.emb[0])):
        ok, err = _close(st[key][0], ref)
        assert ok, (key, err)
    if om.rel is not None:
        ok, err = _close(st["rel"], om.rel)
        assert ok, ("rel", err)


@pytest.mark.parametrize("op,cmp,loss", COMBOS)
def test_score_edges_matches_oracle(op, cmp, loss):
    from paper_1903_12287_amd import pbg
    pb = make_problem(op, cmp, loss, R=_R_for(op, cmp), m=257, seed=5)
    gm = GpuModel(pb)
    try:
        out = torch.empty(pb.src.shape[0], dtype=torch.float32, device="cuda")
        pbg.pbg_score_edges(gm.ctx, 0, 0, gm.src, gm.rel_ids, gm.dst, out)
        got = out.cpu().numpy().astype(np.float64)
    finally:
        gm.close()
    om = oracle_model(pb)
    want = O.score_edges(om, 0, 0, pb.src, pb.rel_ids, pb.dst)
    scale = np.array([max(1.0, float(np.sum(np.abs(pb.parts[0][s] * pb.parts[0][t]))))
                      for s, t in zip(pb.src, pb.dst)])
    assert np.all(np.abs(got - want) <= 1e-5 * scale)


BF16_COMBOS = [
    ("translation", "cos", "ranking"),
    ("identity", "dot", "logistic"),
    ("complex_diagonal", "dot", "softmax"),
    ("diagonal", "dot", "ranking"),
    ("linear", "dot", "logistic"),
    ("linear", "cos", "ranking"),
    ("translation", "dot", "softmax"),
]


def _check_bf16_step(gm):
    """bf16 bar (2e-2), element by element, on one step from the same state
    (teacher_forced_step with eps = 2e-2): hinge terms within 2e-2 * A of the
    kink may take the other branch (counted, and followed by the oracle), the
    step loss within 2e-2 relative, and every embedding, accumulator and
    relation element within the Adagrad-propagated bound of a gradient error
    of 2e-2 * A per element."""
    rep, gl, ol, worst = teacher_forced_step(gm, 0, gm.pb.src.shape[0], 0, 2e-2)
    print(f"census {rep}, loss gpu {gl:.7g} oracle {ol:.7g}, worst error / bound {worst:.3f}", flush=True)
    assert abs(gl - ol) <= 2e-2 * abs(ol), (gl, ol)
    assert worst <= 1.0


@pytest.mark.parametrize("op,cmp,loss", BF16_COMBOS)
def test_bf16_score_path_one_step(op, cmp, loss):
    """bf16 inputs to the three contractions, fp32 accumulation, one step."""
    from paper_1903_12287_amd import pbg
    pb = make_problem(op, cmp, loss, R=_R_for(op, cmp), m=150, C=40, U=24, S=8, seed=13, d=48)
    gm = GpuModel(pb, flags=pbg.F_BF16_SCORE)
    try:
        _check_bf16_step(gm)
    finally:
        gm.close()


def test_bf16_short_chunks_and_ragged_dims():
    """Chunk and candidate counts that are not multiples of the 32-wide bf16
    k-steps, a dim that is not a multiple of 32, and a short last chunk."""
    from paper_1903_12287_amd import pbg
    pb = make_problem("diagonal", "dot", "logistic", R=2, m=77, C=19, U=13, S=5, seed=17, d=37)
    gm = GpuModel(pb, flags=pbg.F_BF16_SCORE)
    try:
        _check_bf16_step(gm)
    finally:
        gm.close()
