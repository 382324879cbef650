"""Training-step parity at the workloads' real shapes (chunk 1,000 edges,
1,000 uniform negatives per side, 40 chunks per step, the configured dim,
operator, comparator, loss and relation count), on entity tables with fewer
rows than the full graphs where the oracle's memory requires it.

Teacher-forced per step: the GPU trains the first steps freely from the
configured initial state (N(0, 0.001) embeddings, relation parameters at the
operator's identity); then for each checked step the oracle is loaded with
the GPU's step-start state (embeddings, Adagrad accumulators, relation
parameters) and computes the step's loss and gradient in fp64.  The GPU's
step loss must be within 1e-5 relative, and every parameter and accumulator
after the step within the bound that a gradient error of 1e-5 * A per
element implies through the Adagrad update (A: the gradient element formed
from absolute values, the scale of float32 summation error; see
gradient_scales), plus float32 rounding of the stored value.  Rows the step
does not touch must be unchanged.

For the ranking loss a hinge whose argument margin - p + n lies within the
float32 score error of the kink may take the other branch on the GPU.  Before
each checked step, pbg_inspect_step exposes the GPU's branch of every hinge
term; the census counts the terms within the error band of the kink and the
flips (terms whose GPU branch differs from the fp64 one), every flip must lie
inside the band, and the oracle's step then takes the GPU's branch for the
flipped terms (side_loss `active`), so the rest of the step is compared
exactly.  Smooth losses (logistic, softmax) need no hinge census; a
free-running prefix of whole steps is compared at 1e-4 max abs (with the
census of first-touch relation elements described there).
"""

import numpy as np
import pytest
import torch

from oracle import pbg_oracle as O
from paper_1903_12287_amd import synth
from tests.pbg_cases import GpuModel, Problem, oracle_model, oracle_step_with_scales, teacher_forced_step

pytestmark = pytest.mark.gpu

# (op, cmp, loss, d, R, n, P, (i, j), C, U, src zipf, dst zipf, rel zipf)
CONFIGS = {
    "tiny_social": ("identity", "dot", "ranking", 32, 1, 10_000, 1, (0, 0), 100, 100, 1.1, 1.1, None),
    "social_network": ("translation", "cos", "ranking", 128, 1, 100_000, 1, (0, 0), 1000, 1000, 1.05, 1.05, None),
    "knowledge_graph": ("complex_diagonal", "dot", "softmax", 400, 1345, 15_000, 1, (0, 0), 1000, 1000, 1.0, 1.0, 1.2),
    # bucket (3, 7) with partition 7 the short last one
    "big_bucket": ("diagonal", "dot", "ranking", 100, 5000, 8 * 25_000 - 1_234, 8, (3, 7), 1000, 1000, 1.0, 1.0, 1.3),
    "follower": ("linear", "dot", "logistic", 100, 1, 8 * 25_000 - 777, 8, (5, 2), 1000, 1000, 1.2, 0.9, None),
}
S = 40


def make_config(name, m, seed=20190010, chunking="consecutive"):
    op, cmp, loss, d, R, n, P, (i, j), C, U, zs, zd, zr = CONFIGS[name]
    rng = synth.rng_for(seed)
    rows = [O.partition_rows(n, P, p) for p in range(P)]
    parts = synth.partition_embeddings(rows, d, rng, 1e-3)
    src = synth.BoundedZipf(rows[i], zs, rng).sample(rng, m)
    dst = synth.BoundedZipf(rows[j], zd, rng).sample(rng, m)
    rel = None if R == 1 else synth.BoundedZipf(R, zr, rng).sample(rng, m).astype(np.int32)
    relp = synth.identity_relation_params(op, R, d)
    if chunking == "by_relation":
        order = np.argsort(rel, kind="stable")
        src, rel, dst = src[order], rel[order], dst[order]
    return Problem(n, P, R, d, op, cmp, loss, 0.1, parts, relp, i, j, src, rel, dst, C, U, S, 0.1, seed + 1,
                   chunking)


def _model_from(pb, st):
    return O.Model.create(pb.n, pb.P, pb.R, pb.d, pb.op, pb.cmp, pb.loss, pb.margin, st["emb"],
                          st.get("rel"), G_parts=st["G"], relG=st.get("relG"))


def _step_edges(pb, t):
    """Edges [lo, hi) of step t (S chunks of the call's chunking)."""
    ch = O.make_chunks(len(pb.src), pb.C, pb.rel_ids, pb.chunking)
    lo, hi = ch[t * S][1], ch[min(len(ch), (t + 1) * S) - 1][2]
    rel = None if pb.rel_ids is None else pb.rel_ids[lo:hi]
    return lo, hi, pb.src[lo:hi], rel, pb.dst[lo:hi]


def _oracle_step(pb, om, t):
    lo, hi, src, rel, dst = _step_edges(pb, t)
    return oracle_step_with_scales(pb, om, src, rel, dst, t * S)


@pytest.mark.parametrize("name,warm,forced,chunking", [("tiny_social", 3, 2, "consecutive"),
                                                       ("social_network", 2, 2, "consecutive"),
                                                       ("knowledge_graph", 1, 1, "consecutive"),
                                                       ("knowledge_graph", 1, 1, "by_relation"),
                                                       ("big_bucket", 2, 2, "consecutive"),
                                                       ("follower", 2, 2, "consecutive")])
def test_teacher_forced_steps(name, warm, forced, chunking):
    C = CONFIGS[name][8]
    per = S * C
    m = (warm + forced) * per
    pb = make_config(name, m, chunking=chunking)
    print(f"\n[{name}] C={pb.C} U={pb.U} S={S} d={pb.d} R={pb.R} P={pb.P} bucket=({pb.i},{pb.j}) "
          f"warm={warm} forced={forced} chunking={chunking}", flush=True)
    gm = GpuModel(pb)
    try:
        gm.train(0, _step_edges(pb, warm)[0], 0)
        for t in range(warm, warm + forced):
            lo, hi = _step_edges(pb, t)[:2]
            rep, gl, ol, worst = teacher_forced_step(gm, lo, hi, t * S, 1e-5)
            if rep is not None:
                print(f"  step {t} census: {rep['near_kink']} hinge terms within the float32 error band "
                      f"of the kink, {rep['flips']} flipped", flush=True)
            print(f"  step {t} loss gpu {gl:.9g} oracle {ol:.9g}; parameters and accumulators: "
                  f"worst error / bound = {worst:.3f}", flush=True)
            assert abs(gl - ol) <= 1e-5 * abs(ol)
            assert worst <= 1.0
    finally:
        gm.close()


@pytest.mark.parametrize("name,steps", [("follower", 3), ("knowledge_graph", 2)])
def test_free_running_prefix(name, steps):
    """Smooth losses: whole steps from the configured initial state on both
    sides, each side on its own state; the embeddings are compared at 1e-4
    max abs.

    An element touched for the first time moves by exactly lr * sign(g)
    (element-wise Adagrad on relations), so an element whose gradient lies
    within float32 rounding of zero may move the other way on the GPU: the
    census counts the first-touch relation elements with |g| <= 1e-5 A, every
    sign that differs must be one of them, and the oracle then takes the
    GPU's value for it, as it takes the GPU's branch of a hinge at its kink.

    Relation parameters are reported, not bounded, here: the element-wise
    update lr * g / sqrt(G + g^2) of an element whose gradients are small
    sums of many terms is as sensitive as A / |g| to any difference in the
    state it is computed from, and once the two runs' states differ by
    float32 rounding such elements drift apart by much more than the
    embeddings do.  The teacher-forced test bounds every relation update from
    a common state exactly."""
    C = CONFIGS[name][8]
    m = steps * S * C
    pb = make_config(name, m, seed=20190020)
    gm = GpuModel(pb)
    om = oracle_model(pb)
    try:
        for t in range(steps):
            lo, hi, src, rel, dst = _step_edges(pb, t)
            before = gm.state()
            gl = gm.train(lo, hi, t * S)
            after = gm.state()
            G0 = None if om.relG is None else om.relG.copy()
            r0 = None if om.rel is None else om.rel.copy()
            ol, grads, rel_grad, ent_sc, rel_sc = _oracle_step(pb, om, t)
            O.adagrad_update(om, grads, rel_grad, pb.lr)
            print(f"\n[{name}] step {t}: loss gpu {gl:.9g} oracle {ol:.9g}", flush=True)
            assert abs(gl - ol) <= 1e-5 * abs(ol)
            if rel_grad is not None:
                ids, g = rel_grad
                first = G0[ids] == 0.0
                near = first & (np.abs(g) <= 1e-5 * rel_sc[1])
                d_gpu = after["rel"][ids] - before["rel"][ids]
                d_orc = om.rel[ids] - r0[ids]
                flip = first & (np.sign(d_gpu) != np.sign(d_orc))
                print(f"  census: {int(near.sum())} first-touch relation elements with |g| within the float32 "
                      f"error band of 0, {int(flip.sum())} moved the other way", flush=True)
                assert not (flip & ~near).any()
                rows, cols = np.nonzero(flip)
                om.rel[ids[rows], cols] = after["rel"][ids[rows], cols]
                om.relG[ids[rows], cols] = after["relG"][ids[rows], cols]
        st = gm.state()
    finally:
        gm.close()
    for p in sorted({pb.i, pb.j}):
        err = float(np.max(np.abs(st["emb"][p] - om.emb[p])))
        print(f"  emb[{p}] max abs err {err:.3e}", flush=True)
        assert err <= 1e-4
    if om.rel is not None:
        diff = np.abs(st["rel"] - om.rel)
        print(f"  relation parameters (reported): max abs err {float(diff.max()):.3e}, "
              f"{int((diff > 1e-4).sum())} of {diff.size} elements above 1e-4", flush=True)
