"""Element-wise parity of the forward half of a training step (the chunk score
contraction K3, its loss epilogue and the per-edge finalisation) at the
workloads' real chunk shapes, through pbg_inspect_step.

For every chunk of the inspected step and both corruption sides, each
element is compared with the oracle's fp64 value (O7 scores, O8 losses):
  * positive scores p_e: |gpu - oracle| <= 1e-5 * A_p;
  * candidate scores S[e, t]: <= tol * A[e, t], tol = 1e-5 (float32 path) or
    2e-2 (bf16 inputs), with A = sum_k |a_k| |b_k| over the factors the
    score is formed from (absolute values taken inside the operator too);
  * per-edge side losses: within the propagation of those score bounds
    through the loss (ranking: the sum of the terms' bounds; logistic: the
    bound of p plus the mean bound of the negatives; softmax: the largest
    bound plus twice that of p), plus 1e-5 relative;
  * dL/dS: ranking 0 / 1 equal to the oracle's [margin - p + n > 0] except
    for terms whose hinge lies within the score bounds of the kink (counted
    and reported as flips); logistic sigmoid(n) / K_e and softmax
    exp(n - lse) within the propagated bounds.
Edges and entities are drawn like the workloads (Zipf endpoints, Zipf
relation frequencies); embeddings are drawn at a scale where scores spread
over the hinge (N(0, 0.1)) and relation parameters are perturbed around the
identity, so that every operator term and both hinge branches occur.
"""

import numpy as np
import pytest
import torch

from oracle import pbg_oracle as O
from paper_1903_12287_amd import synth
from tests.pbg_cases import (GpuModel, Problem, check_inspection, gpu_inspect, oracle_model,
                             score_scales)

pytestmark = pytest.mark.gpu

# (op, cmp, loss, d, R, n, P, (i, j), C, U, src zipf, dst zipf, rel zipf)
SHAPES = {
    "tiny_social": ("identity", "dot", "ranking", 32, 1, 10_000, 1, (0, 0), 100, 100, 1.1, 1.1, None),
    "social_network": ("translation", "cos", "ranking", 128, 1, 100_000, 1, (0, 0), 1000, 1000, 1.05, 1.05, None),
    "knowledge_graph": ("complex_diagonal", "dot", "softmax", 400, 1345, 15_000, 1, (0, 0), 1000, 1000, 1.0, 1.0, 1.2),
    # partition 7 is the short last one: 8 * 12_500 - 1_234 entities
    "big_bucket": ("diagonal", "dot", "ranking", 100, 5000, 8 * 12_500 - 1_234, 8, (3, 7), 1000, 1000, 1.0, 1.0, 1.3),
    "follower": ("linear", "dot", "logistic", 100, 1, 8 * 12_500 - 777, 8, (5, 2), 1000, 1000, 1.2, 0.9, None),
    # d > 128 row kernels (four floats a lane), ragged tiles
    "wide_rows": ("diagonal", "dot", "logistic", 200, 7, 5_000, 1, (0, 0), 300, 260, 1.1, 1.1, 1.0),
    "translation_dot": ("translation", "dot", "softmax", 64, 9, 3_000, 2, (1, 0), 256, 300, 1.1, 1.1, 1.0),
    # relation-grouped chunks: cos with an operator and 40 relations (each
    # chunk's relation applied to its source candidates)
    "grouped_cos": ("translation", "cos", "ranking", 64, 40, 20_000, 1, (0, 0), 1000, 1000, 1.0, 1.0, 0.8),
    # cos with the value losses at chunks holding full 128-row score tiles: side
    # 1's in-chunk tiles come transposed from side 0's (shared block)
    "cos_logistic": ("diagonal", "cos", "logistic", 64, 1, 20_000, 1, (0, 0), 300, 260, 1.1, 1.1, None),
    "cos_softmax": ("translation", "cos", "softmax", 96, 1, 20_000, 1, (0, 0), 400, 300, 1.1, 1.1, None),
}
GROUPED = {"grouped_cos"}


def make_shape(name, m, sigma=0.1, seed=5):
    op, cmp, loss, d, R, n, P, (i, j), C, U, zs, zd, zr = SHAPES[name]
    rng = synth.rng_for(seed)
    rows = [O.partition_rows(n, P, p) for p in range(P)]
    parts = synth.partition_embeddings(rows, d, rng, sigma)
    src = synth.BoundedZipf(rows[i], zs, rng).sample(rng, m)
    dst = synth.BoundedZipf(rows[j], zd, rng).sample(rng, m)
    rel = None if R == 1 else synth.BoundedZipf(R, zr, rng).sample(rng, m).astype(np.int32)
    relp = synth.perturbed_relation_params(op, R, d, rng, 0.3)
    if op == "linear":
        relp = (synth.identity_relation_params(op, R, d) + 0.05 * rng.standard_normal((R, d * d))).astype(np.float32)
    chunking = "by_relation" if name in GROUPED else "consecutive"
    if chunking == "by_relation":
        order = np.argsort(rel, kind="stable")
        src, rel, dst = src[order], rel[order], dst[order]
    return Problem(n, P, R, d, op, cmp, loss, 0.1, parts, relp, i, j, src, rel, dst, C, U, 40, 0.1, seed + 99,
                   chunking)


CASES = [(name, bf16) for name in SHAPES for bf16 in (False, True)]


@pytest.mark.parametrize("name,bf16", CASES)
def test_step_forward_elementwise(name, bf16):
    from paper_1903_12287_amd import pbg
    C = SHAPES[name][8]
    m = 5 * C + C // 2 + 3          # five whole chunks and a short one
    pb = make_shape(name, m)
    print(f"\n[{name} bf16={bf16}] m={m} C={pb.C} U={pb.U} d={pb.d} R={pb.R}", flush=True)
    gm = GpuModel(pb, flags=pbg.F_BF16_SCORE if bf16 else 0)
    try:
        before = gm.state()
        gpu, gloss = gpu_inspect(gm, 0, m, 7)
        after = gm.state()
    finally:
        gm.close()
    # nothing is updated
    for p in range(pb.P):
        assert np.array_equal(before["emb"][p], after["emb"][p])
        assert np.array_equal(before["G"][p], after["G"][p])
    if "rel" in before:
        assert np.array_equal(before["rel"], after["rel"])
    om = oracle_model(pb)
    orc = O.inspect_step(om, pb.i, pb.j, pb.src, pb.rel_ids, pb.dst, pb.C, pb.U, pb.seed, 7, pb.chunking)
    scales = score_scales(om, pb.i, pb.j, pb.src, pb.rel_ids, pb.dst, pb.C, pb.U, pb.seed, 7, pb.chunking)
    rep = check_inspection(om, gpu, orc, scales, 2e-2 if bf16 else 1e-5)
    print(f"[{name} bf16={bf16}] {rep}", flush=True)
    assert rep["p_ratio"] <= 1.0 and rep["s_ratio"] <= 1.0
    assert rep["loss_ratio"] <= 1.0 and rep["ds_ratio"] <= 1.0
    ol = sum(float(o["loss0"].sum() + o["loss1"].sum()) for o in orc)
    gl_rows = sum(float(g["loss0"].sum() + g["loss1"].sum()) for g in gpu)
    assert abs(gl_rows - gloss) <= 1e-6 * abs(gloss)
    assert abs(gloss - ol) <= (2e-2 if bf16 else 1e-5) * abs(ol)
    if not bf16 and pb.loss == "ranking":
        # float32: the branch of a hinge may differ from the fp64 one only
        # within rounding of the kink, which is rare
        assert rep["flips"] <= max(5, 1e-6 * sum(o["S0"].size * 2 for o in orc))


def test_inspect_rejects_more_than_one_step():
    from paper_1903_12287_amd import pbg
    pb = make_shape("tiny_social", 250)
    pb.S = 2
    gm = GpuModel(pb)
    try:
        with pytest.raises(pbg.PbgError) as ei:
            gpu_inspect(gm, 0, 250, 0)
        assert ei.value.status_name == "INVALID_ARG"
    finally:
        gm.close()
