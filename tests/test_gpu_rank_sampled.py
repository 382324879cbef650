"""Raw ranks against sampled candidates (pbg_rank_sampled) against the oracle
(needs an MI355X).  The ranks are integers decided by float comparisons, as
for the filtered ranks: the oracle's rank bounds for scores within tol must
hold every GPU rank, and most ranks must match outright (the tolerance
argument is the one of test_gpu_rank.py)."""

import numpy as np
import pytest
import torch

from oracle import pbg_oracle as O
from paper_1903_12287_amd import synth

from test_gpu_rank import _tol

pytestmark = pytest.mark.gpu


def _gpu_sampled(n, R, d, op, cmp, emb, relp, src, rel, dst, cand):
    from paper_1903_12287_amd import pbg
    dev = torch.device("cuda")
    ctx = pbg.pbg_bucket_init(n, 1, R, d, op, cmp, "softmax")
    try:
        pbg.pbg_bind_partition(ctx, 0, torch.from_numpy(emb).to(dev), torch.zeros(n, dtype=torch.float32, device=dev))
        if relp is not None:
            rp = torch.from_numpy(relp).to(dev)
            pbg.pbg_bind_relations(ctx, rp, torch.zeros_like(rp))
        pbg.pbg_set_streams(ctx, torch.cuda.current_stream(), None)
        t = lambda a: None if a is None else torch.from_numpy(np.ascontiguousarray(a, np.int32)).to(dev)
        ranks = torch.zeros(2 * len(src), dtype=torch.int32, device=dev)
        mrr, hits = pbg.pbg_rank_sampled(ctx, t(src), t(rel), t(dst), t(cand), ranks)
        return ranks.cpu().numpy().astype(np.int64), mrr, hits
    finally:
        pbg.pbg_free(ctx)


def _check(n, R, d, op, cmp, emb, relp, src, rel, dst, cand, sample=None, min_exact=0.97):
    got, mrr, hits = _gpu_sampled(n, R, d, op, cmp, emb, relp, src, rel, dst, cand)
    assert abs(mrr - float(np.mean(1.0 / got))) <= 1e-12
    assert abs(hits - float(np.mean(got <= 10))) <= 1e-12
    model = O.Model.create(n, 1, R, d, op, cmp, "softmax", 0.1, [emb.astype(np.float64)],
                           None if relp is None else relp.astype(np.float64))
    m = len(src)
    idx = np.arange(m) if sample is None else sample
    want, _, _, lo, hi = O.rank_sampled(model, src[idx], None if rel is None else rel[idx], dst[idx], cand,
                                        tol=_tol(op, cmp, emb, relp))
    g = np.concatenate([got[idx], got[m + idx]])
    assert np.all(g >= lo) and np.all(g <= hi), np.nonzero((g < lo) | (g > hi))[0][:10]
    assert np.mean(g == want) >= min_exact
    return got


@pytest.mark.parametrize("op,cmp,R", [
    ("complex_diagonal", "dot", 7),
    ("translation", "dot", 5),
    ("linear", "dot", 1),
    ("identity", "dot", 1),
    ("translation", "cos", 1),
    ("identity", "cos", 3),
])
def test_rank_sampled_matches_oracle(op, cmp, R):
    n, d, m_train, m_eval = 300, 24, 3000, 200
    rng = synth.rng_for(61 + R)
    emb = (rng.standard_normal((n, d)) * 0.3).astype(np.float32)
    relp = synth.perturbed_relation_params(op, R, d, rng, 0.3)
    src, dst = synth.zipf_edges(n, m_train + m_eval, 1.0, 1.0, rng)
    rel = rng.integers(0, R, m_train + m_eval).astype(np.int32) if R > 1 else None
    # 1,000 candidates drawn by prevalence (repeats and the true ids included)
    cand = synth.prevalence_candidates(src[:m_train], dst[:m_train], n, 1000, rng)
    er = None if rel is None else rel[m_train:]
    _check(n, R, d, op, cmp, emb, relp, src[m_train:], er, dst[m_train:], cand)


def test_rank_sampled_edges_and_errors():
    from paper_1903_12287_amd import pbg
    n, d = 50, 8
    rng = synth.rng_for(9)
    emb = (rng.standard_normal((n, d)) * 0.3).astype(np.float32)
    src, dst = synth.zipf_edges(n, 40, 1.0, 1.0, rng)
    # one candidate; the true ids only (rank 1 on both sides); a ragged count
    for cand in (np.array([7], np.int32), np.unique(np.concatenate([src[:1], dst[:1]])).astype(np.int32),
                 rng.integers(0, n, 77).astype(np.int32)):
        got = _check(n, 1, d, "identity", "dot", emb, None, src, None, dst, cand)
        assert int(got.max()) <= len(cand) + 1
    # the true destination as the only candidate: destination rank 1
    got = _check(n, 1, d, "identity", "dot", emb, None, src[:1], None, dst[:1], np.array([dst[0]], np.int32))
    assert got[0] == 1
    dev = torch.device("cuda")
    ctx = pbg.pbg_bucket_init(n, 1, 1, d, "identity", "dot", "softmax")
    try:
        pbg.pbg_bind_partition(ctx, 0, torch.from_numpy(emb).to(dev), torch.zeros(n, dtype=torch.float32, device=dev))
        z = torch.zeros(4, dtype=torch.int32, device=dev)
        bad = torch.tensor([1, 2, n, 3], dtype=torch.int32, device=dev)
        ranks = torch.full((8,), -3, dtype=torch.int32, device=dev)
        with pytest.raises(pbg.PbgError) as ei:
            pbg.pbg_rank_sampled(ctx, z, None, z, bad, ranks)
        assert ei.value.status_name == "INVALID_ARG"
        assert bool((ranks == -3).all())
        with pytest.raises(pbg.PbgError) as ei:
            pbg.pbg_rank_sampled(ctx, z, None, z, torch.zeros(0, dtype=torch.int32, device=dev), ranks)
        assert ei.value.status_name == "INVALID_ARG"
    finally:
        pbg.pbg_free(ctx)


def test_rank_sampled_knowledge_graph_full_size():
    """15,000 entities, d = 400 complex_diagonal with dot: all 50,000
    held-out triples ranked on both sides against 10,000 prevalence-sampled
    candidates; 120 sampled triples checked against the oracle."""
    w = synth.knowledge_graph()
    rng = synth.rng_for(w.seed + 1)
    emb = (rng.standard_normal((w.n, w.d)) * 0.05).astype(np.float32)
    relp = synth.perturbed_relation_params("complex_diagonal", w.R, w.d, rng, 0.3)
    cand = synth.prevalence_candidates(w.src, w.dst, w.n, 10_000, synth.rng_for(w.seed + 2))
    sample = synth.rng_for(8).choice(len(w.held_src), 120, replace=False)
    got = _check(w.n, w.R, w.d, "complex_diagonal", "dot", emb, relp, w.held_src, w.held_rel, w.held_dst, cand,
                 sample=sample, min_exact=0.95)
    assert got.shape == (100_000,) and int(got.min()) >= 1 and int(got.max()) <= 10_001
