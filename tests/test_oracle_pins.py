"""Pins of the CPU oracle against what the paper and the mathematics fix.

Every check here compares the oracle with something other than itself: the
published Philox known-answer vectors, the paper's worked negative count,
Python big-integer and complex arithmetic, explicit per-pair loops on tiny
inputs, closed-form losses and gradients, central finite differences, the
bucketing and bucket-order invariants, and brute-force filtered ranks.
"""

import itertools
import math
import os

import numpy as np
import pytest
import torch

from oracle import pbg_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
F64 = torch.float64


# ---------------------------------------------------------------- Philox (O4)
def _read_golden(name):
    rows = []
    with open(os.path.join(GOLDEN, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                rows.append(line.split())
    return rows


def test_philox_known_answers():
    for row in _read_golden("philox4x32_10_kat.txt"):
        vals = [int(x, 16) for x in row]
        ctr, key, want = vals[0:4], vals[4:6], vals[6:10]
        got = O.philox4x32_10(np.array(ctr, np.uint64), np.array(key, np.uint64))
        assert [int(x) for x in got] == want


def test_uniform_negative_map_is_exact_floor():
    # u = floor(w * n / 2**32) in Python big integers, from the KAT-checked words
    for n_rows in (1, 2, 3, 97, 5_206_529, 7_576_046, 2**31 - 1, 2**31):
        for seed in (0, 1, 0xFFFFFFFF, 0x123456789ABCDEF0):
            U = 9
            got = O.uniform_negatives(seed, 5, 11, 1, U, n_rows)
            for k in range(U):
                words = O.philox4x32_10(np.array([k >> 2, 11, 5, 1], np.uint64),
                                        np.array([seed & 0xFFFFFFFF, seed >> 32], np.uint64))
                w = int(words[k & 3])
                want = (w * n_rows) // (1 << 32)
                assert int(got[k]) == want
                assert 0 <= want < n_rows
    # extreme words: w = 2**32 - 1 maps to n - 1 for every n
    for n_rows in (1, 2, 2**31):
        assert ((2**32 - 1) * n_rows) >> 32 == n_rows - 1


def test_uniform_negatives_are_uniform():
    n_rows, U = 97, 4096
    counts = np.zeros(n_rows)
    for chunk in range(25):
        counts += np.bincount(O.uniform_negatives(20190001, 0, chunk, 0, U, n_rows),
                              minlength=n_rows)
    expected = counts.sum() / n_rows
    chi2 = ((counts - expected) ** 2 / expected).sum()
    # 96 degrees of freedom: the 1e-6 upper quantile is about 180
    assert chi2 < 180


def test_negative_streams_differ_by_side_chunk_bucket_and_seed():
    base = O.uniform_negatives(7, 3, 4, 0, 64, 10**6)
    for args in ((7, 3, 4, 1), (7, 3, 5, 0), (7, 2, 4, 0), (8, 3, 4, 0)):
        other = O.uniform_negatives(args[0], args[1], args[2], args[3], 64, 10**6)
        assert not np.array_equal(base, other)


# -------------------------------------------------- partitions, buckets (O1, O2)
def test_partition_sizes():
    assert O.partition_size(121_216_723, 16) == 7_576_046
    assert O.partition_size(41_652_230, 8) == 5_206_529
    for n, P in ((10, 3), (121_216_723, 16), (41_652_230, 8), (7, 7), (1000, 1)):
        rows = [O.partition_rows(n, P, p) for p in range(P)]
        assert sum(rows) == n
        assert all(r == O.partition_size(n, P) for r in rows[:-1])
        assert 0 < rows[-1] <= O.partition_size(n, P)


def test_bucketing_brute_force():
    rng = np.random.default_rng(3)
    n, P, E = 10, 3, 200
    src = rng.integers(0, n, E)
    dst = rng.integers(0, n, E)
    rel = rng.integers(0, 4, E).astype(np.int32)
    offsets, sl, rl, dl = O.bucket_edges(src, rel, dst, n, P)
    # brute force: a dict of lists, filled in input order
    ps = -(-n // P)
    want = {}
    for e in range(E):
        want.setdefault((src[e] // ps, dst[e] // ps), []).append(
            (src[e] % ps, rel[e], dst[e] % ps))
    assert offsets[0] == 0 and offsets[-1] == E
    assert np.all(np.diff(offsets) >= 0)
    for i in range(P):
        for j in range(P):
            b = i * P + j
            lo, hi = offsets[b], offsets[b + 1]
            got = list(zip(sl[lo:hi].tolist(), rl[lo:hi].tolist(), dl[lo:hi].tolist()))
            assert got == [tuple(int(v) for v in t) for t in want.get((i, j), [])]
            assert np.all(sl[lo:hi] < O.partition_rows(n, P, i))
            assert np.all(dl[lo:hi] < O.partition_rows(n, P, j))
    # every edge lands in exactly one bucket, with part(src) = i and part(dst) = j
    back_src = np.concatenate([sl[offsets[i * P + j]:offsets[i * P + j + 1]] + i * ps
                               for i in range(P) for j in range(P)])
    assert sorted(back_src.tolist()) == sorted(src.tolist())


def test_bucketing_rejects_out_of_range():
    with pytest.raises(ValueError):
        O.bucket_edges([0, 10], [0, 0], [1, 2], 10, 2)


@pytest.mark.parametrize("P", [1, 2, 3, 4, 5, 8, 16])
def test_inside_out_order_invariant(P):
    order = O.inside_out_order(P)
    assert order[0] == (0, 0)
    assert sorted(order) == [(i, j) for i in range(P) for j in range(P)]
    seen = set()
    for k, (i, j) in enumerate(order):
        if k:
            assert i in seen or j in seen      # shares a partition with an earlier bucket
        seen.update((i, j))


# -------------------------------------------------------- negatives count (O7)
def test_paper_negative_count():
    (C, U, want), = [tuple(int(v) for v in r) for r in _read_golden("batched_negatives_count.txt")]
    mask = O.valid_mask(C, U)
    assert int(mask.sum().item()) * 2 == want          # two corruption sides
    assert 2 * C * (C + U) - 2 * C == want


# ------------------------------------------------ operators, comparators (O5, O6)
def test_complex_diagonal_matches_complex128():
    rng = np.random.default_rng(1)
    d = 10
    h = d // 2
    x, th, y = (rng.standard_normal(d) for _ in range(3))
    g = O.apply_operator("complex_diagonal", torch.tensor(x), torch.tensor(th)).numpy()
    xc = x[:h] + 1j * x[h:]
    tc = th[:h] + 1j * th[h:]
    yc = y[:h] + 1j * y[h:]
    prod = xc * tc
    assert np.allclose(g[:h], prod.real, rtol=0, atol=1e-14)
    assert np.allclose(g[h:], prod.imag, rtol=0, atol=1e-14)
    # the comparator's real dot on the split layout is Re <a, conj(b)>
    score = O.compare_rows("dot", torch.tensor(g)[None], torch.tensor(y)[None]).item()
    assert abs(score - np.real(np.sum(prod * np.conj(yc)))) < 1e-13


def test_linear_operator_matches_matmul():
    rng = np.random.default_rng(2)
    d = 5
    A = rng.standard_normal((d, d))
    x = rng.standard_normal(d)
    g = O.apply_operator("linear", torch.tensor(x), torch.tensor(A.reshape(-1))).numpy()
    assert np.allclose(g, A @ x, atol=1e-14)
    assert not np.allclose(g, A.T @ x)


def test_translation_and_diagonal():
    x = torch.tensor([1.0, -2.0, 3.0], dtype=F64)
    t = torch.tensor([0.5, 4.0, -1.0], dtype=F64)
    assert O.apply_operator("translation", x, t).tolist() == [1.5, 2.0, 2.0]
    assert O.apply_operator("diagonal", x, t).tolist() == [0.5, -8.0, -3.0]
    assert O.apply_operator("identity", x, None) is x


@pytest.mark.parametrize("op", O.OPERATORS)
def test_identity_parameters_reduce_to_identity(op):
    from paper_1903_12287_amd import synth
    d = 6
    x = torch.tensor(np.random.default_rng(5).standard_normal((3, d)))
    p = synth.identity_relation_params(op, 1, d)
    th = None if p is None else torch.tensor(p[0].astype(np.float64))
    assert torch.allclose(O.apply_operator(op, x, th), x, atol=0, rtol=0)


def test_cos_comparator():
    a = torch.tensor([[3.0, 4.0], [0.0, 0.0]], dtype=F64)
    b = torch.tensor([[1.0, 0.0], [0.0, -2.0]], dtype=F64)
    s = O.compare_all("cos", a, b)
    assert abs(s[0, 0].item() - 0.6) < 1e-15
    assert abs(s[0, 1].item() + 0.8) < 1e-15
    assert s[1, 0].item() == 0.0 and s[1, 1].item() == 0.0      # zero norm is clamped
    r = O.compare_rows("cos", a, b)
    assert abs(r[0].item() - 0.6) < 1e-15


# ---------------------------------------------------------- chunk scores (O7)
def _py_operator(op, x, th):
    """Explicit loops / Python complex numbers: an independent statement of g."""
    d = len(x)
    if op == "identity":
        return list(x)
    if op == "translation":
        return [x[k] + th[k] for k in range(d)]
    if op == "diagonal":
        return [x[k] * th[k] for k in range(d)]
    if op == "linear":
        return [sum(th[k * d + l] * x[l] for l in range(d)) for k in range(d)]
    h = d // 2
    z = [complex(x[k], x[h + k]) * complex(th[k], th[h + k]) for k in range(h)]
    return [v.real for v in z] + [v.imag for v in z]


def _py_sim(cmp, a, b):
    if cmp == "dot":
        return sum(u * v for u, v in zip(a, b))
    na = max(math.sqrt(sum(u * u for u in a)), 1e-12)
    nb = max(math.sqrt(sum(v * v for v in b)), 1e-12)
    return sum(u * v for u, v in zip(a, b)) / (na * nb)


@pytest.mark.parametrize("op,cmp", [(o, c) for o in O.OPERATORS for c in O.COMPARATORS])
def test_chunk_scores_brute_force(op, cmp):
    rng = np.random.default_rng(11)
    d, C, U, R = 4, 3, 2, 3
    width = O.relation_param_width(op, d)
    src_rows = rng.standard_normal((C + U, d))
    dst_rows = rng.standard_normal((C + U, d))
    rel_params = rng.standard_normal((R, max(width, 1)))
    rel_e = np.array([2, 0, 2])
    xs, xd = torch.tensor(src_rows[:C]), torch.tensor(dst_rows[:C])
    cand_dst, cand_src = torch.tensor(dst_rows), torch.tensor(src_rows)
    theta_e = None if width == 0 else torch.tensor(rel_params[rel_e])
    theta_of = (lambda r: None) if width == 0 else (lambda r: torch.tensor(rel_params[r]))
    p, S0, S1 = O.chunk_scores(op, cmp, xs, xd, theta_e, rel_e, cand_dst, cand_src, theta_of)
    for e in range(C):
        th = list(rel_params[rel_e[e]])
        ge = _py_operator(op, list(src_rows[e]), th)
        assert abs(p[e].item() - _py_sim(cmp, ge, list(dst_rows[e]))) < 1e-12
        for t in range(C + U):
            # destination corruption: f(s_e, r_e, candidate t)
            assert abs(S0[e, t].item() - _py_sim(cmp, ge, list(dst_rows[t]))) < 1e-12
            # source corruption: f(candidate t, r_e, d_e)
            gt = _py_operator(op, list(src_rows[t]), th)
            assert abs(S1[e, t].item() - _py_sim(cmp, gt, list(dst_rows[e]))) < 1e-12


def test_identity_dot_scores_are_a_product():
    rng = np.random.default_rng(4)
    xs, xd = torch.tensor(rng.standard_normal((5, 3))), torch.tensor(rng.standard_normal((5, 3)))
    p, S0, S1 = O.chunk_scores("identity", "dot", xs, xd, None, np.zeros(5, int), xd, xs,
                               lambda r: None)
    assert np.allclose(S0.numpy(), xs.numpy() @ xd.numpy().T, atol=1e-14)
    assert np.allclose(S1.numpy(), xd.numpy() @ xs.numpy().T, atol=1e-14)
    assert np.allclose(np.diag(S0.numpy()), p.numpy())


# ----------------------------------------------------------------- losses (O8)
def _single_edge_losses(loss, p, n0, n1, margin=0.1):
    """C = 1, U = 1: the only valid negative on each side is the uniform one."""
    pt = torch.tensor([p], dtype=F64)
    valid = O.valid_mask(1, 1)
    assert valid.tolist() == [[0.0, 1.0]]
    S0 = torch.tensor([[123.0, n0]], dtype=F64)     # the masked diagonal must not matter
    S1 = torch.tensor([[-77.0, n1]], dtype=F64)
    return (O.side_loss(loss, margin, pt, S0, valid).item(),
            O.side_loss(loss, margin, pt, S1, valid).item())


def test_loss_closed_forms_single_edge():
    p, n0, n1, lam = 0.3, 0.35, -0.9, 0.1
    a, b = _single_edge_losses("ranking", p, n0, n1, lam)
    assert abs(a - max(0.0, lam - p + n0)) < 1e-15 and abs(b - max(0.0, lam - p + n1)) < 1e-15
    a, b = _single_edge_losses("softmax", p, n0, n1)
    assert abs(a - math.log1p(math.exp(n0 - p))) < 1e-15
    assert abs(b - math.log1p(math.exp(n1 - p))) < 1e-15
    a, b = _single_edge_losses("logistic", p, n0, n1)
    sp = lambda v: math.log1p(math.exp(v))
    assert abs(a - (sp(-p) + sp(n0))) < 1e-15 and abs(b - (sp(-p) + sp(n1))) < 1e-15


def test_ranking_sign_penalises_high_negatives():
    # f is maximised on true edges: a negative scored above the positive costs more
    lo, _ = _single_edge_losses("ranking", 1.0, -1.0, -1.0)
    hi, _ = _single_edge_losses("ranking", 1.0, 2.0, -1.0)
    assert lo == 0.0 and hi > 1.0


def test_logistic_averages_negatives_over_k():
    p = torch.tensor([0.2], dtype=F64)
    S = torch.tensor([[9.0, 0.5, -0.25]], dtype=F64)      # C = 1, U = 2: K_e = 2
    L = O.side_loss("logistic", 0.1, p, S, O.valid_mask(1, 2)).item()
    sp = lambda v: math.log1p(math.exp(v))
    assert abs(L - (sp(-0.2) + 0.5 * (sp(0.5) + sp(-0.25)))) < 1e-15


@pytest.mark.parametrize("loss", O.LOSSES)
def test_losses_invariant_to_negative_order(loss):
    rng = np.random.default_rng(9)
    C, U = 4, 5
    p = torch.tensor(rng.standard_normal(C))
    S = torch.tensor(rng.standard_normal((C, C + U)))
    v = O.valid_mask(C, U)
    base = O.side_loss(loss, 0.1, p, S, v)
    perm = np.concatenate([np.arange(C), C + rng.permutation(U)])
    assert torch.allclose(O.side_loss(loss, 0.1, p, S[:, perm], v), base, atol=1e-14, rtol=0)


def test_softmax_gradient_closed_form():
    p = torch.tensor([0.4, -0.2], dtype=F64, requires_grad=True)
    S = torch.tensor([[0.0, 0.3, 1.1, -0.5], [2.0, 0.0, 0.1, 0.7]], dtype=F64, requires_grad=True)
    v = O.valid_mask(2, 2)
    O.side_loss("softmax", 0.1, p, S, v).sum().backward()
    for e in range(2):
        logits = [p[e].item()] + [S[e, t].item() for t in range(4) if t != e]
        z = sum(math.exp(x) for x in logits)
        sm = [math.exp(x) / z for x in logits]
        assert abs(p.grad[e].item() - (sm[0] - 1.0)) < 1e-14
        cols = [t for t in range(4) if t != e]
        for k, t in enumerate(cols):
            assert abs(S.grad[e, t].item() - sm[k + 1]) < 1e-14
        assert S.grad[e, e].item() == 0.0


# ----------------------------------------------- step gradient, Adagrad (O9, O10)
def _tiny_model(op, cmp, loss, n=9, P=2, R=2, d=4, seed=0, scale=0.5, margin=0.1):
    rng = np.random.default_rng(seed)
    parts = [rng.standard_normal((O.partition_rows(n, P, p), d)) * scale for p in range(P)]
    width = O.relation_param_width(op, d)
    relp = None if width == 0 else rng.standard_normal((R, width)) * 0.5 + (
        np.eye(d).reshape(-1) if op == "linear" else 0.0)
    return O.Model.create(n, P, R, d, op, cmp, loss, margin, parts, relp)


def _tiny_edges(model, i, j, m, seed):
    rng = np.random.default_rng(seed + 100)
    src = rng.integers(0, model.emb[i].shape[0], m)
    dst = rng.integers(0, model.emb[j].shape[0], m)
    rel = rng.integers(0, model.R, m)
    return src, rel, dst


def _near_kink(model, i, j, src, rel, dst, step, negs):
    """Smallest |margin - p + n| over the step's valid ranking pairs."""
    worst = np.inf
    for (c, lo, hi), (u_dst, u_src) in zip(step, negs):
        xs = torch.tensor(model.emb[i][src[lo:hi]])
        xd = torch.tensor(model.emb[j][dst[lo:hi]])
        cd = torch.cat([xd, torch.tensor(model.emb[j][u_dst])])
        cs = torch.cat([xs, torch.tensor(model.emb[i][u_src])])
        th = None if model.rel is None else torch.tensor(model.rel[rel[lo:hi]])
        tof = (lambda r: None) if model.rel is None else (lambda r: torch.tensor(model.rel[r]))
        p, S0, S1 = O.chunk_scores(model.op, model.cmp, xs, xd, th, rel[lo:hi], cd, cs, tof)
        v = O.valid_mask(hi - lo, len(u_dst)).bool()
        for S in (S0, S1):
            z = (model.margin - p[:, None] + S)[v]
            worst = min(worst, float(z.abs().min()))
    return worst


COMBOS = [(o, c, l) for o in O.OPERATORS for c in O.COMPARATORS for l in O.LOSSES]


@pytest.mark.parametrize("op,cmp,loss", COMBOS)
@pytest.mark.parametrize("bucket", [(0, 1), (1, 1)])
def test_step_gradient_matches_finite_differences(op, cmp, loss, bucket):
    i, j = bucket
    R = 1 if (cmp == "cos" and op != "identity") else 2
    for seed in range(20):
        model = _tiny_model(op, cmp, loss, R=R, seed=seed)
        src, rel, dst = _tiny_edges(model, i, j, 7, seed)
        step = O.chunk_ranges(7, 3)[:2] + [(2, 6, 7)]     # chunks of 3, 3 and a short 1
        negs = O.step_negatives(model, i, j, step, seed + 5, 2)
        if loss != "ranking" or _near_kink(model, i, j, src, rel, dst, step, negs) > 1e-3:
            break
    loss0, grads, rel_grad = O.step_loss_and_grad(model, i, j, src, rel, dst, step, negs)
    h = 1e-6

    def f():
        return O.step_loss_and_grad(model, i, j, src, rel, dst, step, negs, with_grad=False)[0]

    checked = 0
    for p, (ids, g) in grads.items():
        for a, row in enumerate(ids):
            for k in range(model.d):
                keep = model.emb[p][row, k]
                model.emb[p][row, k] = keep + h
                up = f()
                model.emb[p][row, k] = keep - h
                dn = f()
                model.emb[p][row, k] = keep
                fd = (up - dn) / (2 * h)
                assert abs(fd - g[a, k]) <= 1e-6 * max(1.0, abs(g[a, k])), (p, row, k, fd, g[a, k])
                checked += 1
    if rel_grad is not None:
        ids, g = rel_grad
        for a, r in enumerate(ids):
            for k in range(model.rel.shape[1]):
                keep = model.rel[r, k]
                model.rel[r, k] = keep + h
                up = f()
                model.rel[r, k] = keep - h
                dn = f()
                model.rel[r, k] = keep
                fd = (up - dn) / (2 * h)
                assert abs(fd - g[a, k]) <= 1e-6 * max(1.0, abs(g[a, k])), ("rel", r, k, fd, g[a, k])
                checked += 1
    assert checked > 0


def test_ranking_gradient_one_active_pair():
    """identity + dot, one edge (s, d), uniform negatives d' and s': with only the
    destination-side hinge active, dL/ds = x_d' - x_d, dL/dd = -x_s, dL/dd' = x_s."""
    n, d = 8, 3
    for seed in range(1000):
        u_dst = int(O.uniform_negatives(seed, 0, 0, 0, 1, n)[0])
        u_src = int(O.uniform_negatives(seed, 0, 0, 1, 1, n)[0])
        if len({0, 1, u_dst, u_src}) == 4:
            break
    E = np.zeros((n, d))
    E[0] = [1.0, 0.5, 0.0]       # s
    E[1] = [0.2, 0.1, 0.0]       # d
    E[u_dst] = [0.3, -0.2, 0.4]  # d': lambda - <s,d> + <s,d'> = 0.1 - 0.25 + 0.2 > 0
    E[u_src] = [-5.0, 0.0, 1.0]  # s': lambda - <s,d> + <s',d> = 0.1 - 0.25 - 1.0 < 0
    model = O.Model.create(n, 1, 1, d, "identity", "dot", "ranking", 0.1, [E])
    step = O.chunk_ranges(1, 1)
    negs = O.step_negatives(model, 0, 0, step, seed, 1)
    loss, grads, _ = O.step_loss_and_grad(model, 0, 0, np.array([0]), np.array([0]),
                                          np.array([1]), step, negs)
    assert abs(loss - (0.1 - 0.25 + 0.2)) < 1e-15
    ids, g = grads[0]
    gd = {int(r): g[k] for k, r in enumerate(ids)}
    assert np.allclose(gd[0], E[u_dst] - E[1], atol=1e-15)
    assert np.allclose(gd[1], -E[0], atol=1e-15)
    assert np.allclose(gd[u_dst], E[0], atol=1e-15)
    assert np.allclose(gd[u_src], 0.0, atol=0)


def test_adagrad_closed_form():
    n, d, lr = 8, 3, 0.1
    rng = np.random.default_rng(0)
    E = rng.standard_normal((n, d))
    model = O.Model.create(n, 1, 1, d, "identity", "dot", "logistic", 0.1, [E.copy()])
    step = O.chunk_ranges(2, 2)
    src, dst, rel = np.array([0, 2]), np.array([1, 3]), np.array([0, 0])
    negs = O.step_negatives(model, 0, 0, step, 4, 2)
    _, g1, _ = O.step_loss_and_grad(model, 0, 0, src, rel, dst, step, negs)
    O.adagrad_update(model, g1, None, lr)
    ids, g = g1[0]
    for k, r in enumerate(ids):
        norm = np.linalg.norm(g[k])
        moved = np.linalg.norm(model.emb[0][r] - E[r])
        assert abs(moved - lr * norm / (norm + O.EPS_ADAGRAD)) < 1e-14
        assert abs(model.G[0][r] - norm ** 2) < 1e-15 * max(1, norm ** 2)
    # second step: the accumulator holds |g1|^2 + |g2|^2
    before = model.emb[0].copy()
    _, g2, _ = O.step_loss_and_grad(model, 0, 0, src, rel, dst, step, negs)
    G_before = model.G[0].copy()
    O.adagrad_update(model, g2, None, lr)
    ids2, gg = g2[0]
    for k, r in enumerate(ids2):
        G = G_before[r] + np.sum(gg[k] ** 2)
        assert abs(model.G[0][r] - G) < 1e-14
        assert np.allclose(model.emb[0][r], before[r] - lr * gg[k] / (np.sqrt(G) + 1e-10), atol=1e-15)


def test_relation_adagrad_is_elementwise():
    model = _tiny_model("diagonal", "dot", "logistic", P=1, n=6, R=2, seed=3)
    th0 = model.rel.copy()
    src, rel, dst = np.array([0, 1, 2]), np.array([1, 1, 1]), np.array([3, 4, 5])
    step = O.chunk_ranges(3, 3)
    negs = O.step_negatives(model, 0, 0, step, 1, 2)
    _, grads, (rids, rg) = O.step_loss_and_grad(model, 0, 0, src, rel, dst, step, negs)
    O.adagrad_update(model, grads, (rids, rg), 0.05)
    assert list(rids) == [1]
    want = th0[1] - 0.05 * rg[0] / (np.abs(rg[0]) + 1e-10)
    assert np.allclose(model.rel[1], want, atol=1e-15)
    assert np.array_equal(model.rel[0], th0[0])           # untouched relation


def test_step_gradient_is_taken_at_step_start():
    """With S = 2 the two chunks' gradients are both evaluated before any update
    (one Adagrad step with their sum); with S = 1 the second chunk sees the
    first chunk's update."""
    def run(S):
        model = _tiny_model("translation", "dot", "softmax", P=1, n=6, R=1, seed=8)
        src, dst = np.array([0, 1, 2, 0]), np.array([1, 2, 3, 4])
        O.train_bucket(model, 0, 0, src, None, dst, 2, 2, S, 0.1, 9)
        return model
    m2 = run(2)
    ref = _tiny_model("translation", "dot", "softmax", P=1, n=6, R=1, seed=8)
    step = O.chunk_ranges(4, 2)
    negs = O.step_negatives(ref, 0, 0, step, 9, 2)
    src, dst, rel = np.array([0, 1, 2, 0]), np.array([1, 2, 3, 4]), np.zeros(4, int)
    _, ga, ra = O.step_loss_and_grad(ref, 0, 0, src, rel, dst, step[:1], negs[:1])
    _, gb, rb = O.step_loss_and_grad(ref, 0, 0, src, rel, dst, step[1:], negs[1:])
    tot = {}
    for gg in (ga, gb):
        for p, (ids, g) in gg.items():
            for k, r in enumerate(ids):
                tot[int(r)] = tot.get(int(r), 0.0) + g[k]
    ids = np.array(sorted(tot))
    rel_tot = (ra[0], ra[1] + rb[1])
    O.adagrad_update(ref, {0: (ids, np.stack([tot[r] for r in ids]))}, rel_tot, 0.1)
    assert np.allclose(m2.emb[0], ref.emb[0], atol=1e-15)
    assert np.allclose(m2.rel, ref.rel, atol=1e-15)
    m1 = run(1)
    assert not np.allclose(m1.emb[0], m2.emb[0], atol=1e-9)


def test_short_last_chunk_and_chunk_offset():
    """A call starting at chunk c0 draws the same negatives as the full pass."""
    model_a = _tiny_model("diagonal", "dot", "ranking", P=1, n=9, R=2, seed=4)
    model_b = _tiny_model("diagonal", "dot", "ranking", P=1, n=9, R=2, seed=4)
    src, rel, dst = _tiny_edges(model_a, 0, 0, 10, 4)
    la, steps_a = O.train_bucket(model_a, 0, 0, src, rel, dst, 3, 2, 2, 0.1, 17, return_steps=True)
    assert len(steps_a) == 2                      # chunks 3,3,3,1 -> steps of 2 chunks
    lb1 = O.train_bucket(model_b, 0, 0, src[:6], rel[:6], dst[:6], 3, 2, 2, 0.1, 17)
    lb2 = O.train_bucket(model_b, 0, 0, src[6:], rel[6:], dst[6:], 3, 2, 2, 0.1, 17, first_chunk=2)
    assert abs(la - (lb1 + lb2)) < 1e-12
    assert np.array_equal(model_a.emb[0], model_b.emb[0])


# ------------------------------------------------------------ ranking (O11)
def test_rank_eval_brute_force():
    rng = np.random.default_rng(12)
    n, R, d = 7, 2, 4
    E = rng.standard_normal((n, d))
    model = O.Model.create(n, 1, R, d, "diagonal", "dot", "ranking", 0.1, [E],
                           rng.standard_normal((R, d)))
    src = np.array([0, 3, 5, 5])
    rel = np.array([1, 0, 1, 1])
    dst = np.array([2, 4, 6, 0])
    ks = np.concatenate([src, [0, 0, 1]])
    kr = np.concatenate([rel, [1, 0, 1]])
    kd = np.concatenate([dst, [5, 2, 6]])
    known = set(zip(ks.tolist(), kr.tolist(), kd.tolist()))
    ranks, mrr, hits = O.rank_eval(model, src, rel, dst, ks, kr, kd)
    for e in range(len(src)):
        s, r, t = int(src[e]), int(rel[e]), int(dst[e])
        pos = O.score_edges(model, 0, 0, [s], [r], [t])[0]
        rd = 1 + sum(1 for c in range(n) if c != t and (s, r, c) not in known
                     and O.score_edges(model, 0, 0, [s], [r], [c])[0] >= pos)
        rs = 1 + sum(1 for c in range(n) if c != s and (c, r, t) not in known
                     and O.score_edges(model, 0, 0, [c], [r], [t])[0] >= pos)
        assert ranks[e] == rd and ranks[len(src) + e] == rs
    assert abs(mrr - np.mean(1.0 / ranks)) < 1e-15
    assert abs(hits - np.mean(ranks <= 10)) < 1e-15


def test_rank_sampled_hand_worked():
    """identity + dot on 1-d embeddings x_v = v + 1: f(s, r, d) = (s + 1)(d + 1).
    Triple (0, 1): f = 2.  Candidates [3, 2, 1, 1, 0]: destination scores
    4, 3, 2, 2, 1, the two copies of the true destination 1 left out -> rank 3;
    source scores f(c, 1) = 2 (c + 1) = 8, 6, 4, 4, 2, the true source 0 left
    out, both copies of 1 counted -> rank 5."""
    E = np.arange(1.0, 5.0).reshape(4, 1)
    model = O.Model.create(4, 1, 1, 1, "identity", "dot", "ranking", 0.1, [E])
    ranks, mrr, hits = O.rank_sampled(model, [0], None, [1], [3, 2, 1, 1, 0])
    assert ranks.tolist() == [3, 5]
    assert abs(mrr - (1 / 3 + 1 / 5) / 2) < 1e-15 and hits == 1.0


def test_rank_sampled_brute_force():
    """Each rank recounted candidate by candidate from single-edge scores."""
    rng = np.random.default_rng(33)
    n, R, d = 8, 3, 6
    model = O.Model.create(n, 1, R, d, "complex_diagonal", "dot", "ranking", 0.1, [rng.standard_normal((n, d))],
                           rng.standard_normal((R, d)))
    src, rel, dst = np.array([1, 6, 2]), np.array([2, 0, 1]), np.array([5, 6, 0])
    cand = np.array([0, 5, 5, 7, 1, 3, 6, 2])
    ranks, _, _ = O.rank_sampled(model, src, rel, dst, cand)
    for e in range(len(src)):
        s, r, t = int(src[e]), int(rel[e]), int(dst[e])
        pos = O.score_edges(model, 0, 0, [s], [r], [t])[0]
        rd = 1 + sum(1 for c in cand.tolist() if c != t and O.score_edges(model, 0, 0, [s], [r], [c])[0] >= pos)
        rs = 1 + sum(1 for c in cand.tolist() if c != s and O.score_edges(model, 0, 0, [c], [r], [t])[0] >= pos)
        assert (ranks[e], ranks[len(src) + e]) == (rd, rs)


def test_rank_sampled_invariants():
    rng = np.random.default_rng(21)
    n, R, d = 9, 2, 5
    E = rng.standard_normal((n, d))
    for op, cmp in (("translation", "cos"), ("complex_diagonal", "dot"), ("diagonal", "dot")):
        model = O.Model.create(n, 1, R, d if op != "complex_diagonal" else 6, op, cmp, "ranking", 0.1,
                               [E if op != "complex_diagonal" else rng.standard_normal((n, 6))],
                               rng.standard_normal((R, d if op != "complex_diagonal" else 6)))
        src, rel, dst = np.array([0, 4, 8]), np.array([1, 0, 1]), np.array([3, 3, 2])
        # every entity once, nothing known: the filtered ranks without a filter
        full, _, _ = O.rank_sampled(model, src, rel, dst, np.arange(n))
        want, _, _ = O.rank_eval(model, src, rel, dst, [], [], [])
        assert np.array_equal(full, want)
        cand = rng.integers(0, n, 15)
        r1, _, _ = O.rank_sampled(model, src, rel, dst, cand)
        assert np.all(r1 >= 1) and np.all(r1 <= len(cand) + 1)
        # every candidate listed twice: every count doubles
        r2, _, _ = O.rank_sampled(model, src, rel, dst, np.concatenate([cand, cand]))
        assert np.array_equal(r2 - 1, 2 * (r1 - 1))


def test_rank_eval_monotone_construction():
    """identity + dot with x_v = (v + 1) e_1: f(s, r, d) = (s + 1)(d + 1), so the
    destination rank of d among unfiltered candidates is 1 + #{d' > d}."""
    n = 12
    E = np.zeros((n, 2))
    E[:, 0] = np.arange(1, n + 1)
    model = O.Model.create(n, 1, 1, 2, "identity", "dot", "ranking", 0.1, [E])
    src, dst = np.array([2, 7, 0]), np.array([5, 1, 11])
    ranks, _, _ = O.rank_eval(model, src, None, dst, src, None, dst)
    for e in range(3):
        assert ranks[e] == 1 + (n - 1 - dst[e])
        assert ranks[3 + e] == 1 + (n - 1 - src[e])
    # filtering a higher-scored candidate lowers the rank by one; ties count against
    ranks2, _, _ = O.rank_eval(model, src[:1], None, dst[:1],
                               np.array([2, 2]), None, np.array([5, 9]))
    assert ranks2[0] == 1 + (n - 1 - 5) - 1
    E2 = E.copy()
    E2[4] = E2[5]                      # candidate 4 now ties with the true destination 5
    model2 = O.Model.create(n, 1, 1, 2, "identity", "dot", "ranking", 0.1, [E2])
    ranks3, _, _ = O.rank_eval(model2, src[:1], None, dst[:1], src[:1], None, dst[:1])
    assert ranks3[0] == 1 + (n - 1 - 5) + 1


# ------------------------------------------- forward half of a step (inspection)
def _sigmoid(v):
    return 1.0 / (1.0 + math.exp(-v))


@pytest.mark.parametrize("op,cmp,loss", [("identity", "dot", "ranking"), ("translation", "cos", "ranking"),
                                         ("diagonal", "dot", "logistic"), ("complex_diagonal", "dot", "softmax"),
                                         ("linear", "dot", "logistic"), ("linear", "cos", "softmax"),
                                         ("translation", "dot", "softmax")])
def test_inspect_step_pair_loops(op, cmp, loss):
    """Scores, per-edge side losses and dL/dS of every chunk against explicit
    per-pair Python loops and the closed forms of each loss's derivative:
    ranking [margin - p + n > 0], logistic sigmoid(n) / K_e, softmax
    exp(n) / (exp(p) + sum of exp over the valid negatives)."""
    R = 1 if (cmp == "cos" and op != "identity") else 3
    model = _tiny_model(op, cmp, loss, n=11, P=1, R=R, d=4, seed=2)
    rng = np.random.default_rng(5)
    m, C, U, seed = 7, 3, 2, 77
    src, dst = rng.integers(0, 11, m), rng.integers(0, 11, m)
    rel = rng.integers(0, R, m)
    out = O.inspect_step(model, 0, 0, src, rel, dst, C, U, seed)
    E = model.emb[0]
    for k, (c, lo, hi) in enumerate(O.chunk_ranges(m, C)):
        rec = out[k]
        Cc = hi - lo
        u_dst = O.uniform_negatives(seed, 0, c, 0, U, 11)
        u_src = O.uniform_negatives(seed, 0, c, 1, U, 11)
        cd = list(dst[lo:hi]) + list(u_dst)
        cs = list(src[lo:hi]) + list(u_src)
        for e in range(Cc):
            th = [] if model.rel is None else list(model.rel[rel[lo + e]])
            ge = _py_operator(op, list(E[src[lo + e]]), th)
            p = _py_sim(cmp, ge, list(E[dst[lo + e]]))
            assert abs(rec["p"][e] - p) < 1e-12
            for side in (0, 1):
                scores = []
                for t in range(Cc + U):
                    if side == 0:
                        v = _py_sim(cmp, ge, list(E[cd[t]]))
                    else:
                        v = _py_sim(cmp, _py_operator(op, list(E[cs[t]]), th), list(E[dst[lo + e]]))
                    assert abs(rec[f"S{side}"][e, t] - v) < 1e-12
                    scores.append(v)
                negs = [scores[t] for t in range(Cc + U) if t != e]
                K = len(negs)
                if loss == "ranking":
                    want_l = sum(max(0.0, model.margin - p + v) for v in negs)
                    want_d = [0.0 if t == e else float(model.margin - p + scores[t] > 0) for t in range(Cc + U)]
                elif loss == "logistic":
                    sp = lambda v: math.log1p(math.exp(v))
                    want_l = sp(-p) + sum(sp(v) for v in negs) / K
                    want_d = [0.0 if t == e else _sigmoid(scores[t]) / K for t in range(Cc + U)]
                else:
                    z = math.exp(p) + sum(math.exp(v) for v in negs)
                    want_l = math.log(z) - p
                    want_d = [0.0 if t == e else math.exp(scores[t]) / z for t in range(Cc + U)]
                assert abs(rec[f"loss{side}"][e] - want_l) < 1e-12
                assert np.allclose(rec[f"dS{side}"][e], want_d, atol=1e-14, rtol=0)


def test_branch_override_natural_choice_is_identity():
    """Fixing every hinge branch to the side it falls on reproduces the plain step."""
    model = _tiny_model("diagonal", "dot", "ranking", n=11, P=1, R=2, d=4, seed=3, scale=0.6)
    src, rel, dst = _tiny_edges(model, 0, 0, 7, 3)
    rec = O.inspect_step(model, 0, 0, src, rel, dst, 3, 2, 9)
    branches = [(r["dS0"] > 0, r["dS1"] > 0) for r in rec]
    step = O.chunk_ranges(7, 3)
    negs = O.step_negatives(model, 0, 0, step, 9, 2)
    l0, g0, r0 = O.step_loss_and_grad(model, 0, 0, src, rel, dst, step, negs)
    l1, g1, r1 = O.step_loss_and_grad(model, 0, 0, src, rel, dst, step, negs, branches=branches)
    assert abs(l0 - l1) < 1e-14
    assert np.array_equal(g0[0][0], g1[0][0]) and np.allclose(g0[0][1], g1[0][1], atol=1e-14, rtol=0)
    assert np.allclose(r0[1], r1[1], atol=1e-14, rtol=0)


def test_branch_override_one_flipped_pair():
    """identity + dot, one edge (s, d) and one destination-side uniform
    negative d' whose hinge is inactive: forcing it active adds the pair's
    closed-form gradient (x_d' - x_d to s, -x_s to d, x_s to d') and its
    value lambda - <s,d> + <s,d'> to the loss."""
    n, d = 8, 3
    for seed in range(1000):
        u_dst = int(O.uniform_negatives(seed, 0, 0, 0, 1, n)[0])
        u_src = int(O.uniform_negatives(seed, 0, 0, 1, 1, n)[0])
        if len({0, 1, u_dst, u_src}) == 4:
            break
    E = np.zeros((n, d))
    E[0] = [1.0, 0.5, 0.0]
    E[1] = [0.2, 0.1, 0.0]
    E[u_dst] = [-0.3, 0.2, 0.4]   # 0.1 - 0.25 - 0.2 < 0: inactive
    E[u_src] = [-5.0, 0.0, 1.0]
    model = O.Model.create(n, 1, 1, d, "identity", "dot", "ranking", 0.1, [E])
    step = O.chunk_ranges(1, 1)
    negs = O.step_negatives(model, 0, 0, step, seed, 1)
    args = (model, 0, 0, np.array([0]), np.array([0]), np.array([1]), step, negs)
    l0, g0, _ = O.step_loss_and_grad(*args)
    flip = [(np.array([[0.0, 1.0]]), np.array([[0.0, 0.0]]))]
    l1, g1, _ = O.step_loss_and_grad(*args, branches=flip)
    assert l0 == 0.0 and abs(l1 - (0.1 - 0.25 - 0.2)) < 1e-15
    ids = [int(r) for r in g0[0][0]]
    diff = {r: g1[0][1][k] - g0[0][1][k] for k, r in enumerate(ids)}
    assert np.allclose(diff[0], E[u_dst] - E[1], atol=1e-15)
    assert np.allclose(diff[1], -E[0], atol=1e-15)
    assert np.allclose(diff[u_dst], E[0], atol=1e-15)
    assert np.allclose(diff[u_src], 0.0, atol=0)


def test_inspect_step_positive_gradient_closed_form():
    """dL/dp of each edge: ranking -(number of active hinges on both sides),
    logistic 2 (sigmoid(p) - 1), softmax sum over sides of (softmax_p - 1)."""
    for loss in O.LOSSES:
        model = _tiny_model("diagonal", "dot", loss, n=11, P=1, R=2, d=4, seed=4, scale=0.7)
        src, rel, dst = _tiny_edges(model, 0, 0, 5, 4)
        for rec in O.inspect_step(model, 0, 0, src, rel, dst, 5, 3, 21):
            p = rec["p"]
            for e in range(p.shape[0]):
                if loss == "ranking":
                    want = -float((rec["dS0"][e] > 0).sum() + (rec["dS1"][e] > 0).sum())
                elif loss == "logistic":
                    want = 2.0 * (_sigmoid(p[e]) - 1.0)
                else:
                    want = 0.0
                    for side in (0, 1):
                        S = rec[f"S{side}"][e]
                        vals = [p[e]] + [S[t] for t in range(S.shape[0]) if t != e]
                        z = sum(math.exp(v) for v in vals)
                        want += math.exp(p[e]) / z - 1.0
                assert abs(rec["dp"][e] - want) < 1e-12


# ----------------------------------------------- relation-grouped chunks (O3)
def test_relation_grouped_chunks_brute_force():
    """Every chunk holds one relation and at most C edges, chunks cover the
    edges in order, and only the last chunk of each relation's run is short;
    unsorted relations are refused."""
    rng = np.random.default_rng(3)
    for C in (1, 3, 7):
        rel = np.sort(rng.integers(0, 6, 50))
        ch = O.chunk_ranges_by_relation(rel, C)
        assert [c for c, _, _ in ch] == list(range(len(ch)))
        pos = 0
        for k, (c, lo, hi) in enumerate(ch):
            assert lo == pos and 0 < hi - lo <= C
            assert len(set(rel[lo:hi].tolist())) == 1
            run_continues = hi < len(rel) and rel[hi] == rel[lo]
            if hi - lo < C:
                assert not run_continues
            pos = hi
        assert pos == len(rel)
        # the number of chunks is the sum over runs of ceil(run / C)
        _, counts = np.unique(rel, return_counts=True)
        assert len(ch) == sum(-(-int(n) // C) for n in counts)
    with pytest.raises(ValueError):
        O.chunk_ranges_by_relation(np.array([0, 2, 1]), 4)
    # one relation: the same chunks as consecutive chunking
    assert O.chunk_ranges_by_relation(np.zeros(10, int), 4) == O.chunk_ranges(10, 4)


def test_relation_grouped_training_matches_explicit_chunks():
    """train_bucket with grouped chunking equals training the chunks one call
    per chunk with consecutive chunking and the right chunk numbers (S = 1),
    so the grouping only moves chunk boundaries."""
    model = _tiny_model("diagonal", "cos", "softmax", n=11, P=1, R=3, d=4, seed=6, scale=0.6)
    rng = np.random.default_rng(8)
    m = 13
    rel = np.sort(rng.integers(0, 3, m))
    src, dst = rng.integers(0, 11, m), rng.integers(0, 11, m)
    a = O.Model.create(11, 1, 3, 4, "diagonal", "cos", "softmax", 0.1, [model.emb[0].copy()], model.rel.copy())
    b = O.Model.create(11, 1, 3, 4, "diagonal", "cos", "softmax", 0.1, [model.emb[0].copy()], model.rel.copy())
    la = O.train_bucket(a, 0, 0, src, rel, dst, 3, 2, 1, 0.1, 5, chunking="by_relation")
    lb = 0.0
    for c, lo, hi in O.chunk_ranges_by_relation(rel, 3):
        lb += O.train_bucket(b, 0, 0, src[lo:hi], rel[lo:hi], dst[lo:hi], 3, 2, 1, 0.1, 5, first_chunk=c)
    assert abs(la - lb) < 1e-12
    assert np.allclose(a.emb[0], b.emb[0], atol=1e-15, rtol=0) and np.allclose(a.rel, b.rel, atol=1e-15, rtol=0)


# ------------------------------------------------ reciprocal predicates (Sec. 5.4)
def _adjoint_params(op, th):
    """Parameters of the operator that is the adjoint of g(., th) under the dot
    product: theta itself for diagonal (and identity), conj(theta) for complex."""
    th = np.asarray(th, dtype=np.float64)
    if op == "complex_diagonal":
        h = th.shape[-1] // 2
        return np.concatenate([th[..., :h], -th[..., h:]], -1)
    return th.copy()


def _reciprocal_twin(base, rev_rows):
    return O.Model.create(base.n, base.P, base.R, base.d, base.op, base.cmp, base.loss, base.margin,
                          [base.emb[p] for p in range(base.P)], np.concatenate([base.rel, rev_rows]),
                          reciprocal=True)


@pytest.mark.parametrize("op", ["diagonal", "complex_diagonal"])
@pytest.mark.parametrize("loss", O.LOSSES)
def test_reciprocal_with_adjoint_rows_reproduces_the_shared_operator(op, loss):
    """With dot, <g(x_t, th), x_d> = <x_t, g*(x_d, th)>.  A reciprocal model whose
    source-side rows r + R hold the adjoint's parameters scores every source
    corruption as the ordinary model does: same scores, losses and entity
    gradients, and the ordinary model's relation gradient is row r's plus row
    r + R's mapped back through the adjoint (a self-inverse linear map).
    Complex parameters make rows r and r + R differ, so reading row r on the
    source side fails here."""
    base = _tiny_model(op, "dot", loss, R=3, seed=3)
    recip = _reciprocal_twin(base, _adjoint_params(op, base.rel))
    i, j = 0, 1
    src, rel, dst = _tiny_edges(base, i, j, 7, 3)
    step = O.chunk_ranges(7, 3)
    negs = O.step_negatives(base, i, j, step, 9, 2)
    la, ga, ra = O.step_loss_and_grad(base, i, j, src, rel, dst, step, negs)
    lb, gb, rb = O.step_loss_and_grad(recip, i, j, src, rel, dst, step, negs)
    assert abs(la - lb) < 1e-12 * max(1.0, abs(la))
    for p in ga:
        assert np.array_equal(ga[p][0], gb[p][0])
        assert np.allclose(ga[p][1], gb[p][1], atol=1e-12, rtol=0)
    ids_b = list(rb[0])
    for a, r in enumerate(ra[0]):
        fwd = rb[1][ids_b.index(r)]
        rev = rb[1][ids_b.index(r + base.R)]
        assert np.allclose(ra[1][a], fwd + _adjoint_params(op, rev), atol=1e-12, rtol=0)
    ins_a = O.inspect_step(base, i, j, src, rel, dst, 3, 2, 9)
    ins_b = O.inspect_step(recip, i, j, src, rel, dst, 3, 2, 9)
    for ca, cb in zip(ins_a, ins_b):
        for key in ("S0", "S1", "loss0", "loss1", "dS0", "dS1"):
            assert np.allclose(ca[key], cb[key], atol=1e-12, rtol=0), key
        assert np.allclose(cb["p1"], ca["p"], atol=1e-12, rtol=0)
        assert np.allclose(cb["dp"] + cb["dp1"], ca["dp"], atol=1e-12, rtol=0)


@pytest.mark.parametrize("op,cmp", [(o, c) for o in O.OPERATORS for c in O.COMPARATORS])
def test_reciprocal_sides_swap_roles(op, cmp):
    """The source side of edge (s, r, d) is the destination side of (d, r + R, s)
    with the row roles exchanged; and each entry is the explicit-loop
    operator and comparator (the independent statement pinned above)."""
    rng = np.random.default_rng(21)
    d, C, U = 4, 3, 2
    w = max(O.relation_param_width(op, d), 1)
    src_rows = rng.standard_normal((C + U, d))
    dst_rows = rng.standard_normal((C + U, d))
    thf = rng.standard_normal((C, w))
    thr = rng.standard_normal((C, w))
    xs, xd = torch.tensor(src_rows[:C]), torch.tensor(dst_rows[:C])
    cs, cd = torch.tensor(src_rows), torch.tensor(dst_rows)
    tf = None if op == "identity" else torch.tensor(thf)
    tr = None if op == "identity" else torch.tensor(thr)
    p0, p1, S0, S1 = O.chunk_scores_reciprocal(op, cmp, xs, xd, tf, tr, cd, cs)
    q0, q1, T0, T1 = O.chunk_scores_reciprocal(op, cmp, xd, xs, tr, tf, cs, cd)
    assert torch.equal(p0, q1) and torch.equal(p1, q0)
    assert torch.equal(S0, T1) and torch.equal(S1, T0)
    for e in range(C):
        gq = _py_operator(op, list(src_rows[e]), list(thf[e]))
        gk = _py_operator(op, list(dst_rows[e]), list(thr[e]))
        assert abs(p0[e].item() - _py_sim(cmp, gq, list(dst_rows[e]))) < 1e-12
        assert abs(p1[e].item() - _py_sim(cmp, gk, list(src_rows[e]))) < 1e-12
        for t in range(C + U):
            assert abs(S0[e, t].item() - _py_sim(cmp, gq, list(dst_rows[t]))) < 1e-12
            assert abs(S1[e, t].item() - _py_sim(cmp, gk, list(src_rows[t]))) < 1e-12


def test_reciprocal_translation_logistic_gradient_closed_form():
    """translation + dot + logistic, reciprocal: with k_e = x_d + theta_{r+R},
    p1 = <k_e, x_s> and S1[e, t] = <k_e, c_t>, the source side contributes
    dL/dtheta_{r+R} = sum over the edges of r of (sigmoid(p1) - 1) x_s +
    (1 / K_e) sum over valid t of sigmoid(S1[e, t]) c_t, and nothing to theta_r;
    the destination side likewise gives theta_r's gradient with x_s + theta_r."""
    base = _tiny_model("translation", "dot", "logistic", R=2, seed=8)
    rng = np.random.default_rng(8)
    recip = _reciprocal_twin(base, rng.standard_normal(base.rel.shape) * 0.5)
    i, j = 1, 0
    src, rel, dst = _tiny_edges(base, i, j, 5, 8)
    step = O.chunk_ranges(5, 5)
    negs = O.step_negatives(base, i, j, step, 4, 3)
    _, _, (ids, g) = O.step_loss_and_grad(recip, i, j, src, rel, dst, step, negs)
    R = base.R
    expect = {r: np.zeros(base.d) for r in range(2 * R)}
    u_dst, u_src = negs[0]
    Xs, Xd = recip.emb[i][src], recip.emb[j][dst]
    cand_src = np.concatenate([Xs, recip.emb[i][u_src]])
    cand_dst = np.concatenate([Xd, recip.emb[j][u_dst]])
    sig = lambda v: 1.0 / (1.0 + math.exp(-v))
    for e in range(len(src)):
        r = int(rel[e])
        for row, anchor, other, cands in ((r, Xs[e], Xd[e], cand_dst), (r + R, Xd[e], Xs[e], cand_src)):
            k = anchor + recip.rel[row]
            K = len(cands) - 1
            acc = (sig(float(k @ other)) - 1.0) * other
            for t in range(len(cands)):
                if t != e:
                    acc = acc + sig(float(k @ cands[t])) * cands[t] / K
            expect[row] += acc
    for a, row in enumerate(ids):
        assert np.allclose(g[a], expect[int(row)], atol=1e-12, rtol=0), row


RECIP_COMBOS = [("translation", "cos", "ranking"), ("complex_diagonal", "dot", "softmax"),
                ("linear", "cos", "logistic"), ("diagonal", "cos", "softmax"), ("linear", "dot", "ranking"),
                ("identity", "dot", "logistic")]


@pytest.mark.parametrize("op,cmp,loss", RECIP_COMBOS)
def test_reciprocal_step_gradient_matches_finite_differences(op, cmp, loss):
    """The reciprocal step gradient (several relations, relations mixed inside
    the chunks, cos with an operator included) against central differences of
    the step loss."""
    i, j = 0, 1
    for seed in range(20):
        base = _tiny_model(op, cmp, loss, R=2, seed=seed)
        rev = None if base.rel is None else base.rel[::-1].copy() * 0.9
        model = base if base.rel is None else _reciprocal_twin(base, rev)
        model.reciprocal = True
        src, rel, dst = _tiny_edges(model, i, j, 7, seed)
        step = O.chunk_ranges(7, 3)
        negs = O.step_negatives(model, i, j, step, seed + 5, 2)
        if loss != "ranking":
            break
        ins = O.inspect_step(model, i, j, src, rel, dst, 3, 2, seed + 5)
        z = [np.abs(model.margin - c[pk][:, None] + c[sk])[O.valid_mask(len(c[pk]), 2).numpy() > 0]
             for c in ins for pk, sk in (("p", "S0"), ("p1", "S1"))]
        if min(float(v.min()) for v in z) > 1e-3:
            break
    _, grads, rel_grad = O.step_loss_and_grad(model, i, j, src, rel, dst, step, negs)
    h = 1e-6

    def f():
        return O.step_loss_and_grad(model, i, j, src, rel, dst, step, negs, with_grad=False)[0]

    def check(arr, idx, gval):
        keep = arr[idx]
        arr[idx] = keep + h
        up = f()
        arr[idx] = keep - h
        dn = f()
        arr[idx] = keep
        fd = (up - dn) / (2 * h)
        assert abs(fd - gval) <= 1e-6 * max(1.0, abs(gval)), (idx, fd, gval)

    for p, (ids, g) in grads.items():
        for a, row in enumerate(ids):
            for k in range(model.d):
                check(model.emb[p], (row, k), g[a, k])
    if rel_grad is not None:
        ids, g = rel_grad
        assert set(ids.tolist()) - set(range(model.R)), "no source-side row was touched"
        for a, r in enumerate(ids):
            for k in range(0, model.rel.shape[1], max(1, model.rel.shape[1] // 8)):
                check(model.rel, (r, k), g[a, k])


@pytest.mark.parametrize("op", ["diagonal", "complex_diagonal"])
def test_reciprocal_ranks_with_adjoint_rows_equal_the_shared_operator(op):
    rng = np.random.default_rng(31)
    n, R, d = 9, 2, 4
    E = rng.standard_normal((n, d))
    th = rng.standard_normal((R, d))
    base = O.Model.create(n, 1, R, d, op, "dot", "ranking", 0.1, [E], th)
    recip = _reciprocal_twin(base, _adjoint_params(op, th))
    src = np.array([0, 3, 5, 5, 8])
    rel = np.array([1, 0, 1, 1, 0])
    dst = np.array([2, 4, 6, 0, 1])
    ka = O.rank_eval(base, src, rel, dst, src, rel, dst)[0]
    kb = O.rank_eval(recip, src, rel, dst, src, rel, dst)[0]
    assert np.array_equal(ka, kb)
    cand = rng.integers(0, n, 12)
    assert np.array_equal(O.rank_sampled(base, src, rel, dst, cand)[0], O.rank_sampled(recip, src, rel, dst, cand)[0])


def test_reciprocal_rank_eval_brute_force():
    """Source side of a reciprocal model: 1 + #{c != s, (c, r, d) not known,
    sim(g(x_d, theta_{r+R}), x_c) >= sim(g(x_d, theta_{r+R}), x_s)}; translation
    with cos, explicit loops."""
    rng = np.random.default_rng(33)
    n, R, d = 8, 2, 3
    E = rng.standard_normal((n, d))
    rows = rng.standard_normal((2 * R, d))
    model = O.Model.create(n, 1, R, d, "translation", "cos", "ranking", 0.1, [E], rows, reciprocal=True)
    src = np.array([0, 3, 5, 7])
    rel = np.array([1, 0, 1, 0])
    dst = np.array([2, 4, 6, 1])
    ks = np.concatenate([src, [0, 2, 1]])
    kr = np.concatenate([rel, [1, 0, 1]])
    kd = np.concatenate([dst, [5, 4, 6]])
    known = set(zip(ks.tolist(), kr.tolist(), kd.tolist()))
    ranks = O.rank_eval(model, src, rel, dst, ks, kr, kd)[0]
    cand = np.array([1, 1, 4, 0, 6, 3])
    sranks = O.rank_sampled(model, src, rel, dst, cand)[0]
    for e in range(len(src)):
        s, r, t = int(src[e]), int(rel[e]), int(dst[e])
        q = _py_operator("translation", list(E[s]), list(rows[r]))
        k = _py_operator("translation", list(E[t]), list(rows[r + R]))
        p0, p1 = _py_sim("cos", q, list(E[t])), _py_sim("cos", k, list(E[s]))
        rd = 1 + sum(1 for c in range(n) if c != t and (s, r, c) not in known and _py_sim("cos", q, list(E[c])) >= p0)
        rs = 1 + sum(1 for c in range(n) if c != s and (c, r, t) not in known and _py_sim("cos", k, list(E[c])) >= p1)
        assert ranks[e] == rd and ranks[len(src) + e] == rs
        sd = 1 + sum(1 for c in cand if c != t and _py_sim("cos", q, list(E[c])) >= p0)
        ss = 1 + sum(1 for c in cand if c != s and _py_sim("cos", k, list(E[c])) >= p1)
        assert sranks[e] == sd and sranks[len(src) + e] == ss


# --------------------------------- entity types and relation weights (NEXT-4)
def _typed(counts, partitioned, rel_src, rel_dst, P, d, op, cmp, loss, seed, R=None, weights=None, scale=0.5):
    types = O.EntityTypes(list(counts), list(partitioned), np.asarray(rel_src), np.asarray(rel_dst))
    R = len(rel_src) if R is None else R
    rng = np.random.default_rng(seed)
    tables = {(t, p): rng.standard_normal((types.rows(t, P, p), d)) * scale
              for t in range(types.count) for p in range(types.parts(t, P))}
    w = O.relation_param_width(op, d)
    relp = None if w == 0 else rng.standard_normal((R, w)) * 0.5 + (np.eye(d).reshape(-1) if op == "linear" else 0)
    return O.Model.create_typed(types, P, R, d, op, cmp, loss, 0.1, tables, relp, weights=weights)


def test_typed_bucketing_brute_force():
    """Three types, type 2 kept whole: bucket = (partition of s in its type,
    partition of d in its type), local ids, stable order, by explicit loops."""
    counts, part = [10, 7, 4], [True, True, False]
    rel_src, rel_dst = np.array([0, 1, 2, 0]), np.array([1, 2, 0, 0])
    types = O.EntityTypes(counts, part, rel_src, rel_dst)
    P = 3
    rng = np.random.default_rng(3)
    m = 60
    rel = rng.integers(0, 4, m)
    src = np.array([rng.integers(0, counts[rel_src[r]]) for r in rel])
    dst = np.array([rng.integers(0, counts[rel_dst[r]]) for r in rel])
    off, sl, rl, dl = O.bucket_edges_typed(src, rel, dst, types, P)
    want = {}
    for e in range(m):
        r = int(rel[e])
        loc = []
        for t, v in ((rel_src[r], src[e]), (rel_dst[r], dst[e])):
            size = -(-counts[t] // P) if part[t] else counts[t]
            loc.append((int(v) // size, int(v) % size))
        want.setdefault(loc[0][0] * P + loc[1][0], []).append((loc[0][1], r, loc[1][1]))
    for b in range(P * P):
        got = list(zip(sl[off[b]:off[b + 1]].tolist(), rl[off[b]:off[b + 1]].tolist(), dl[off[b]:off[b + 1]].tolist()))
        assert got == want.get(b, []), b


def test_typed_bucketing_unpartitioned_destinations_give_p_buckets():
    """If every destination type is kept whole, edges fall into the P buckets
    (i, 0) only (Sec. 4.1)."""
    types = O.EntityTypes([1000, 30], [True, False], np.array([0, 0]), np.array([1, 1]))
    P = 4
    rng = np.random.default_rng(5)
    rel = rng.integers(0, 2, 500)
    src, dst = rng.integers(0, 1000, 500), rng.integers(0, 30, 500)
    off = O.bucket_edges_typed(src, rel, dst, types, P)[0]
    counts = np.diff(off).reshape(P, P)
    assert counts[:, 1:].sum() == 0 and np.all(counts[:, 0] > 0)


def test_one_type_typed_model_is_the_untyped_model():
    P, d = 2, 4
    typed = _typed([9], [True], [0, 0], [0, 0], P, d, "diagonal", "dot", "logistic", 11)
    untyped = O.Model.create(9, P, 2, d, "diagonal", "dot", "logistic", 0.1,
                             [typed.emb[(0, p)] for p in range(P)], typed.rel)
    src, rel, dst = _tiny_edges(untyped, 0, 1, 11, 11)
    order = np.argsort(rel, kind="stable")
    src, rel, dst = src[order], rel[order], dst[order]
    la = O.train_bucket(typed, 0, 1, src, rel, dst, 3, 2, 2, 0.1, 8, chunking="by_relation")
    lb = O.train_bucket(untyped, 0, 1, src, rel, dst, 3, 2, 2, 0.1, 8, chunking="by_relation")
    assert la == lb
    for p in range(P):
        assert np.array_equal(typed.emb[(0, p)], untyped.emb[p])
    assert np.array_equal(typed.rel, untyped.rel)


def test_runs_of_disjoint_type_pairs_train_independently():
    """Relations 0: type 0 -> 1 and 1: type 2 -> 3 touch disjoint tables.  A pass
    over both equals a pass over relation 0's edges followed by one over
    relation 1's with the chunk numbering continued: runs never share a step,
    and each run draws its negatives from its own tables."""
    mk = lambda: _typed([6, 9, 5, 8], [False] * 4, [0, 2], [1, 3], 1, 4, "translation", "cos", "softmax", 17)
    rng = np.random.default_rng(17)
    m0, m1 = 7, 5
    src = np.concatenate([rng.integers(0, 6, m0), rng.integers(0, 5, m1)])
    dst = np.concatenate([rng.integers(0, 9, m0), rng.integers(0, 8, m1)])
    rel = np.array([0] * m0 + [1] * m1)
    a, b = mk(), mk()
    la = O.train_bucket(a, 0, 0, src, rel, dst, 3, 2, 4, 0.1, 21, chunking="by_relation")
    n0 = len(O.chunk_ranges(m0, 3))
    lb = (O.train_bucket(b, 0, 0, src[:m0], rel[:m0], dst[:m0], 3, 2, 4, 0.1, 21, chunking="by_relation")
          + O.train_bucket(b, 0, 0, src[m0:], rel[m0:], dst[m0:], 3, 2, 4, 0.1, 21, first_chunk=n0,
                           chunking="by_relation"))
    assert abs(la - lb) < 1e-12
    for k in a.emb:
        assert np.array_equal(a.emb[k], b.emb[k]), k
    assert np.array_equal(a.rel, b.rel)


def test_negatives_come_from_the_relation_types():
    """Relation 0 goes from a type of 7 entities to one of 3,000: the destination
    side's draws cover the large type and the source side's stay below 7, and
    only rows of those two tables move."""
    model = _typed([7, 3000, 50], [False] * 3, [0], [1], 1, 4, "identity", "dot", "ranking", 23)
    rng = np.random.default_rng(23)
    src, dst, rel = rng.integers(0, 7, 40), rng.integers(0, 3000, 40), np.zeros(40, int)
    chunks = O.chunk_ranges(40, 10)
    ((run, tables),) = O.type_runs(model, 0, 0, chunks, rel)
    assert tables == ((0, 0), (1, 0))
    negs = O.step_negatives(model, 0, 0, run, 29, 100, 0, tables)
    dst_draws = np.concatenate([u for u, _ in negs])
    src_draws = np.concatenate([v for _, v in negs])
    assert src_draws.max() < 7 and dst_draws.max() > 2000
    before = {k: v.copy() for k, v in model.emb.items()}
    O.train_bucket(model, 0, 0, src, rel, dst, 10, 100, 2, 0.1, 29, chunking="by_relation")
    assert np.array_equal(before[(2, 0)], model.emb[(2, 0)])
    assert not np.array_equal(before[(0, 0)], model.emb[(0, 0)])


def test_uniform_relation_weight_scales_loss_and_gradient():
    model = _tiny_model("complex_diagonal", "dot", "softmax", R=2, seed=4)
    src, rel, dst = _tiny_edges(model, 0, 1, 7, 4)
    step = O.chunk_ranges(7, 3)
    negs = O.step_negatives(model, 0, 1, step, 6, 2)
    l1, g1, r1 = O.step_loss_and_grad(model, 0, 1, src, rel, dst, step, negs)
    model.weights = np.array([2.5, 2.5])
    l2, g2, r2 = O.step_loss_and_grad(model, 0, 1, src, rel, dst, step, negs)
    assert abs(l2 - 2.5 * l1) < 1e-12 * abs(l2)
    for p in g1:
        assert np.allclose(g2[p][1], 2.5 * g1[p][1], atol=1e-13, rtol=1e-13)
    assert np.allclose(r2[1], 2.5 * r1[1], atol=1e-13, rtol=1e-13)


def test_relation_weights_weigh_each_chunk():
    """Relation-grouped chunks, weights (0.5, 0, 3): the step's gradient is the
    sum over chunks of the chunk's relation weight times its unit-weight
    gradient, and a relation of weight 0 has no effect."""
    model = _tiny_model("translation", "cos", "logistic", R=3, seed=9)
    src, rel, dst = _tiny_edges(model, 1, 0, 12, 9)
    order = np.argsort(rel, kind="stable")
    src, rel, dst = src[order], rel[order], dst[order]
    step = O.chunk_ranges_by_relation(rel, 3)
    negs = O.step_negatives(model, 1, 0, step, 2, 2)
    w = np.array([0.5, 0.0, 3.0])
    total_l, total = 0.0, {}
    for ch, ng in zip(step, negs):
        l, g, rg = O.step_loss_and_grad(model, 1, 0, src, rel, dst, [ch], [ng])
        wc = w[rel[ch[1]]]
        total_l += wc * l
        for p, (ids, gr) in g.items():
            for a, row in enumerate(ids):
                total[(p, row)] = total.get((p, row), 0) + wc * gr[a]
        for a, r in enumerate(rg[0]):
            total[("rel", r)] = total.get(("rel", r), 0) + wc * rg[1][a]
    model.weights = w
    l, g, rg = O.step_loss_and_grad(model, 1, 0, src, rel, dst, step, negs)
    assert abs(l - total_l) < 1e-12 * max(1.0, abs(l))
    for p, (ids, gr) in g.items():
        for a, row in enumerate(ids):
            assert np.allclose(gr[a], total[(p, row)], atol=1e-12, rtol=0)
    for a, r in enumerate(rg[0]):
        assert np.allclose(rg[1][a], total[("rel", r)], atol=1e-12, rtol=0)
        if r == 1:
            assert not rg[1][a].any()


def test_typed_weighted_step_matches_finite_differences():
    """Unbalanced types (5 vs 40 entities), two type pairs, weights; the first
    run holds the chunks of two relations of one type pair: central
    differences of its step."""
    model = _typed([5, 40], [False, False], [0, 0, 1], [1, 1, 1], 1, 3, "diagonal", "dot", "logistic", 31,
                   weights=[0.7, 1.9, 1.3])
    rng = np.random.default_rng(31)
    rel = np.array([0, 0, 0, 0, 1, 1, 2, 2, 2])
    src = np.array([rng.integers(0, 5 if r < 2 else 40) for r in rel])
    dst = rng.integers(0, 40, len(rel))
    chunks = O.chunk_ranges_by_relation(rel, 3)
    runs = O.type_runs(model, 0, 0, chunks, rel)
    assert [t for _, t in runs] == [((0, 0), (1, 0)), ((1, 0), (1, 0))]
    run, tables = runs[0]
    negs = O.step_negatives(model, 0, 0, run, 3, 2, 0, tables)
    _, grads, rel_grad = O.step_loss_and_grad(model, tables[0], tables[1], src, rel, dst, run, negs)
    f = lambda: O.step_loss_and_grad(model, tables[0], tables[1], src, rel, dst, run, negs, with_grad=False)[0]
    h = 1e-6
    for key, (ids, g) in grads.items():
        for a, row in enumerate(ids):
            for k in range(model.d):
                keep = model.emb[key][row, k]
                model.emb[key][row, k] = keep + h
                up = f()
                model.emb[key][row, k] = keep - h
                dn = f()
                model.emb[key][row, k] = keep
                assert abs((up - dn) / (2 * h) - g[a, k]) <= 1e-6 * max(1.0, abs(g[a, k]))
    ids, g = rel_grad
    for a, r in enumerate(ids):
        for k in range(model.d):
            keep = model.rel[r, k]
            model.rel[r, k] = keep + h
            up = f()
            model.rel[r, k] = keep - h
            dn = f()
            model.rel[r, k] = keep
            assert abs((up - dn) / (2 * h) - g[a, k]) <= 1e-6 * max(1.0, abs(g[a, k]))


def test_whole_type_lives_in_partition_zero():
    """P = 2, users split in two, items kept whole; relations user -> item,
    item -> user, user -> user.  Bucketing puts item endpoints in partition 0,
    every bucket with edges trains against its relation's tables (an epoch in
    inside-out order), and asking for item-source edges in bucket (1, 0) is
    an error."""
    types = O.EntityTypes([20, 6], [True, False], np.array([0, 1, 0]), np.array([1, 0, 0]))
    P, d = 2, 3
    rng = np.random.default_rng(37)
    tables = {(t, p): rng.standard_normal((types.rows(t, P, p), d)) * 0.5
              for t in range(2) for p in range(types.parts(t, P))}
    model = O.Model.create_typed(types, P, 3, d, "translation", "dot", "ranking", 0.1, tables,
                                 rng.standard_normal((3, d)) * 0.3)
    m = 90
    rel = rng.integers(0, 3, m)
    src = np.array([rng.integers(0, types.counts[types.rel_src[r]]) for r in rel])
    dst = np.array([rng.integers(0, types.counts[types.rel_dst[r]]) for r in rel])
    off, sl, rl, dl = O.bucket_edges_typed(src, rel, dst, types, P)
    per = np.diff(off).reshape(P, P)
    assert per[1, 1] == 0 or np.all(rl[off[3]:off[4]] == 2)
    # item endpoints: the item-source relation only in buckets (0, *), the item-destination one only in (*, 0)
    for b in range(P * P):
        r_b = rl[off[b]:off[b + 1]]
        if b // P == 1:
            assert not np.any(r_b == 1)
        if b % P == 1:
            assert not np.any(r_b == 0)
    # sort each bucket by relation for the relation-grouped chunks
    for b in range(P * P):
        lo, hi = off[b], off[b + 1]
        o = np.argsort(rl[lo:hi], kind="stable")
        sl[lo:hi], rl[lo:hi], dl[lo:hi] = sl[lo:hi][o], rl[lo:hi][o], dl[lo:hi][o]
    before = {k: v.copy() for k, v in model.emb.items()}
    O.train_epoch(model, off, sl, rl, dl, 4, 3, 2, 0.1, 41, chunking="by_relation")
    assert all(not np.array_equal(before[k], model.emb[k]) for k in model.emb)
    with pytest.raises(ValueError):
        O.train_bucket(model, 1, 0, np.array([0, 1]), np.array([1, 1]), np.array([0, 1]), 4, 3, 2, 0.1, 41,
                       chunking="by_relation")
