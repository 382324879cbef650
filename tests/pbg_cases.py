"""Shared set-up for the GPU parity tests: one seeded problem fed identically
to the HIP library (through the C ABI binding) and to the CPU oracle."""

from __future__ import annotations

from dataclasses import dataclass

import numpy as np
import torch

from oracle import pbg_oracle as O
from paper_1903_12287_amd import synth


@dataclass
class Problem:
    n: int
    P: int
    R: int
    d: int
    op: str
    cmp: str
    loss: str
    margin: float
    parts: list            # float32 numpy per partition
    rel: np.ndarray | None  # float32 [R, width]
    i: int
    j: int
    src: np.ndarray         # local ids
    rel_ids: np.ndarray | None
    dst: np.ndarray
    C: int
    U: int
    S: int
    lr: float
    seed: int
    chunking: str = "consecutive"
    reciprocal: bool = False   # rel holds 2R rows: theta_r, then the source side's theta_{r+R}


def make_problem(op, cmp, loss, n=60, P=1, R=1, d=16, m=300, C=20, U=12, S=4, i=0, j=0,
                 seed=1, sigma=0.3, rel_scale=0.3, lr=0.1, margin=0.1, zipf=1.1, chunking="consecutive",
                 reciprocal=False):
    """A small seeded problem with Zipf endpoints (duplicates in chunks) and
    perturbed relation parameters (2R rows with reciprocal predicates); with
    chunking='by_relation' the edges are sorted by relation (stably)."""
    rng = synth.rng_for(seed)
    rows = [O.partition_rows(n, P, p) for p in range(P)]
    parts = synth.partition_embeddings(rows, d, rng, sigma)
    src = synth.BoundedZipf(rows[i], zipf, rng).sample(rng, m)
    dst = synth.BoundedZipf(rows[j], zipf, rng).sample(rng, m)
    rel_ids = None if R == 1 else rng.integers(0, R, m).astype(np.int32)
    relp = synth.perturbed_relation_params(op, 2 * R if reciprocal else R, d, rng, rel_scale)
    if chunking == "by_relation" and rel_ids is not None:
        order = np.argsort(rel_ids, kind="stable")
        src, rel_ids, dst = src[order], rel_ids[order], dst[order]
    return Problem(n, P, R, d, op, cmp, loss, margin, parts, relp, i, j, src, rel_ids, dst,
                   C, U, S, lr, seed + 1000, chunking, reciprocal)


def oracle_model(pb: Problem) -> O.Model:
    return O.Model.create(pb.n, pb.P, pb.R, pb.d, pb.op, pb.cmp, pb.loss, pb.margin,
                          [p.astype(np.float64) for p in pb.parts],
                          None if pb.rel is None else pb.rel.astype(np.float64), reciprocal=pb.reciprocal)


class GpuModel:
    """Device tensors of a problem bound to a library context."""

    def __init__(self, pb: Problem, flags: int = 0):
        from paper_1903_12287_amd import pbg
        self.pbg = pbg
        self.pb = pb
        dev = torch.device("cuda")
        if pb.reciprocal:
            flags |= pbg.F_RECIPROCAL
        self.ctx = pbg.pbg_bucket_init(pb.n, pb.P, pb.R, pb.d, pb.op, pb.cmp, pb.loss, pb.margin, flags)
        self.emb = [torch.from_numpy(p.copy()).to(dev) for p in pb.parts]
        self.G = [torch.zeros(p.shape[0], dtype=torch.float32, device=dev) for p in pb.parts]
        for p in range(pb.P):
            pbg.pbg_bind_partition(self.ctx, p, self.emb[p], self.G[p])
        self.relp = self.relG = None
        if pb.rel is not None:
            self.relp = torch.from_numpy(pb.rel.copy()).to(dev)
            self.relG = torch.zeros_like(self.relp)
            pbg.pbg_bind_relations(self.ctx, self.relp, self.relG)
        pbg.pbg_set_streams(self.ctx, torch.cuda.current_stream(), None)
        self.src = torch.from_numpy(pb.src.astype(np.int32)).to(dev)
        self.dst = torch.from_numpy(pb.dst.astype(np.int32)).to(dev)
        self.rel_ids = None if pb.rel_ids is None else torch.from_numpy(pb.rel_ids).to(dev)

    def train(self, lo=0, hi=None, first_chunk=0):
        pb = self.pb
        hi = pb.src.shape[0] if hi is None else hi
        r = None if self.rel_ids is None else self.rel_ids[lo:hi]
        return self.pbg.pbg_train_bucket(self.ctx, pb.i, pb.j, self.src[lo:hi], r, self.dst[lo:hi],
                                         pb.C, pb.U, pb.S, pb.lr, pb.seed, first_chunk, pb.chunking)

    def state(self):
        torch.cuda.synchronize()
        out = {"emb": [e.cpu().numpy().astype(np.float64) for e in self.emb],
               "G": [g.cpu().numpy().astype(np.float64) for g in self.G]}
        if self.relp is not None:
            out["rel"] = self.relp.cpu().numpy().astype(np.float64)
            out["relG"] = self.relG.cpu().numpy().astype(np.float64)
        return out

    def close(self):
        self.pbg.pbg_free(self.ctx)


# ---------------------------------------------------------------------------
# Error scales of the float32 scores: every bound in the parity tests is a
# multiple of A = sum_k |a_k| |b_k| over the products the kernels form for a
# score, with each factor replaced by the absolute values it is built from
# (so that cancellation inside the operator cannot make the bound too tight).
# ---------------------------------------------------------------------------
def _abs_forward(op, x, th):
    """|g(x)| bound, elementwise: x, th already absolute values."""
    if op == "identity":
        return x
    if op == "translation":
        return x + th
    if op == "diagonal":
        return x * th
    if op == "linear":
        d = x.shape[-1]
        A = th.reshape(*th.shape[:-1], d, d)
        return np.einsum("...kl,...l->...k", A, x)
    h = x.shape[-1] // 2
    xr, xi, tr, ti = x[..., :h], x[..., h:], th[..., :h], th[..., h:]
    return np.concatenate([xr * tr + xi * ti, xr * ti + xi * tr], -1)


def _abs_adjoint(op, y, th):
    """|g*(y)| bound: the kernels score the source side as <x_t, g*(y)>."""
    if op in ("identity", "translation"):
        return y
    if op == "diagonal":
        return y * th
    if op == "linear":
        d = y.shape[-1]
        A = th.reshape(*th.shape[:-1], d, d)
        return np.einsum("...kl,...k->...l", A, y)
    h = y.shape[-1] // 2
    yr, yi, tr, ti = y[..., :h], y[..., h:], th[..., :h], th[..., h:]
    return np.concatenate([tr * yr + ti * yi, tr * yi + ti * yr], -1)


def _norm(v):
    return np.maximum(np.linalg.norm(v, axis=-1), O.EPS_NORM)


def score_scales(model, i, j, src, rel, dst, C, U, seed, first_chunk=0, chunking="consecutive", tables=None):
    """Per chunk of a step: (Ap (C_c,), A0 (C_c, N_c), A1 (C_c, N_c), Ap1 (C_c,)),
    Ap1 the source side's positive score scale (reciprocal predicates; else Ap).
    tables: the keys of the source and destination tables (entity types;
    by default partitions i and j)."""
    src = np.asarray(src, np.int64)
    dst = np.asarray(dst, np.int64)
    m = src.shape[0]
    step = O.make_chunks(m, C, rel, chunking)
    rel = np.zeros(m, np.int64) if rel is None else np.asarray(rel, np.int64)
    negs = O.step_negatives(model, i, j, step, seed, U, first_chunk, tables)
    ti, tj = (i, j) if tables is None else tables
    Ei, Ej = model.emb[ti], model.emb[tj]
    out = []
    for (c, lo, hi), (u_dst, u_src) in zip(step, negs):
        xs, xd = Ei[src[lo:hi]], Ej[dst[lo:hi]]
        cd = np.concatenate([xd, Ej[u_dst]], 0)
        cs = np.concatenate([xs, Ei[u_src]], 0)
        th = None if model.rel is None else model.rel[rel[lo:hi]]
        ath = None if th is None else np.abs(th)
        aq = _abs_forward(model.op, np.abs(xs), ath)
        if model.reciprocal:
            # both queries carry an operator: Q = g(x_s, theta_r), K = g(x_d, theta_{r+R})
            thr = None if model.rel is None else model.rel[model.reverse_rel(rel[lo:hi])]
            ak = _abs_forward(model.op, np.abs(xd), None if thr is None else np.abs(thr))
            acd, acs, ay, ax = np.abs(cd), np.abs(cs), np.abs(xd), np.abs(xs)
            if model.cmp == "cos":
                tq = None if th is None else torch.tensor(th)
                tk = None if thr is None else torch.tensor(thr)
                aq = aq / _norm(O.apply_operator(model.op, torch.tensor(xs), tq).numpy())[:, None]
                ak = ak / _norm(O.apply_operator(model.op, torch.tensor(xd), tk).numpy())[:, None]
                acd, acs = acd / _norm(cd)[:, None], acs / _norm(cs)[:, None]
                ay, ax = ay / _norm(xd)[:, None], ax / _norm(xs)[:, None]
            out.append((np.sum(aq * ay, 1), aq @ acd.T, ak @ acs.T, np.sum(ak * ax, 1)))
            continue
        if model.cmp == "cos":
            gq = O.apply_operator(model.op, torch.tensor(xs), None if th is None else torch.tensor(th)).numpy()
            aq = aq / _norm(gq)[:, None]
            acd = np.abs(cd) / _norm(cd)[:, None]
            th0 = None if model.rel is None else model.rel[rel[lo]]   # the chunk's relation
            gcs = O.apply_operator(model.op, torch.tensor(cs), None if th0 is None else torch.tensor(th0)).numpy()
            acs = _abs_forward(model.op, np.abs(cs), None if th0 is None else np.abs(th0)) / _norm(gcs)[:, None]
            ay = np.abs(xd) / _norm(xd)[:, None]
            Ap = np.sum(aq * ay, 1)
            A0 = aq @ acd.T
            A1 = ay @ acs.T
        else:
            Ap = np.sum(aq * np.abs(xd), 1)
            A0 = aq @ np.abs(cd).T
            ak = _abs_adjoint(model.op, np.abs(xd), ath)
            A1 = np.einsum("ek,tk->et", ak, np.abs(cs))
            if model.op == "translation":
                A1 = A1 + np.sum(ath * np.abs(xd), 1)[:, None]
        out.append((Ap, A0, A1, Ap))
    return out


def gpu_inspect(gm, lo, hi, first_chunk):
    """pbg_inspect_step on edges [lo, hi) of a GpuModel: per chunk a dict of
    float64 arrays p, S0, S1, loss0, loss1, dS0, dS1 cut to the chunk's
    C_c rows and C_c + U columns, and the step loss."""
    pb = gm.pbg, gm.pb
    pbg, p = pb
    n = hi - lo
    C, U = p.C, p.U
    rel_h = None if p.rel_ids is None else p.rel_ids[lo:hi]
    nch = len(O.make_chunks(n, C, rel_h, p.chunking))
    N = C + U
    dev = torch.device("cuda")
    scores = torch.empty(nch * 2 * C * N, dtype=torch.float32, device=dev)
    dscores = torch.empty_like(scores)
    row_loss = torch.empty(nch * 2 * C, dtype=torch.float32, device=dev)
    psides = 2 if p.reciprocal else 1
    pos = torch.empty(nch * psides * C, dtype=torch.float32, device=dev)
    r = None if gm.rel_ids is None else gm.rel_ids[lo:hi]
    loss = pbg.pbg_inspect_step(gm.ctx, p.i, p.j, gm.src[lo:hi], r, gm.dst[lo:hi], C, U, p.S, p.seed,
                                first_chunk, scores, dscores, row_loss, pos, p.chunking, nch)
    S = scores.view(nch, 2, C, N).cpu().numpy().astype(np.float64)
    dS = dscores.view(nch, 2, C, N).cpu().numpy().astype(np.float64)
    L = row_loss.view(nch, 2, C).cpu().numpy().astype(np.float64)
    P_ = pos.view(nch, psides, C).cpu().numpy().astype(np.float64)
    out = []
    for c, clo, chi in O.make_chunks(n, C, rel_h, p.chunking):
        Cc = chi - clo
        Nc = Cc + U
        # outside the chunk's block every output is zero
        assert not S[c, :, Cc:].any() and not S[c, :, :, Nc:].any()
        assert not dS[c, :, Cc:].any() and not dS[c, :, :, Nc:].any()
        rec = {"p": P_[c, 0, :Cc], "S0": S[c, 0, :Cc, :Nc], "S1": S[c, 1, :Cc, :Nc],
               "loss0": L[c, 0, :Cc], "loss1": L[c, 1, :Cc],
               "dS0": dS[c, 0, :Cc, :Nc], "dS1": dS[c, 1, :Cc, :Nc]}
        if p.reciprocal:
            rec["p1"] = P_[c, 1, :Cc]
            assert not P_[c, :, Cc:].any()
        out.append(rec)
    return out, loss


def check_inspection(model, gpu, orc, scales, tol_s, tol_p=1e-5, margin=0.1):
    """Element-wise comparison of one step's forward half (see the bounds in
    test_gpu_inspect).  Returns a report dict: worst error ratios and, for the
    ranking loss, the number of hinge terms whose branch differs (each of them
    must lie within the score error bound of the kink)."""
    rep = {"s_ratio": 0.0, "p_ratio": 0.0, "loss_ratio": 0.0, "ds_ratio": 0.0, "flips": 0, "near_kink": 0}
    for g, o, (Ap0, A0, A1, Ap1) in zip(gpu, orc, scales):
        Cc = o["p"].shape[0]
        valid = np.ones_like(A0, dtype=bool)
        valid[np.arange(Cc), np.arange(Cc)] = False
        for side, A, Ap in ((0, A0, Ap0), (1, A1, Ap1)):
            pk = "p1" if (side == 1 and "p1" in o) else "p"   # each side's positive score
            eP = tol_p * Ap + 1e-30
            rep["p_ratio"] = max(rep["p_ratio"], float(np.max(np.abs(g[pk] - o[pk]) / eP)))
            eS = tol_s * A + 1e-30
            dS_o, dS_g = o[f"dS{side}"], g[f"dS{side}"]
            rep["s_ratio"] = max(rep["s_ratio"], float(np.max((np.abs(g[f"S{side}"] - o[f"S{side}"]) / eS)[valid])))
            K = valid.sum(1)
            if model.loss == "ranking":
                z = margin - o[pk][:, None] + o[f"S{side}"]
                band = eS + eP[:, None]
                near = valid & (np.abs(z) <= band)
                flip = valid & ((dS_g > 0) != (z > 0))
                rep["near_kink"] += int(near.sum())
                rep["flips"] += int(flip.sum())
                assert not (flip & ~near).any(), "a hinge branch differs outside the rounding band of its kink"
                assert np.all(np.isin(dS_g[valid], (0.0, 1.0))) and not dS_g[~valid].any()
                lscale = np.sum(np.where(valid, band + tol_p * np.abs(z), 0.0), 1)
            elif model.loss == "logistic":
                tol_ds = (eS / 4 + tol_s * np.abs(dS_o) * K[:, None]) / K[:, None]
                rep["ds_ratio"] = max(rep["ds_ratio"], float(np.max(np.abs(dS_g - dS_o) / tol_ds)))
                lscale = eP + np.sum(np.where(valid, eS, 0.0), 1) / K + tol_p * np.abs(o[f"loss{side}"])
            else:
                lse_err = np.max(np.where(valid, eS, 0.0), 1) + 2 * eP
                tol_ds = dS_o * (eS + lse_err[:, None] + tol_s) + 1e-12
                rep["ds_ratio"] = max(rep["ds_ratio"], float(np.max(np.abs(dS_g - dS_o) / tol_ds)))
                lscale = lse_err + tol_p * np.abs(o[f"loss{side}"])
            rep["loss_ratio"] = max(rep["loss_ratio"],
                                    float(np.max(np.abs(g[f"loss{side}"] - o[f"loss{side}"]) / (lscale + 1e-30))))
    return rep


# ---------------------------------------------------------------------------
# Error scales of the step gradient.  A float32 sum of terms is within a small
# multiple of the unit round-off times the sum of the terms' absolute values,
# so the bound of each gradient element is eps * A, A = the same gradient
# with every factor replaced by its absolute value: the gradient of
#   sum |dL/dS| * S_abs + |dL/dp| * p_abs
# where S_abs and p_abs are the scores formed from absolute values (inside the
# operator too), as the kernels form them (the source side through the
# adjoint for dot).  For cos the norms are held constant and A doubled (the
# projection of the normalisation's backward adds at most as much again).
# ---------------------------------------------------------------------------
def _abs_fwd_t(op, x, th):
    if op == "identity":
        return x
    if op == "translation":
        return x + th
    if op == "diagonal":
        return x * th
    if op == "linear":
        d = x.shape[-1]
        return (th.reshape(*th.shape[:-1], d, d) @ x.unsqueeze(-1)).squeeze(-1)
    h = x.shape[-1] // 2
    xr, xi, tr, ti = x[..., :h], x[..., h:], th[..., :h], th[..., h:]
    return torch.cat([xr * tr + xi * ti, xr * ti + xi * tr], -1)


def _abs_adj_t(op, y, th):
    if op in ("identity", "translation"):
        return y
    if op == "diagonal":
        return y * th
    if op == "linear":
        d = y.shape[-1]
        return (th.reshape(*th.shape[:-1], d, d).transpose(-1, -2) @ y.unsqueeze(-1)).squeeze(-1)
    h = y.shape[-1] // 2
    yr, yi, tr, ti = y[..., :h], y[..., h:], th[..., :h], th[..., h:]
    return torch.cat([tr * yr + ti * yi, tr * yi + ti * yr], -1)


def gradient_scales(model, i, j, src, rel, dst, C, U, seed, first_chunk, insp, chunking="consecutive"):
    """A of every gradient element of one step (insp: O.inspect_step of the
    same edges at the same state).  Returns ({partition: (row ids, A rows)},
    (relation ids, A rows) or None), ids as in O.step_loss_and_grad."""
    src = np.asarray(src, np.int64)
    dst = np.asarray(dst, np.int64)
    m = src.shape[0]
    step = O.make_chunks(m, C, rel, chunking)
    rel = np.zeros(m, np.int64) if rel is None else np.asarray(rel, np.int64)
    negs = O.step_negatives(model, i, j, step, seed, U, first_chunk)
    touched = {i: [], j: []}
    for (c, lo, hi), (u_dst, u_src) in zip(step, negs):
        touched[i] += [src[lo:hi], u_src]
        touched[j] += [dst[lo:hi], u_dst]
    leaf, ids_of, raw = {}, {}, {}
    for p, lists in touched.items():
        ids = np.unique(np.concatenate(lists))
        raw[p] = torch.tensor(model.emb[p][ids], dtype=torch.float64)
        leaf[p] = raw[p].abs().requires_grad_(True)
        ids_of[p] = ids
    step_rels = np.unique(np.concatenate([rel[lo:hi] for (_, lo, hi) in step]))
    if model.reciprocal:
        step_rels = np.unique(np.concatenate([step_rels, model.reverse_rel(step_rels)]))
    rleaf = None
    if model.rel is not None:
        rraw = torch.tensor(model.rel[step_rels], dtype=torch.float64)
        rleaf = rraw.abs().requires_grad_(True)
    cos = model.cmp == "cos"

    def rows(p, ids, absolute=True):
        k = torch.from_numpy(np.searchsorted(ids_of[p], ids))
        return leaf[p][k] if absolute else raw[p][k]

    for (c, lo, hi), (u_dst, u_src), rec in zip(step, negs, insp):
        r_e = rel[lo:hi]
        th = None if rleaf is None else rleaf[torch.from_numpy(np.searchsorted(step_rels, r_e))]
        xs, xd = rows(i, src[lo:hi]), rows(j, dst[lo:hi])
        cd = torch.cat([xd, rows(j, u_dst)], 0)
        cs = torch.cat([xs, rows(i, u_src)], 0)
        W0 = torch.from_numpy(np.abs(rec["dS0"]))
        W1 = torch.from_numpy(np.abs(rec["dS1"]))
        wp = torch.from_numpy(np.abs(rec["dp"]))
        if model.reciprocal:
            # Q = g(x_s, theta_r) against the destination candidates, K =
            # g(x_d, theta_{r+R}) against the source candidates, a positive
            # score per side
            rk = model.reverse_rel(r_e)
            thk = None if rleaf is None else rleaf[torch.from_numpy(np.searchsorted(step_rels, rk))]
            wp1 = torch.from_numpy(np.abs(rec["dp1"]))
            q, k = _abs_fwd_t(model.op, xs, th), _abs_fwd_t(model.op, xd, thk)
            cdh, csh, yh, xh = cd, cs, xd, xs
            if cos:
                tq = None if rleaf is None else torch.tensor(model.rel[r_e], dtype=torch.float64)
                tk = None if rleaf is None else torch.tensor(model.rel[rk], dtype=torch.float64)
                raw_xs, raw_xd = rows(i, src[lo:hi], False), rows(j, dst[lo:hi], False)
                raw_cd = torch.cat([raw_xd, rows(j, u_dst, False)], 0)
                raw_cs = torch.cat([raw_xs, rows(i, u_src, False)], 0)
                q = q / O._clamped_norm(O.apply_operator(model.op, raw_xs, tq)).unsqueeze(-1)
                k = k / O._clamped_norm(O.apply_operator(model.op, raw_xd, tk)).unsqueeze(-1)
                cdh = cd / O._clamped_norm(raw_cd).unsqueeze(-1)
                csh = cs / O._clamped_norm(raw_cs).unsqueeze(-1)
                yh = xd / O._clamped_norm(raw_xd).unsqueeze(-1)
                xh = xs / O._clamped_norm(raw_xs).unsqueeze(-1)
            L = ((W0 * (q @ cdh.T)).sum() + (W1 * (k @ csh.T)).sum() + (wp * (q * yh).sum(1)).sum()
                 + (wp1 * (k * xh).sum(1)).sum())
            L.backward()
            continue
        if cos:
            thr = None if rleaf is None else torch.tensor(model.rel[r_e], dtype=torch.float64)
            raw_xs, raw_xd = rows(i, src[lo:hi], False), rows(j, dst[lo:hi], False)
            raw_cd = torch.cat([raw_xd, rows(j, u_dst, False)], 0)
            raw_cs = torch.cat([raw_xs, rows(i, u_src, False)], 0)
            nq = O._clamped_norm(O.apply_operator(model.op, raw_xs, thr)).unsqueeze(-1)
            k0 = 0 if rleaf is None else int(np.searchsorted(step_rels, r_e[0]))   # the chunk's relation
            th0 = None if rleaf is None else rleaf[k0].expand(raw_cs.shape[0], -1)
            thr0 = None if rleaf is None else torch.tensor(model.rel[r_e[0]], dtype=torch.float64)
            ncs = O._clamped_norm(O.apply_operator(model.op, raw_cs, thr0)).unsqueeze(-1)
            q = _abs_fwd_t(model.op, xs, th) / nq
            yh = xd / O._clamped_norm(raw_xd).unsqueeze(-1)
            S0 = q @ (cd / O._clamped_norm(raw_cd).unsqueeze(-1)).T
            S1 = yh @ (_abs_fwd_t(model.op, cs, th0) / ncs).T
            pa = (q * yh).sum(1)
        else:
            q = _abs_fwd_t(model.op, xs, th)
            pa = (q * xd).sum(1)
            S0 = q @ cd.T
            S1 = _abs_adj_t(model.op, xd, th) @ cs.T
            if model.op == "translation":
                S1 = S1 + (th * xd).sum(1, keepdim=True)
        L = (W0 * S0).sum() + (W1 * S1).sum() + (wp * pa).sum()
        L.backward()
    k = 2.0 if cos else 1.0
    ent = {p: (ids_of[p], k * leaf[p].grad.numpy()) for p in leaf}
    rl = None if rleaf is None else (step_rels, k * rleaf.grad.numpy())
    return ent, rl


def check_adagrad_step(pb, before, after, grads, rel_grad, scales, rel_scales, lr, eps=1e-5):
    """Teacher-forced step check.  before / after: the GPU's state (float64
    arrays) around the step; grads / rel_grad: the oracle's step gradient at
    `before` (O.step_loss_and_grad); scales: gradient_scales.  Each gradient
    element may differ by eps * A; the bound is carried through the Adagrad
    update exactly to first order (row-wise for entities, element-wise for
    relations), plus the float32 rounding of the stored values.  Rows the step
    does not touch must not change.  Returns the worst ratio error / bound."""
    u = 2.0 ** -23
    worst = 0.0
    for p, (ids, g) in grads.items():
        A = scales[p][1]
        assert np.array_equal(scales[p][0], ids)
        th0, th1 = before["emb"][p], after["emb"][p]
        G0, G1 = before["G"][p], after["G"][p]
        untouched = np.ones(th0.shape[0], bool)
        untouched[ids] = False
        assert np.array_equal(th0[untouched], th1[untouched]) and np.array_equal(G0[untouched], G1[untouched])
        Gw = G0[ids] + np.sum(g * g, 1)
        s = np.sqrt(Gw)[:, None] + 1e-10
        want = th0[ids] - lr * g / s
        nA = np.linalg.norm(A, axis=1, keepdims=True)
        ng = np.linalg.norm(g, axis=1, keepdims=True)
        bth = lr * np.minimum(2.0, 2.0 * eps * (A + np.abs(g) * nA / s) / s) + u * (np.abs(th0[ids]) + np.abs(want)) + 1e-30
        worst = max(worst, float(np.max(np.abs(th1[ids] - want) / bth)))
        bG = 2 * eps * ng[:, 0] * nA[:, 0] + eps * eps * nA[:, 0] ** 2 + u * Gw + 1e-30
        worst = max(worst, float(np.max(np.abs(G1[ids] - Gw) / bG)))
    if rel_grad is not None:
        ids, g = rel_grad
        A = rel_scales[1]
        th0, th1 = before["rel"], after["rel"]
        G0, G1 = before["relG"], after["relG"]
        untouched = np.ones(th0.shape[0], bool)
        untouched[ids] = False
        assert np.array_equal(th0[untouched], th1[untouched])
        Gw = G0[ids] + g * g
        s = np.sqrt(Gw) + 1e-10
        want = th0[ids] - lr * g / s
        bth = lr * np.minimum(2.0, 2.0 * eps * A / s) + u * (np.abs(th0[ids]) + np.abs(want)) + 1e-30
        worst = max(worst, float(np.max(np.abs(th1[ids] - want) / bth)))
        bG = 2 * eps * np.abs(g) * A + (eps * A) ** 2 + u * Gw + 1e-30
        worst = max(worst, float(np.max(np.abs(G1[ids] - Gw) / bG)))
    return worst


def oracle_step_with_scales(pb, om, src, rel, dst, first_chunk, branches=None):
    """The oracle's loss, gradient and gradient error scales of one step of
    these edges at om's state (om is not updated).  With `branches` (ranking)
    the step takes those hinge branches and the scales weigh every term that
    either branch makes active."""
    m = len(src)
    insp = O.inspect_step(om, pb.i, pb.j, src, rel, dst, pb.C, pb.U, pb.seed, first_chunk, pb.chunking)
    if branches is not None:
        for rec, (a0, a1) in zip(insp, branches):
            rec["dS0"] = np.maximum(np.abs(rec["dS0"]), a0)
            rec["dS1"] = np.maximum(np.abs(rec["dS1"]), a1)
    step = O.make_chunks(m, pb.C, rel, pb.chunking)
    negs = O.step_negatives(om, pb.i, pb.j, step, pb.seed, pb.U, first_chunk)
    rel_a = np.zeros(m, np.int64) if rel is None else rel
    loss, grads, rel_grad = O.step_loss_and_grad(om, pb.i, pb.j, src, rel_a, dst, step, negs, branches=branches)
    ent_sc, rel_sc = gradient_scales(om, pb.i, pb.j, src, rel, dst, pb.C, pb.U, pb.seed, first_chunk, insp,
                                     pb.chunking)
    return loss, grads, rel_grad, ent_sc, rel_sc


def teacher_forced_step(gm, lo, hi, first_chunk, eps):
    """One step of edges [lo, hi) of a GpuModel (one call, at most one step),
    checked against the oracle loaded with the GPU's step-start state: the
    ranking census and branches (hinge terms within eps * A of the kink may
    take the GPU's branch), the step loss within eps relative, and every
    parameter and accumulator within the Adagrad-propagated bound of a
    gradient error eps * A.  Returns (census report or None, gpu loss,
    oracle loss, worst error / bound)."""
    pb = gm.pb
    before = gm.state()
    om = O.Model.create(pb.n, pb.P, pb.R, pb.d, pb.op, pb.cmp, pb.loss, pb.margin, before["emb"],
                        before.get("rel"), G_parts=before["G"], relG=before.get("relG"),
                        reciprocal=pb.reciprocal)
    src, dst = pb.src[lo:hi], pb.dst[lo:hi]
    rel = None if pb.rel_ids is None else pb.rel_ids[lo:hi]
    rep = branches = None
    if pb.loss == "ranking":
        gpu, _ = gpu_inspect(gm, lo, hi, first_chunk)
        orc = O.inspect_step(om, pb.i, pb.j, src, rel, dst, pb.C, pb.U, pb.seed, first_chunk, pb.chunking)
        scales = score_scales(om, pb.i, pb.j, src, rel, dst, pb.C, pb.U, pb.seed, first_chunk, pb.chunking)
        rep = check_inspection(om, gpu, orc, scales, eps)
        branches = [(g["dS0"] > 0, g["dS1"] > 0) for g in gpu]
        del gpu, orc, scales
    gl = gm.train(lo, hi, first_chunk)
    after = gm.state()
    ol, grads, rel_grad, ent_sc, rel_sc = oracle_step_with_scales(pb, om, src, rel, dst, first_chunk, branches)
    worst = check_adagrad_step(pb, before, after, grads, rel_grad, ent_sc, rel_sc, pb.lr, eps)
    return rep, gl, ol, worst
