"""Seeded synthetic graphs shaped like the paper's workloads.

The paper trains on LiveJournal, FB15k, full Freebase and Twitter (Sec. 5);
none of these datasets is available, so every input here is synthetic: node
ids drawn from bounded Zipf laws over a seeded random permutation (heavy-tailed
degrees, as in the social and knowledge graphs of Sec. 5), relation ids from a
Zipf law, embeddings from N(0, sigma) with sigma = 0.001 and relation
parameters at the operator's identity element.

This module holds no arithmetic of the method itself (no scores, losses,
gradients, partition maps or bucketing): it only draws inputs.  Both the HIP
path and the CPU oracle are fed from it.
"""

from __future__ import annotations

from dataclasses import dataclass

import numpy as np


def rng_for(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


class BoundedZipf:
    """P(rank k) proportional to k**-s for k = 1..n, sampled by inverse CDF;
    rank k maps to node perm[k-1] (a seeded permutation of 0..n-1)."""

    def __init__(self, n: int, s: float, rng: np.random.Generator):
        self.n = int(n)
        w = np.arange(1, self.n + 1, dtype=np.float64) ** (-float(s))
        cdf = np.cumsum(w)
        self.cdf = cdf / cdf[-1]
        self.perm = rng.permutation(self.n).astype(np.int64)

    def sample(self, rng: np.random.Generator, size: int, block: int = 1 << 24) -> np.ndarray:
        out = np.empty(size, dtype=np.int64)
        for lo in range(0, size, block):
            hi = min(size, lo + block)
            r = np.searchsorted(self.cdf, rng.random(hi - lo), side="right")
            np.minimum(r, self.n - 1, out=r)
            out[lo:hi] = self.perm[r]
        return out


def zipf_edges(n: int, E: int, s_src: float, s_dst: float, rng, resample_self_loops=True):
    """E directed edges with Zipf out-degree (source law) and in-degree
    (destination law); self-loops are redrawn on the destination side."""
    zs = BoundedZipf(n, s_src, rng)
    zd = zs if s_dst == s_src else BoundedZipf(n, s_dst, rng)
    src = zs.sample(rng, E)
    dst = zd.sample(rng, E)
    if resample_self_loops and n > 1:
        bad = np.nonzero(src == dst)[0]
        while bad.size:
            dst[bad] = zd.sample(rng, bad.size)
            bad = bad[src[bad] == dst[bad]]
    return src, dst


def init_embeddings(rows: int, d: int, rng, sigma: float = 1e-3) -> np.ndarray:
    """N(0, sigma) float32 rows (sigma is the standard deviation)."""
    return (rng.standard_normal((rows, d), dtype=np.float32) * np.float32(sigma))


def identity_relation_params(op: str, R: int, d: int) -> np.ndarray | None:
    """Relation parameters that make g the identity map: translation 0,
    diagonal 1, complex 1 + 0i, linear the identity matrix."""
    if op == "identity":
        return None
    if op == "translation":
        return np.zeros((R, d), np.float32)
    if op == "diagonal":
        return np.ones((R, d), np.float32)
    if op == "complex_diagonal":
        p = np.zeros((R, d), np.float32)
        p[:, : d // 2] = 1.0
        return p
    if op == "linear":
        return np.broadcast_to(np.eye(d, dtype=np.float32).reshape(1, d * d), (R, d * d)).copy()
    raise ValueError(op)


def perturbed_relation_params(op: str, R: int, d: int, rng, scale: float = 0.3):
    """Identity-element parameters plus seeded noise: used by tests so that
    every operator term is exercised (identity parameters hide some of them)."""
    p = identity_relation_params(op, R, d)
    if p is None:
        return None
    return (p + scale * rng.standard_normal(p.shape, dtype=np.float32)).astype(np.float32)


@dataclass
class Workload:
    """One synthetic training problem (global ids unless `local` is set)."""
    name: str
    n: int
    P: int
    R: int
    d: int
    op: str
    cmp: str
    loss: str
    margin: float
    C: int
    U: int
    S: int
    lr: float
    seed: int
    src: np.ndarray
    rel: np.ndarray | None
    dst: np.ndarray
    bucket: tuple | None = None     # (i, j) when src/dst are local ids of one bucket
    held_src: np.ndarray | None = None
    held_rel: np.ndarray | None = None
    held_dst: np.ndarray | None = None

    @property
    def E(self) -> int:
        return int(self.src.shape[0])


def _zipf_relations(R: int, E: int, s: float, rng):
    if R == 1:
        return np.zeros(E, np.int32)
    return BoundedZipf(R, s, rng).sample(rng, E).astype(np.int32)


def tiny_social(n=10_000, E=100_000, d=32, C=100, U=100, S=40, seed=20190001):
    """Tiny social graph: one relation, one partition, Zipf(1.1) endpoints;
    identity operator, dot, ranking loss (margin 0.1), lr 0.1."""
    rng = rng_for(seed)
    src, dst = zipf_edges(n, E, 1.1, 1.1, rng)
    return Workload("tiny_social", n, 1, 1, d, "identity", "dot", "ranking", 0.1,
                    C, U, S, 0.1, seed, src, None, dst)


def social_network(n=4_847_571, E=68_993_773, d=128, C=1000, U=1000, S=40, seed=20190002):
    """Social-network-shaped graph (LiveJournal counts, Sec. 5.2): Zipf(1.05)
    out- and in-degree, one relation, one partition; translation operator,
    cos comparator, ranking loss (margin 0.1), lr 0.1."""
    rng = rng_for(seed)
    src, dst = zipf_edges(n, E, 1.05, 1.05, rng)
    return Workload("social_network", n, 1, 1, d, "translation", "cos", "ranking", 0.1,
                    C, U, S, 0.1, seed, src, None, dst)


def knowledge_graph(n=15_000, R=1_345, n_triples=533_000, n_held=50_000, d=400,
                    C=1000, U=1000, S=40, seed=20190003):
    """Knowledge-graph-shaped multi-relation graph (FB15k sizes, Sec. 5.4):
    Zipf(1.2) relation frequencies over a permuted relation list; per relation,
    Zipf(1.0) endpoints over per-relation permutations; unique triples without
    self-loops, shuffled and split into train / held-out; complex_diagonal
    operator, dot comparator, softmax loss, lr 0.1."""
    rng = rng_for(seed)
    rel_law = BoundedZipf(R, 1.2, rng)
    w = np.arange(1, n + 1, dtype=np.float64) ** -1.0
    cdf = np.cumsum(w)
    cdf /= cdf[-1]
    perms = {}

    def perm(r):
        if r not in perms:
            sub = rng_for(seed * 7919 + r)
            perms[r] = (sub.permutation(n), sub.permutation(n))
        return perms[r]

    keys = np.empty(0, np.int64)
    parts = []
    count = 0
    while count < n_triples:
        need = int((n_triples - count) * 1.3) + 64
        rels = rel_law.sample(rng, need)
        s = np.minimum(np.searchsorted(cdf, rng.random(need), side="right"), n - 1)
        t = np.minimum(np.searchsorted(cdf, rng.random(need), side="right"), n - 1)
        for r in np.unique(rels):
            idx = np.nonzero(rels == r)[0]
            ps_, pd_ = perm(int(r))
            s[idx] = ps_[s[idx]]
            t[idx] = pd_[t[idx]]
        ok = s != t
        rels, s, t = rels[ok], s[ok], t[ok]
        k = (s * R + rels) * n + t
        allk = np.concatenate([keys, k])
        _, first = np.unique(allk, return_index=True)
        first = np.sort(first[first >= keys.size]) - keys.size
        first = first[: n_triples - count]
        keys = np.concatenate([keys, k[first]])
        parts.append(np.stack([s[first], rels[first], t[first]], 1))
        count += first.size
    arr = np.concatenate(parts, 0)
    arr = arr[rng.permutation(len(arr))]
    train, held = arr[: n_triples - n_held], arr[n_triples - n_held:]
    return Workload("knowledge_graph", n, 1, R, d, "complex_diagonal", "dot", "softmax", 0.1,
                    C, U, S, 0.1, seed, train[:, 0].copy(), train[:, 1].astype(np.int32),
                    train[:, 2].copy(), held_src=held[:, 0].copy(),
                    held_rel=held[:, 1].astype(np.int32), held_dst=held[:, 2].copy())


def big_bucket(n=121_216_723, P=16, rows_i=7_576_046, rows_j=7_576_046, R=5_000,
               E_bucket=9_375_000, d=100, C=1000, U=1000, S=40, i=3, j=7, seed=20190004):
    """One bucket (i, j) of a large partitioned knowledge-graph-shaped run
    (full-Freebase sizes, Sec. 5.4: 121,216,723 entities in 16 partitions of
    7,576,046 rows): edges drawn directly as local ids of partitions i and j
    (rows_i, rows_j rows) with Zipf(1.0) endpoints, relations Zipf(1.3);
    diagonal operator, dot comparator, ranking loss (margin 0.1), lr 0.1."""
    rng = rng_for(seed)
    src = BoundedZipf(rows_i, 1.0, rng).sample(rng, E_bucket)
    dst = BoundedZipf(rows_j, 1.0, rng).sample(rng, E_bucket)
    rel = _zipf_relations(R, E_bucket, 1.3, rng)
    return Workload("big_bucket", n, P, R, d, "diagonal", "dot", "ranking", 0.1,
                    C, U, S, 0.1, seed, src, rel, dst, bucket=(i, j))


def follower_graph(n=41_652_230, E=1_468_365_182, P=8, d=100, C=1000, U=1000, S=40,
                   seed=20190005):
    """Follower-graph-shaped partitioned epoch (Twitter counts, Sec. 5.5):
    Zipf(1.2) sources, Zipf(0.9) destinations, one relation, P partitions;
    linear operator, dot comparator, logistic loss, lr 0.1."""
    rng = rng_for(seed)
    src, dst = zipf_edges(n, E, 1.2, 0.9, rng)
    return Workload("follower_graph", n, P, 1, d, "linear", "dot", "logistic", 0.1,
                    C, U, S, 0.1, seed, src, None, dst)


def prevalence_candidates(src, dst, n: int, k: int, rng) -> np.ndarray:
    """k entity ids drawn with replacement in proportion to each entity's
    count among the training edges' endpoints (its prevalence), as the
    candidates of a sampled-candidate evaluation; int32 [k]."""
    deg = np.bincount(np.concatenate([np.asarray(src, np.int64), np.asarray(dst, np.int64)]),
                      minlength=n).astype(np.float64)
    return rng.choice(n, size=k, replace=True, p=deg / deg.sum()).astype(np.int32)


def partition_embeddings(rows, d: int, rng, sigma: float = 1e-3):
    """Initial N(0, sigma) embeddings for partitions of the given row counts."""
    return [init_embeddings(int(r), d, rng, sigma) for r in rows]


# ---------------------------------------------------------------------------
# On-device generation for the large workloads (same recipes, drawn with a
# seeded torch generator on the GPU: seconds instead of minutes on the host).
# ---------------------------------------------------------------------------
def _torch():
    import torch
    return torch


def device_generator(seed: int, device="cuda"):
    torch = _torch()
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    return g


def zipf_device(n: int, s: float, size: int, gen, device="cuda", block: int = 1 << 26):
    """Bounded Zipf(s) over n ranks mapped through a seeded permutation."""
    torch = _torch()
    w = torch.arange(1, n + 1, dtype=torch.float64, device=device).pow_(-float(s))
    cdf = torch.cumsum(w, 0)
    cdf /= cdf[-1].clone()
    perm = torch.randperm(n, generator=gen, device=device)
    out = torch.empty(size, dtype=torch.int64, device=device)
    for lo in range(0, size, block):
        hi = min(size, lo + block)
        u = torch.rand(hi - lo, generator=gen, device=device, dtype=torch.float64)
        r = torch.searchsorted(cdf, u, right=True).clamp_(max=n - 1)
        out[lo:hi] = perm[r]
    return out, (cdf, perm)


def zipf_edges_device(n: int, E: int, s_src: float, s_dst: float, gen, device="cuda"):
    torch = _torch()
    src, _ = zipf_device(n, s_src, E, gen, device)
    dst, (cdf_d, perm_d) = zipf_device(n, s_dst, E, gen, device)
    while True:
        bad = torch.nonzero(src == dst).flatten()
        if bad.numel() == 0:
            break
        u = torch.rand(bad.numel(), generator=gen, device=device, dtype=torch.float64)
        dst[bad] = perm_d[torch.searchsorted(cdf_d, u, right=True).clamp_(max=n - 1)]
    return src, dst


def init_embeddings_device(rows: int, d: int, gen, sigma: float = 1e-3, device="cuda"):
    torch = _torch()
    return torch.randn((rows, d), generator=gen, device=device, dtype=torch.float32).mul_(sigma)


def social_network_device(n=4_847_571, E=68_993_773, d=128, seed=20190002, device="cuda"):
    """The social-network-shaped workload (see social_network) drawn on the
    device: (src, dst) int32 device tensors and the initial embedding table."""
    torch = _torch()
    gen = device_generator(seed, device)
    src, dst = zipf_edges_device(n, E, 1.05, 1.05, gen, device)
    emb = init_embeddings_device(n, d, gen, 1e-3, device)
    return src.to(torch.int32), dst.to(torch.int32), emb
