"""CPU oracle for the PyTorch-BigGraph per-bucket training step (Lerer et al.,
"PyTorch-BigGraph: A Large-scale Graph Embedding System", SysML 2019).

THIS MODULE IS TEST INFRASTRUCTURE.  Only the test suite, the package smoke
check and the benchmark's CPU-baseline leg may import or run it.  The product
path (the HIP library and its Python binding) never imports it, and this module
imports nothing from the product path.

It is a plain, slow, fp64 restatement of what the method computes, step by
step, in the order and notation of the paper:

  O1  partition map            Sec. 4.1 (entities split into P parts; "uniformly")
  O2  edge bucketing           Sec. 4.1 (bucket (p1, p2) by source/destination partition)
  O3  chunks and steps         Sec. 4.3 (a batch is broken into chunks that share negatives)
  O4  uniform negatives        Sec. 4.3 + Philox4x32-10 (Salmon et al., SC'11)
  O5  relation operators       Sec. 3.1, operator/comparator table
  O6  comparators              Sec. 3.1, operator/comparator table
  O7  chunk scores             Sec. 3.1 score function f, Sec. 4.3 batched negatives, Fig. 3
  O8  losses                   Sec. 3.1 ranking objective, logistic and softmax alternatives
  O9  step gradient            Sec. 3.1 minibatch SGD (exact gradient by torch autograd, fp64)
  O10 row-wise Adagrad         Sec. 3.1 (accumulator summed over each embedding vector)
  O11 scoring and ranking      Sec. 5 filtered link-prediction metrics (MRR, Hits@10)
  --  bucket order             Sec. 4.1 / Fig. 1 right ("inside-out")

Readings of points where the paper is silent or garbled (each one is listed,
with its reason, in the design notes of the repository):
  * ranking loss is max(0, margin - f(e) + f(e')) (the printed sign would reward
    negatives, while f is maximised on true edges);
  * g acts on the source embedding only, for both corruption sides;
  * complex layout is [re(0..h-1) | im(0..h-1)], h = d/2;
  * linear operator is g(x) = A x with A row-major d x d;
  * chunk c of a bucket holds edges [cC, min((c+1)C, m)); a step holds S chunks;
    relation-grouped chunks (Sec. 4.3, batches sharing a relation type) cut
    each relation's run of relation-sorted edges into chunks of C, the run's
    last chunk holding the rest;
  * separate uniform negative sets per side, U each, also for the short last chunk;
  * only the induced positive (the diagonal t = e) is excluded from the
    in-chunk negatives;
  * logistic loss: positive once per side, negatives averaged over K_e;
  * softmax loss: one softmax per side over {p_e} and that side's negatives;
  * losses are summed over edges, negatives, sides and chunks;
  * cos clamps each norm at 1e-12; Adagrad uses eps = 1e-10 after the root and
    starts from G = 0; relations use element-wise Adagrad with the same lr;
  * the gradient of a step is taken at the step-start parameters (batch-
    synchronous update of S chunks; S = 40 by default);
  * rank ties count against the model; filtered = known triples removed;
  * reciprocal predicates (Sec. 5.4, separate relation parameters for the
    source and destination negatives): relation r keeps a second parameter
    row r + R; the source-corruption side scores sim(g(x_d, theta_{r+R}), x_t)
    with its own positive sim(g(x_d, theta_{r+R}), x_s), while the destination
    side and the edge score f keep theta_r;
  * entity types (Sec. 3.1 negatives of the relation's types, Sec. 4.1
    unpartitioned types): each relation fixes a source and a destination type,
    a type is split into P parts or kept whole (its partition index is 0), and
    an edge's bucket is (partition of s in its type, partition of d in its
    type).  A bucket's edges, sorted by relation, train in runs of consecutive
    chunks whose relations share the (source type, destination type) pair;
    the negatives of a run's chunks come from the tables of that pair, and a
    step never spans two runs;
  * per-relation edge weights (Sec. 1 and 6, per-relation configuration):
    the weight of an edge's relation multiplies that edge's loss on both sides.
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np
import torch

OPERATORS = ("identity", "translation", "diagonal", "linear", "complex_diagonal")
COMPARATORS = ("dot", "cos")
LOSSES = ("ranking", "logistic", "softmax")

EPS_NORM = 1e-12      # cos: each norm is clamped at this value
EPS_ADAGRAD = 1e-10   # Adagrad: added after the square root

_F64 = torch.float64


# --------------------------------------------------------------------------
# O1 partition map (Sec. 4.1: P parts sized to fit memory, assigned uniformly)
# --------------------------------------------------------------------------
def partition_size(n: int, P: int) -> int:
    """Rows in every partition but possibly the last: ceil(n / P)."""
    return -(-int(n) // int(P))


def partition_rows(n: int, P: int, p: int) -> int:
    """Rows of partition p; the last one holds the remainder."""
    ps = partition_size(n, P)
    return max(0, min(ps, int(n) - p * ps))


def partition_of(v, n: int, P: int):
    """Partition of global entity id v (contiguous ranges of ceil(n/P) ids)."""
    return np.asarray(v, dtype=np.int64) // partition_size(n, P)


def local_id(v, n: int, P: int):
    """Row of global id v inside its partition."""
    v = np.asarray(v, dtype=np.int64)
    return v - partition_of(v, n, P) * partition_size(n, P)


# --------------------------------------------------------------------------
# O2 edge bucketing (Sec. 4.1: edge (s, r, d) goes to bucket (part(s), part(d)))
# --------------------------------------------------------------------------
def bucket_edges(src, rel, dst, n: int, P: int):
    """Group edges by bucket id b = part(src) * P + part(dst), keeping the input
    order inside each bucket.  Returns (offsets[P*P+1] int64, src_local int32,
    rel int32, dst_local int32)."""
    src = np.asarray(src, dtype=np.int64)
    dst = np.asarray(dst, dtype=np.int64)
    rel = np.asarray(rel, dtype=np.int32)
    if src.size and (src.min() < 0 or dst.min() < 0 or src.max() >= n or dst.max() >= n):
        raise ValueError("entity id out of range")
    b = partition_of(src, n, P) * P + partition_of(dst, n, P)
    order = np.argsort(b, kind="stable")
    counts = np.bincount(b, minlength=P * P)
    offsets = np.zeros(P * P + 1, dtype=np.int64)
    offsets[1:] = np.cumsum(counts)
    return (offsets,
            local_id(src, n, P)[order].astype(np.int32),
            rel[order].astype(np.int32),
            local_id(dst, n, P)[order].astype(np.int32))


# --------------------------------------------------------------------------
# bucket order (Sec. 4.1 / Fig. 1 right): every bucket after the first shares a
# partition with a bucket trained before it
# --------------------------------------------------------------------------
def inside_out_order(P: int):
    """(0,0), then for k = 1..P-1 the shell (k,0),(0,k),(k,1),(1,k),...,
    (k,k-1),(k-1,k),(k,k)."""
    order = [(0, 0)]
    for k in range(1, P):
        for m in range(k):
            order.append((k, m))
            order.append((m, k))
        order.append((k, k))
    return order


# --------------------------------------------------------------------------
# O4 Philox4x32-10 (Salmon, Moraes, Dror, Shaw: "Parallel Random Numbers: As
# Easy as 1, 2, 3", SC'11) and the uniform negative map
# --------------------------------------------------------------------------
_MASK32 = np.uint64(0xFFFFFFFF)
_PHILOX_M = (np.uint64(0xD2511F53), np.uint64(0xCD9E8D57))
_PHILOX_W = (np.uint64(0x9E3779B9), np.uint64(0xBB67AE85))


def philox4x32_10(ctr, key):
    """Counter-based generator: ten rounds of the Philox S-box network on a
    128-bit counter under a 64-bit key.  `ctr` has a trailing axis of 4 words,
    `key` a trailing axis of 2 words (values < 2**32).  Returns uint64 words."""
    ctr = np.asarray(ctr, dtype=np.uint64)
    key = np.asarray(key, dtype=np.uint64)
    x = [ctr[..., w] & _MASK32 for w in range(4)]
    k0 = key[..., 0] & _MASK32
    k1 = key[..., 1] & _MASK32
    for rnd in range(10):
        if rnd:
            k0 = (k0 + _PHILOX_W[0]) & _MASK32
            k1 = (k1 + _PHILOX_W[1]) & _MASK32
        prod0 = _PHILOX_M[0] * x[0]          # < 2**64: exact in uint64
        prod1 = _PHILOX_M[1] * x[2]
        hi0, lo0 = prod0 >> np.uint64(32), prod0 & _MASK32
        hi1, lo1 = prod1 >> np.uint64(32), prod1 & _MASK32
        x = [hi1 ^ x[1] ^ k0, lo1, hi0 ^ x[3] ^ k1, lo0]
    return np.stack(x, axis=-1)


def uniform_negatives(seed: int, bucket: int, chunk: int, side: int, U: int, n_rows: int):
    """U uniform local ids in [0, n_rows) for one chunk and side (0: destination
    corruption, drawn from the destination partition; 1: source corruption,
    drawn from the source partition).  Word k comes from counter
    (k >> 2, chunk, bucket, side) under key (seed low, seed high); the id is
    floor(w * n_rows / 2**32), computed exactly."""
    k = np.arange(U, dtype=np.uint64)
    ctr = np.stack([k >> np.uint64(2),
                    np.full_like(k, chunk & 0xFFFFFFFF),
                    np.full_like(k, bucket & 0xFFFFFFFF),
                    np.full_like(k, side)], axis=-1)
    key = np.array([seed & 0xFFFFFFFF, (seed >> 32) & 0xFFFFFFFF], dtype=np.uint64)
    words = philox4x32_10(ctr, np.broadcast_to(key, (U, 2)))
    w = words[np.arange(U), (k & np.uint64(3)).astype(np.int64)]
    return ((w * np.uint64(n_rows)) >> np.uint64(32)).astype(np.int64)


# --------------------------------------------------------------------------
# O5 relation operators and O6 comparators (Sec. 3.1, operator table)
# --------------------------------------------------------------------------
def relation_param_width(op: str, d: int) -> int:
    """Floats of one relation's parameter vector."""
    return {"identity": 0, "translation": d, "diagonal": d,
            "linear": d * d, "complex_diagonal": d}[op]


def apply_operator(op: str, x, theta):
    """g(x, theta_r) on the last axis of x.  theta has the same leading shape as
    x (one parameter row per vector) or broadcasts against it."""
    if op == "identity":
        return x
    if op == "translation":
        return x + theta
    if op == "diagonal":
        return x * theta
    if op == "linear":
        d = x.shape[-1]
        A = theta.reshape(*theta.shape[:-1], d, d)          # row-major A_r
        return (A @ x.unsqueeze(-1)).squeeze(-1)            # (A x)_k = sum_l A_kl x_l
    if op == "complex_diagonal":
        h = x.shape[-1] // 2
        xr, xi = x[..., :h], x[..., h:]
        tr, ti = theta[..., :h], theta[..., h:]
        return torch.cat([xr * tr - xi * ti, xr * ti + xi * tr], dim=-1)
    raise ValueError(op)


def _clamped_norm(x):
    return torch.clamp(torch.linalg.vector_norm(x, dim=-1), min=EPS_NORM)


def compare_all(cmp: str, a, b):
    """sim(a_e, b_t) for every row e of a and row t of b.  For complex
    embeddings in the split layout, Re<a, conj(b)> is this real dot."""
    dots = a @ b.transpose(-1, -2)
    if cmp == "dot":
        return dots
    if cmp == "cos":
        return dots / (_clamped_norm(a).unsqueeze(-1) * _clamped_norm(b).unsqueeze(-2))
    raise ValueError(cmp)


def compare_rows(cmp: str, a, b):
    """sim(a_e, b_e) row by row."""
    dots = (a * b).sum(-1)
    if cmp == "dot":
        return dots
    if cmp == "cos":
        return dots / (_clamped_norm(a) * _clamped_norm(b))
    raise ValueError(cmp)


# --------------------------------------------------------------------------
# model state: partitions of entity embeddings plus relation parameters
# --------------------------------------------------------------------------
@dataclass
class Model:
    n: int
    P: int
    R: int
    d: int
    op: str
    cmp: str
    loss: str
    margin: float = 0.1
    emb: dict = field(default_factory=dict)      # p -> (rows, d) float64
    G: dict = field(default_factory=dict)        # p -> (rows,) float64, row-summed Adagrad
    rel: np.ndarray | None = None                # (R or 2R, width) float64
    relG: np.ndarray | None = None               # (R or 2R, width) float64, element-wise Adagrad
    reciprocal: bool = False                     # rows R..2R-1 of rel: the source-side parameters
    weights: np.ndarray | None = None            # (R,) per-relation edge weights (None: all 1)
    types: "EntityTypes | None" = None           # entity types (None: one partitioned type; emb keyed
                                                 # by partition p, else by (type, partition))

    @staticmethod
    def create(n, P, R, d, op, cmp, loss, margin, emb_parts, rel_params=None,
               G_parts=None, relG=None, reciprocal=False):
        if op not in OPERATORS or cmp not in COMPARATORS or loss not in LOSSES:
            raise ValueError("unknown operator, comparator or loss")
        if op == "complex_diagonal" and d % 2:
            raise ValueError("complex_diagonal needs an even dimension")
        m = Model(n, P, R, d, op, cmp, loss, float(margin), reciprocal=bool(reciprocal))
        for p in range(P):
            e = np.array(emb_parts[p], dtype=np.float64)
            assert e.shape == (partition_rows(n, P, p), d)
            m.emb[p] = e
            m.G[p] = (np.zeros(e.shape[0]) if G_parts is None
                      else np.array(G_parts[p], dtype=np.float64))
        width = relation_param_width(op, d)
        rows = 2 * R if reciprocal else R
        if width:
            m.rel = np.array(rel_params, dtype=np.float64).reshape(rows, width)
            m.relG = np.zeros_like(m.rel) if relG is None else np.array(relG, np.float64).reshape(rows, width)
        return m

    @staticmethod
    def create_typed(types: "EntityTypes", P, R, d, op, cmp, loss, margin, tables, rel_params=None,
                     weights=None, reciprocal=False):
        """A model over several entity types: tables maps (type, partition) to
        its (rows, d) embedding array, for every partition of every type."""
        if len(types.rel_src) != R or len(types.rel_dst) != R:
            raise ValueError("every relation needs a source and a destination type")
        m = Model.create(P, P, R, d, op, cmp, loss, margin, [np.zeros((1, d)) for _ in range(P)],
                         rel_params, reciprocal=reciprocal)
        m.n = None
        m.emb, m.G = {}, {}
        for t in range(types.count):
            for p in range(types.parts(t, P)):
                e = np.array(tables[(t, p)], dtype=np.float64)
                assert e.shape == (types.rows(t, P, p), d), (t, p, e.shape)
                m.emb[(t, p)] = e
                m.G[(t, p)] = np.zeros(e.shape[0])
        m.types = types
        if weights is not None:
            m.weights = np.array(weights, dtype=np.float64).reshape(R)
        return m

    def edge_weights(self, r):
        """Weight of each edge from its relation (1 without weights)."""
        r = np.asarray(r, dtype=np.int64)
        return np.ones(r.shape) if self.weights is None else self.weights[r]

    def reverse_rel(self, r):
        """Parameter row of the source side of relation r (reciprocal: r + R)."""
        return np.asarray(r, dtype=np.int64) + (self.R if self.reciprocal else 0)


@dataclass
class EntityTypes:
    """Entity types of a graph: counts[t] entities of type t, each type split
    into P contiguous parts or kept whole, and the (source, destination) type of
    every relation."""
    counts: list
    partitioned: list
    rel_src: np.ndarray
    rel_dst: np.ndarray

    @property
    def count(self):
        return len(self.counts)

    def parts(self, t, P):
        return P if self.partitioned[t] else 1

    def rows(self, t, P, p):
        return partition_rows(self.counts[t], self.parts(t, P), p)

    def tables(self, r, i, j):
        """(source table, destination table) of relation r's edges in bucket
        (i, j), or None when its types cannot have edges there (a whole type
        lives in partition 0)."""
        st, dt = int(self.rel_src[r]), int(self.rel_dst[r])
        if (not self.partitioned[st] and i != 0) or (not self.partitioned[dt] and j != 0):
            return None
        return (st, i), (dt, j)


def bucket_edges_typed(src, rel, dst, types: EntityTypes, P: int):
    """Bucketing with entity types (Sec. 4.1): ids are per type; an edge goes
    to bucket part(s) * P + part(d), part(v) its partition within its type (0
    for a type kept whole), keeping the input order inside each bucket.
    Returns (offsets[P*P+1], src_local, rel, dst_local) as bucket_edges."""
    src = np.asarray(src, dtype=np.int64)
    dst = np.asarray(dst, dtype=np.int64)
    rel = np.asarray(rel, dtype=np.int64)
    st, dt = np.asarray(types.rel_src)[rel], np.asarray(types.rel_dst)[rel]
    ns = np.asarray(types.counts, np.int64)[st]
    nd = np.asarray(types.counts, np.int64)[dt]
    if src.size and (src.min() < 0 or dst.min() < 0 or np.any(src >= ns) or np.any(dst >= nd)):
        raise ValueError("entity id out of range for its type")
    parts = np.array([types.parts(t, P) for t in range(types.count)], np.int64)
    ps_s = -(-ns // parts[st])
    ps_d = -(-nd // parts[dt])
    ps_part, pd_part = src // ps_s, dst // ps_d
    b = ps_part * P + pd_part
    order = np.argsort(b, kind="stable")
    counts = np.bincount(b, minlength=P * P)
    offsets = np.zeros(P * P + 1, dtype=np.int64)
    offsets[1:] = np.cumsum(counts)
    return (offsets, (src - ps_part * ps_s)[order].astype(np.int32), rel[order].astype(np.int32),
            (dst - pd_part * ps_d)[order].astype(np.int32))


# --------------------------------------------------------------------------
# O7 chunk scores and O8 losses
# --------------------------------------------------------------------------
def _softplus(x):
    return torch.logaddexp(x, torch.zeros_like(x))


def chunk_scores(op, cmp, xs, xd, theta_e, rel_e, cand_dst, cand_src, theta_of):
    """Scores of one chunk, straight from f(s, r, d) = sim(g(theta_s, theta_r), theta_d).

    xs, xd     (C, d)  source / destination rows of the chunk's edges
    theta_e    (C, w)  relation parameters of each edge (None for identity)
    rel_e      (C,)    relation ids (numpy) used to group the source corruptions
    cand_dst   (N, d)  destination candidates: the chunk's destinations, then U uniform rows
    cand_src   (N, d)  source candidates: the chunk's sources, then U uniform rows
    theta_of   relation id -> parameter row (torch)

    Returns p (C,), S0 (C, N) with S0[e, t] = f(s_e, r_e, cand_dst[t]) and
    S1 (C, N) with S1[e, t] = f(cand_src[t], r_e, d_e)."""
    q = apply_operator(op, xs, theta_e)
    p = compare_rows(cmp, q, xd)
    S0 = compare_all(cmp, q, cand_dst)
    rows = []
    order = []
    for r in np.unique(rel_e):
        idx = np.nonzero(rel_e == r)[0]
        g_cand = apply_operator(op, cand_src, theta_of(int(r)))   # g applied to every candidate
        rows.append(compare_all(cmp, xd[idx], g_cand))
        order.append(idx)
    S1 = torch.cat(rows, 0)[np.argsort(np.concatenate(order), kind="stable")]
    return p, S0, S1


def chunk_scores_reciprocal(op, cmp, xs, xd, theta_fwd, theta_rev, cand_dst, cand_src):
    """Scores of one chunk with reciprocal predicates (Sec. 5.4): each side
    compares the operator applied to the entity it keeps with the raw
    candidates of the side it corrupts.

    theta_fwd (C, w) theta_r of each edge, theta_rev (C, w) theta_{r+R} (None
    for identity).  Returns p0 (C,) = sim(g(x_s, theta_r), x_d), p1 (C,) =
    sim(g(x_d, theta_{r+R}), x_s), S0 (C, N) with S0[e, t] = sim(g(x_s,
    theta_r), cand_dst[t]) and S1 (C, N) with S1[e, t] = sim(g(x_d,
    theta_{r+R}), cand_src[t])."""
    q = apply_operator(op, xs, theta_fwd)
    k = apply_operator(op, xd, theta_rev)
    return (compare_rows(cmp, q, xd), compare_rows(cmp, k, xs),
            compare_all(cmp, q, cand_dst), compare_all(cmp, k, cand_src))


def side_loss(loss, margin, p, S, valid, active=None):
    """Per-edge loss of one corruption side over its valid negatives.

    `active` (ranking only, optional) fixes which hinge terms count: term t of
    edge e contributes (margin - p_e + n_t) * active[e, t] instead of
    max(0, margin - p_e + n_t).  With active = [margin - p + n > 0] the two
    agree; a caller that took the branch of a term lying within rounding
    error of the kink in lower precision passes its own choice here, so that
    the rest of the step can be compared exactly (either branch is within
    that rounding error of the true loss value)."""
    if loss == "ranking":
        z = margin - p.unsqueeze(1) + S
        if active is not None:
            return (z * active * valid).sum(1)
        return (torch.relu(z) * valid).sum(1)
    if loss == "logistic":
        k = valid.sum(1)
        neg = (_softplus(S) * valid).sum(1) / torch.clamp(k, min=1.0)
        return _softplus(-p) + neg
    if loss == "softmax":
        masked = S.masked_fill(valid == 0, -math.inf)
        return torch.logsumexp(torch.cat([p.unsqueeze(1), masked], 1), 1) - p
    raise ValueError(loss)


def valid_mask(C: int, U: int):
    """(C, C+U) mask of the negatives each edge is scored against: every column
    but the induced positive t = e in the in-chunk part."""
    v = torch.ones(C, C + U, dtype=_F64)
    idx = torch.arange(C)
    v[idx, idx] = 0.0
    return v


# --------------------------------------------------------------------------
# O3 chunking, O9 step gradient, O10 row-wise Adagrad
# --------------------------------------------------------------------------
def chunk_ranges(m: int, C: int):
    return [(c, c * C, min((c + 1) * C, m)) for c in range(-(-m // C))]


def chunk_ranges_by_relation(rel, C: int):
    """Relation-grouped chunks (Sec. 4.3: batches of edges that share their
    relation type): the edges must be sorted by relation; each maximal run of
    one relation is cut into chunks of C edges, the run's last chunk holding
    the rest.  Chunks are numbered in edge order."""
    rel = np.asarray(rel, dtype=np.int64)
    if rel.size and np.any(rel[1:] < rel[:-1]):
        raise ValueError("relation-grouped chunks need the edges sorted by relation")
    out = []
    lo = 0
    while lo < rel.size:
        hi = lo
        while hi < rel.size and rel[hi] == rel[lo]:
            hi += 1
        for a in range(lo, hi, C):
            out.append((len(out), a, min(a + C, hi)))
        lo = hi
    return out


def make_chunks(m: int, C: int, rel, chunking: str):
    """Chunks of a call: 'consecutive' (C edges each in the given order) or
    'by_relation' (chunk_ranges_by_relation)."""
    if chunking == "consecutive" or rel is None:
        return chunk_ranges(m, C)
    if chunking == "by_relation":
        return chunk_ranges_by_relation(rel, C)
    raise ValueError(chunking)


def step_negatives(model: Model, i: int, j: int, step, seed: int, U: int, first_chunk: int = 0, tables=None):
    """Uniform negatives (destination side, source side) of each chunk of a step
    of bucket (i, j), drawn over the rows of the source and destination tables
    (tables: their keys, by default partitions i and j)."""
    b = i * model.P + j
    ti, tj = (i, j) if tables is None else tables
    rows_i, rows_j = model.emb[ti].shape[0], model.emb[tj].shape[0]
    return [(uniform_negatives(seed, b, first_chunk + c, 0, U, rows_j),
             uniform_negatives(seed, b, first_chunk + c, 1, U, rows_i)) for (c, _, _) in step]


def train_bucket(model: Model, i: int, j: int, src, rel, dst, C: int, U: int, S: int,
                 lr: float, seed: int, first_chunk: int = 0, return_steps: bool = False,
                 branches=None, chunking: str = "consecutive"):
    """One pass over the edges of bucket (i, j) in the given order.

    Chunk c (counted from `first_chunk`) holds edges [cC, min((c+1)C, m)) of the
    given arrays; a step holds S consecutive chunks; the gradient of the step's
    summed loss is taken at the step-start parameters and then applied by
    row-wise Adagrad (entities) and element-wise Adagrad (relations).
    src/dst are local row ids in partitions i / j; rel may be None when R == 1.
    `branches` (ranking, one step only) gives per chunk of the step the pair
    (active dst side, active src side) of 0/1 arrays [C_c, C_c + U] that fix
    the hinge branches (see side_loss).  chunking: 'consecutive' or
    'by_relation' (make_chunks).
    Returns the summed loss (and the per-step losses)."""
    src = np.asarray(src, dtype=np.int64)
    dst = np.asarray(dst, dtype=np.int64)
    m = src.shape[0]
    chunks = make_chunks(m, C, rel, chunking)
    rel = np.zeros(m, dtype=np.int64) if rel is None else np.asarray(rel, dtype=np.int64)
    runs = type_runs(model, i, j, chunks, rel)
    if branches is not None and (len(runs) > 1 or len(chunks) > S):
        raise ValueError("hinge branches can be given for one step only")
    step_losses = []
    for run, tables in runs:
        for s0 in range(0, len(run), S):
            step = run[s0:s0 + S]
            negs = step_negatives(model, i, j, step, seed, U, first_chunk, tables)
            loss, grads, rel_grad = step_loss_and_grad(model, tables[0], tables[1], src, rel, dst, step, negs,
                                                       branches=branches)
            adagrad_update(model, grads, rel_grad, lr)
            step_losses.append(loss)
    total = float(sum(step_losses))
    return (total, step_losses) if return_steps else total


def type_runs(model: Model, i: int, j: int, chunks, rel):
    """The call's chunks as runs of consecutive chunks that share their
    tables, with those tables' keys: one run over partitions i and j without
    entity types; with types, a new run wherever the (source type,
    destination type) of the chunks' relation changes (the chunks must each
    hold one relation, as relation-grouped chunks do)."""
    if model.types is None:
        return [(list(chunks), (i, j))] if chunks else []
    runs = []
    for ch in chunks:
        r = np.unique(rel[ch[1]:ch[2]])
        if len(r) != 1:
            raise ValueError("with entity types every chunk must hold one relation (relation-grouped chunks)")
        tables = model.types.tables(int(r[0]), i, j)
        if tables is None:
            raise ValueError(f"relation {int(r[0])} has no edges in bucket ({i}, {j})")
        if runs and runs[-1][1] == tables:
            runs[-1][0].append(ch)
        else:
            runs.append(([ch], tables))
    return runs


def step_loss_and_grad(model, i, j, src, rel, dst, step, negs, with_grad=True, branches=None):
    """Summed loss of one step's chunks and its exact gradient (autograd, fp64)
    with respect to every entity row and relation parameter row it touches.

    Returns (loss, {partition: (row ids, grad rows)}, (relation ids, grad rows))."""
    # rows each table contributes to this step (partition i = source side,
    # partition j = destination side; one table when i == j)
    touched = {i: [], j: []}
    for (c, lo, hi), (u_dst, u_src) in zip(step, negs):
        touched[i] += [src[lo:hi], u_src]
        touched[j] += [dst[lo:hi], u_dst]
    leaf, ids_of = {}, {}
    for p, lists in touched.items():
        ids = np.unique(np.concatenate(lists))
        leaf[p] = torch.tensor(model.emb[p][ids], dtype=_F64, requires_grad=with_grad)
        ids_of[p] = ids
    step_rels = np.unique(np.concatenate([rel[lo:hi] for (_, lo, hi) in step]))
    if model.reciprocal:
        step_rels = np.unique(np.concatenate([step_rels, model.reverse_rel(step_rels)]))
    rel_leaf = None
    if model.rel is not None:
        rel_leaf = torch.tensor(model.rel[step_rels], dtype=_F64, requires_grad=with_grad)

    def rows(p, ids):
        return leaf[p][torch.from_numpy(np.searchsorted(ids_of[p], ids))]

    def theta_of(r):
        return None if rel_leaf is None else rel_leaf[int(np.searchsorted(step_rels, r))]

    step_loss = 0.0
    for k, ((c, lo, hi), (u_dst, u_src)) in enumerate(zip(step, negs)):
        Cc = hi - lo
        xs = rows(i, src[lo:hi])
        xd = rows(j, dst[lo:hi])
        cand_dst = torch.cat([xd, rows(j, u_dst)], 0)
        cand_src = torch.cat([xs, rows(i, u_src)], 0)
        r_e = rel[lo:hi]
        theta_e = theta_rev = None
        if rel_leaf is not None:
            theta_e = rel_leaf[torch.from_numpy(np.searchsorted(step_rels, r_e))]
            if model.reciprocal:
                theta_rev = rel_leaf[torch.from_numpy(np.searchsorted(step_rels, model.reverse_rel(r_e)))]
        if model.reciprocal:
            p, p1, S0, S1 = chunk_scores_reciprocal(model.op, model.cmp, xs, xd, theta_e, theta_rev,
                                                    cand_dst, cand_src)
        else:
            p, S0, S1 = chunk_scores(model.op, model.cmp, xs, xd, theta_e, r_e,
                                     cand_dst, cand_src, theta_of)
            p1 = p
        valid = valid_mask(Cc, len(u_dst))
        act0 = act1 = None
        if branches is not None:
            act0 = torch.as_tensor(np.asarray(branches[k][0], dtype=np.float64))
            act1 = torch.as_tensor(np.asarray(branches[k][1], dtype=np.float64))
        w_e = torch.as_tensor(model.edge_weights(r_e))
        loss = ((w_e * side_loss(model.loss, model.margin, p, S0, valid, act0)).sum()
                + (w_e * side_loss(model.loss, model.margin, p1, S1, valid, act1)).sum())
        if with_grad:
            loss.backward()          # gradients of the chunks add up in the leaves
        step_loss += float(loss.detach())

    grads = {}
    for p in leaf:
        g = leaf[p].grad if with_grad else None
        grads[p] = (ids_of[p], np.zeros((len(ids_of[p]), model.d)) if g is None else g.numpy())
    rel_grad = None
    if rel_leaf is not None:
        g = rel_leaf.grad if with_grad else None
        rel_grad = (step_rels, np.zeros(rel_leaf.shape) if g is None else g.numpy())
    return step_loss, grads, rel_grad


def adagrad_update(model: Model, grads, rel_grad, lr: float):
    """Row-wise Adagrad for entity rows (one accumulator per row, summed over
    the row's squared gradient) and element-wise Adagrad for relations."""
    for p, (ids, g) in grads.items():
        model.G[p][ids] += (g * g).sum(1)
        model.emb[p][ids] -= lr * g / (np.sqrt(model.G[p][ids])[:, None] + EPS_ADAGRAD)
    if rel_grad is not None:
        ids, g = rel_grad
        model.relG[ids] += g * g
        model.rel[ids] -= lr * g / (np.sqrt(model.relG[ids]) + EPS_ADAGRAD)


def inspect_step(model: Model, i: int, j: int, src, rel, dst, C: int, U: int, seed: int,
                 first_chunk: int = 0, chunking: str = "consecutive"):
    """The forward half of one step on these edges (all chunks of the call),
    at the current parameters: for each chunk a dict with
      p      (C_c,)           positive scores f(s_e, r_e, d_e)
      S0, S1 (C_c, C_c + U)   destination- and source-side candidate scores
      loss0, loss1 (C_c,)     each edge's loss per side (side_loss)
      dS0, dS1 (C_c, C_c + U) dL/dS of each side with p held fixed, 0 on the
                              excluded induced positive
      dp     (C_c,)           dL/dp_e (both sides, scores held fixed)
    all float64 numpy arrays.  With reciprocal predicates each side has its own
    positive: p and dp belong to the destination side, p1 and dp1 to the
    source side.  Losses and gradients are those of the unweighted loss (a
    relation weight multiplies all of them).  With entity types the chunks
    must share one (source type, destination type) pair."""
    src = np.asarray(src, dtype=np.int64)
    dst = np.asarray(dst, dtype=np.int64)
    m = src.shape[0]
    step = make_chunks(m, C, rel, chunking)
    rel = np.zeros(m, dtype=np.int64) if rel is None else np.asarray(rel, dtype=np.int64)
    runs = type_runs(model, i, j, step, rel)
    if len(runs) > 1:
        raise ValueError("the chunks span several (source type, destination type) pairs")
    ti, tj = runs[0][1] if runs else (i, j)
    negs = step_negatives(model, i, j, step, seed, U, first_chunk, (ti, tj))
    theta_all = None if model.rel is None else torch.tensor(model.rel, dtype=_F64)
    out = []
    with torch.no_grad():
        for (c, lo, hi), (u_dst, u_src) in zip(step, negs):
            xs = torch.tensor(model.emb[ti][src[lo:hi]], dtype=_F64)
            xd = torch.tensor(model.emb[tj][dst[lo:hi]], dtype=_F64)
            cand_dst = torch.cat([xd, torch.tensor(model.emb[tj][u_dst], dtype=_F64)], 0)
            cand_src = torch.cat([xs, torch.tensor(model.emb[ti][u_src], dtype=_F64)], 0)
            r_e = rel[lo:hi]
            theta_e = None if theta_all is None else theta_all[torch.from_numpy(r_e)]
            if model.reciprocal:
                theta_rev = None if theta_all is None else theta_all[torch.from_numpy(model.reverse_rel(r_e))]
                p, p1, S0, S1 = chunk_scores_reciprocal(model.op, model.cmp, xs, xd, theta_e, theta_rev,
                                                        cand_dst, cand_src)
            else:
                p, S0, S1 = chunk_scores(model.op, model.cmp, xs, xd, theta_e, r_e, cand_dst, cand_src,
                                         lambda r: None if theta_all is None else theta_all[r])
            valid = valid_mask(hi - lo, U)
            rec = {"p": p.numpy()}
            pg = p.clone().requires_grad_(True)
            pg1 = p1.clone().requires_grad_(True) if model.reciprocal else pg
            for side, S, pp in ((0, S0, pg), (1, S1, pg1)):
                Sg = S.clone().requires_grad_(True)
                with torch.enable_grad():
                    L = side_loss(model.loss, model.margin, pp, Sg, valid)
                    L.sum().backward()
                rec[f"S{side}"] = S.numpy()
                rec[f"loss{side}"] = L.detach().numpy()
                rec[f"dS{side}"] = Sg.grad.numpy()
            rec["dp"] = pg.grad.numpy()
            if model.reciprocal:
                rec["p1"] = p1.numpy()
                rec["dp1"] = pg1.grad.numpy()
            out.append(rec)
    return out


def train_epoch(model: Model, offsets, src_local, rel, dst_local, C, U, S, lr, seed, chunking="consecutive"):
    """One epoch: every bucket with edges, in inside-out order (Sec. 4.1)."""
    P = model.P
    total = 0.0
    for (i, j) in inside_out_order(P):
        b = i * P + j
        lo, hi = int(offsets[b]), int(offsets[b + 1])
        if hi == lo:
            continue
        r = None if rel is None else rel[lo:hi]
        total += train_bucket(model, i, j, src_local[lo:hi], r, dst_local[lo:hi],
                              C, U, S, lr, seed, chunking=chunking)
    return total


# --------------------------------------------------------------------------
# O11 scoring and filtered ranking (Sec. 5)
# --------------------------------------------------------------------------
def score_edges(model: Model, i: int, j: int, src, rel, dst):
    """f(s, r, d) for each edge (local ids in partitions i and j)."""
    src = np.asarray(src, dtype=np.int64)
    dst = np.asarray(dst, dtype=np.int64)
    rel = np.zeros(len(src), dtype=np.int64) if rel is None else np.asarray(rel, np.int64)
    xs = torch.tensor(model.emb[i][src], dtype=_F64)
    xd = torch.tensor(model.emb[j][dst], dtype=_F64)
    theta = None if model.rel is None else torch.tensor(model.rel[rel], dtype=_F64)
    with torch.no_grad():
        return compare_rows(model.cmp, apply_operator(model.op, xs, theta), xd).numpy()


def rank_eval(model: Model, src, rel, dst, known_src, known_rel, known_dst, tol: float = 0.0):
    """Filtered ranks of each triple among all entities (single partition).

    Destination side: 1 + #{d' != d : (s, r, d') not known, f(s, r, d') >= f(s, r, d)};
    source side symmetric (with reciprocal predicates its scores, the true
    source's included, are sim(g(x_d, theta_{r+R}), x_s')).  Returns (ranks[2n] -- destination side first, then
    source side --, MRR, Hits@10).  With tol > 0 it also returns the ranks that
    count only candidates with f >= f_pos + tol and those counting f >= f_pos - tol:
    bounds for a computation whose scores carry an error up to tol."""
    assert model.P == 1
    E = model.emb[0]
    n = E.shape[0]
    src = np.asarray(src, np.int64)
    dst = np.asarray(dst, np.int64)
    rel = np.zeros(len(src), np.int64) if rel is None else np.asarray(rel, np.int64)
    k_rel = (np.zeros(len(known_src), np.int64) if known_rel is None
             else np.asarray(known_rel, np.int64))
    dsts_of, srcs_of = {}, {}
    for ks, kr, kd in zip(np.asarray(known_src, np.int64).tolist(), k_rel.tolist(),
                          np.asarray(known_dst, np.int64).tolist()):
        dsts_of.setdefault((ks, kr), set()).add(kd)
        srcs_of.setdefault((kr, kd), set()).add(ks)
    allx = torch.tensor(E, dtype=_F64)
    ranks = np.zeros(2 * len(src), np.int64)
    lo_r = np.zeros_like(ranks)
    hi_r = np.zeros_like(ranks)
    with torch.no_grad():
        for e in range(len(src)):
            s, r, d = int(src[e]), int(rel[e]), int(dst[e])
            theta = None if model.rel is None else torch.tensor(model.rel[r], dtype=_F64)
            # destination corruptions f(s, r, d') for every d'
            q = apply_operator(model.op, allx[s:s + 1], theta)
            sc_d = compare_all(model.cmp, q, allx)[0].numpy()
            if model.reciprocal:
                # source corruptions scored by the reciprocal relation:
                # sim(g(x_d, theta_{r+R}), x_s') for every s'
                th_rev = None if model.rel is None else torch.tensor(model.rel[r + model.R], dtype=_F64)
                k = apply_operator(model.op, allx[d:d + 1], th_rev)
                sc_s = compare_all(model.cmp, k, allx)[0].numpy()
            else:
                # source corruptions f(s', r, d) for every s'
                g_all = apply_operator(model.op, allx, theta)
                sc_s = compare_all(model.cmp, allx[d:d + 1], g_all)[0].numpy()
            for side, sc, true_id in ((0, sc_d, d), (1, sc_s, s)):
                keep = np.ones(n, bool)
                keep[true_id] = False
                filt = dsts_of.get((s, r), ()) if side == 0 else srcs_of.get((r, d), ())
                keep[list(filt)] = False
                pos_score = sc[true_id]
                slot = e if side == 0 else len(src) + e
                ranks[slot] = 1 + int(np.count_nonzero(keep & (sc >= pos_score)))
                lo_r[slot] = 1 + int(np.count_nonzero(keep & (sc >= pos_score + tol)))
                hi_r[slot] = 1 + int(np.count_nonzero(keep & (sc >= pos_score - tol)))
    mrr = float(np.mean(1.0 / ranks)) if len(ranks) else 0.0
    hits10 = float(np.mean(ranks <= 10)) if len(ranks) else 0.0
    if tol > 0:
        return ranks, mrr, hits10, lo_r, hi_r
    return ranks, mrr, hits10


def rank_sampled(model: Model, src, rel, dst, cand, tol: float = 0.0):
    """Raw ranks of each triple among a given candidate list (Sec. 5, Freebase
    evaluation, where each eval edge meets candidate nodes sampled by their
    prevalence; the caller draws them).

    Destination side: 1 + #{j : cand[j] != d, f(s, r, cand[j]) >= f(s, r, d)};
    source side: 1 + #{j : cand[j] != s, f(cand[j], r, d) >= f(s, r, d)} (with
    reciprocal predicates sim(g(x_d, theta_{r+R}), .) on both sides of the
    comparison).  No filter; a candidate listed k times counts k times.  Same return values as
    rank_eval (with tol > 0, also the rank bounds for scores within tol)."""
    assert model.P == 1
    E = model.emb[0]
    src = np.asarray(src, np.int64)
    dst = np.asarray(dst, np.int64)
    cand = np.asarray(cand, np.int64)
    rel = np.zeros(len(src), np.int64) if rel is None else np.asarray(rel, np.int64)
    allx = torch.tensor(E, dtype=_F64)
    cx = allx[torch.tensor(cand)]
    ranks = np.zeros(2 * len(src), np.int64)
    lo_r = np.zeros_like(ranks)
    hi_r = np.zeros_like(ranks)
    with torch.no_grad():
        for e in range(len(src)):
            s, r, d = int(src[e]), int(rel[e]), int(dst[e])
            theta = None if model.rel is None else torch.tensor(model.rel[r], dtype=_F64)
            q = apply_operator(model.op, allx[s:s + 1], theta)
            pos_dst = float(compare_rows(model.cmp, q, allx[d:d + 1])[0])
            sc_d = compare_all(model.cmp, q, cx)[0].numpy()                  # f(s, r, c)
            if model.reciprocal:
                th_rev = None if model.rel is None else torch.tensor(model.rel[r + model.R], dtype=_F64)
                k = apply_operator(model.op, allx[d:d + 1], th_rev)
                pos_src = float(compare_rows(model.cmp, k, allx[s:s + 1])[0])
                sc_s = compare_all(model.cmp, k, cx)[0].numpy()
            else:
                pos_src = pos_dst
                sc_s = compare_all(model.cmp, allx[d:d + 1], apply_operator(model.op, cx, theta))[0].numpy()  # f(c, r, d)
            for side, sc, true_id, pos_score in ((0, sc_d, d, pos_dst), (1, sc_s, s, pos_src)):
                keep = cand != true_id
                slot = e if side == 0 else len(src) + e
                ranks[slot] = 1 + int(np.count_nonzero(keep & (sc >= pos_score)))
                lo_r[slot] = 1 + int(np.count_nonzero(keep & (sc >= pos_score + tol)))
                hi_r[slot] = 1 + int(np.count_nonzero(keep & (sc >= pos_score - tol)))
    mrr = float(np.mean(1.0 / ranks)) if len(ranks) else 0.0
    hits10 = float(np.mean(ranks <= 10)) if len(ranks) else 0.0
    if tol > 0:
        return ranks, mrr, hits10, lo_r, hi_r
    return ranks, mrr, hits10
