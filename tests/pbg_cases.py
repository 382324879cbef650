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


def make_problem(op, cmp, loss, n=60, P=1, R=1, d=16, m=300, C=20, U=12, S=4, i=0, j=0,
                 seed=1, sigma=0.3, rel_scale=0.3, lr=0.1, margin=0.1, zipf=1.1):
    """A small seeded problem with Zipf endpoints (duplicates in chunks) and
    perturbed relation parameters."""
    rng = synth.rng_for(seed)
    rows = [O.partition_rows(n, P, p) for p in range(P)]
    parts = synth.partition_embeddings(rows, d, rng, sigma)
    src = synth.BoundedZipf(rows[i], zipf, rng).sample(rng, m)
    dst = synth.BoundedZipf(rows[j], zipf, rng).sample(rng, m)
    rel_ids = None if R == 1 else rng.integers(0, R, m).astype(np.int32)
    relp = synth.perturbed_relation_params(op, R, d, rng, rel_scale)
    return Problem(n, P, R, d, op, cmp, loss, margin, parts, relp, i, j, src, rel_ids, dst,
                   C, U, S, lr, seed + 1000)


def oracle_model(pb: Problem) -> O.Model:
    return O.Model.create(pb.n, pb.P, pb.R, pb.d, pb.op, pb.cmp, pb.loss, pb.margin,
                          [p.astype(np.float64) for p in pb.parts],
                          None if pb.rel is None else pb.rel.astype(np.float64))


class GpuModel:
    """Device tensors of a problem bound to a library context."""

    def __init__(self, pb: Problem, flags: int = 0):
        from paper_1903_12287_amd import pbg
        self.pbg = pbg
        self.pb = pb
        dev = torch.device("cuda")
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
                                         pb.C, pb.U, pb.S, pb.lr, pb.seed, first_chunk)

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
