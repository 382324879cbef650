"""Python binding of the C ABI in include/pbg.h (argument marshalling only).

Every function here has the name of the C entry point it calls and does no
computation of its own: it checks that tensors have the dtype, device and
layout the C side expects, turns them into raw pointers, calls the library
and raises PbgError when the call returns an error status.  Device memory
and streams come from PyTorch; all work runs in the HIP kernels of
lib/libpbg.so.  There is no fallback: without the built library every call
raises.
"""

from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "lib", "libpbg.so")

OPERATORS = {"identity": 0, "translation": 1, "diagonal": 2, "linear": 3, "complex_diagonal": 4}
COMPARATORS = {"dot": 0, "cos": 1}
LOSSES = {"ranking": 0, "logistic": 1, "softmax": 2}
F_BF16_SCORE = 1
F_PHASE_TIMING = 2
F_SCORE_TIMING = 4
F_RECIPROCAL = 8
CHUNKINGS = {"consecutive": 0, "by_relation": 1}
MEM_DEVICE = 0
MEM_PINNED_HOST = 1
NOALLOC_MAX_REL_FLOATS = 2 * 1024 * 1024   # PBG_NOALLOC_MAX_REL_FLOATS

STATUS = {0: "OK", 1: "INVALID_ARG", 2: "UNSUPPORTED", 3: "OUT_OF_MEMORY", 4: "DEVICE", 5: "STATE"}

# every entry point the header declares
EXPORTS = (
    "pbg_bucket_init", "pbg_free", "pbg_last_error", "pbg_partition_rows",
    "pbg_relation_param_floats", "pbg_bucket_edges", "pbg_bind_partition",
    "pbg_bind_relations", "pbg_set_streams", "pbg_train_bucket", "pbg_get_step_losses",
    "pbg_train_epoch", "pbg_score_edges", "pbg_rank_eval", "pbg_rank_sampled", "pbg_get_stats",
    "pbg_sample_negatives", "pbg_inspect_step", "pbg_score_edges_noalloc", "pbg_group_by_relation",
    "pbg_set_entity_types", "pbg_bind_type_partition", "pbg_type_partition_rows", "pbg_set_relation_weights",
)


class PbgError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS.get(status, status)}: {message}")
        self.status = status
        self.status_name = STATUS.get(status, str(status))


class NegConfig(ctypes.Structure):
    _fields_ = [("chunk_size", ctypes.c_int32), ("num_uniform", ctypes.c_int32),
                ("chunks_per_step", ctypes.c_int32), ("chunking", ctypes.c_int32),
                ("first_chunk", ctypes.c_int64)]


class Stats(ctypes.Structure):
    _fields_ = [("edges", ctypes.c_int64), ("chunks", ctypes.c_int64), ("steps", ctypes.c_int64),
                ("total_ms", ctypes.c_double), ("gather_ms", ctypes.c_double),
                ("score_ms", ctypes.c_double), ("epilogue_ms", ctypes.c_double),
                ("backward_ms", ctypes.c_double), ("opbwd_ms", ctypes.c_double),
                ("update_ms", ctypes.c_double), ("gather_bytes", ctypes.c_double),
                ("score_flops", ctypes.c_double), ("update_bytes", ctypes.c_double),
                ("copy_ms", ctypes.c_double), ("partition_loads", ctypes.c_int64),
                ("score_timed_steps", ctypes.c_int64)]

    def as_dict(self):
        return {name: getattr(self, name) for name, _ in self._fields_}


_lib = None


def library() -> ctypes.CDLL:
    """Loads lib/libpbg.so once; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                           "(python paper_1903_12287_amd/build.py)")
    L = ctypes.CDLL(LIB_PATH)
    vp, i32, i64, u32, u64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32, ctypes.c_uint64
    f32, dp = ctypes.c_float, ctypes.POINTER(ctypes.c_double)
    sig = {
        "pbg_bucket_init": ([ctypes.POINTER(vp), i64, i32, i32, i32, i32, i32, i32, f32, u32], i32),
        "pbg_free": ([vp], None),
        "pbg_last_error": ([vp], ctypes.c_char_p),
        "pbg_partition_rows": ([vp, i32], i64),
        "pbg_relation_param_floats": ([vp], i64),
        "pbg_bucket_edges": ([vp, vp, vp, vp, i64, vp, vp, vp, vp], i32),
        "pbg_bind_partition": ([vp, i32, vp, vp, i32], i32),
        "pbg_bind_relations": ([vp, vp, vp], i32),
        "pbg_set_streams": ([vp, vp, vp], i32),
        "pbg_train_bucket": ([vp, i32, i32, vp, vp, vp, i64, ctypes.POINTER(NegConfig), f32, u64, dp], i32),
        "pbg_get_step_losses": ([vp, dp, i64, ctypes.POINTER(ctypes.c_int64)], i32),
        "pbg_train_epoch": ([vp, vp, vp, vp, vp, ctypes.POINTER(NegConfig), f32, u64, i32, dp], i32),
        "pbg_score_edges": ([vp, i32, i32, vp, vp, vp, i64, vp], i32),
        "pbg_score_edges_noalloc": ([vp, i32, i32, vp, vp, vp, i64, vp], i32),
        "pbg_group_by_relation": ([vp, vp, vp, vp, i64, vp, vp, vp], i32),
        "pbg_rank_eval": ([vp, vp, vp, vp, i64, vp, vp, vp, i64, vp, dp, dp], i32),
        "pbg_rank_sampled": ([vp, vp, vp, vp, i64, vp, i64, vp, dp, dp], i32),
        "pbg_get_stats": ([vp, ctypes.POINTER(Stats)], i32),
        "pbg_sample_negatives": ([vp, i32, i32, i64, i64, i32, u64, vp], i32),
        "pbg_inspect_step": ([vp, i32, i32, vp, vp, vp, i64, ctypes.POINTER(NegConfig), u64, vp, vp, vp, vp,
                              dp], i32),
        "pbg_set_entity_types": ([vp, i32, vp, vp, vp, vp], i32),
        "pbg_bind_type_partition": ([vp, i32, i32, vp, vp, i32], i32),
        "pbg_type_partition_rows": ([vp, i32, i32], i64),
        "pbg_set_relation_weights": ([vp, vp], i32),
    }
    for name, (args, res) in sig.items():
        fn = getattr(L, name)
        fn.argtypes = args
        fn.restype = res
    _lib = L
    return L


def _check(ctx, status):
    if status != 0:
        msg = library().pbg_last_error(ctx)
        raise PbgError(status, msg.decode() if msg else "")


def _ptr(t, dtype, what, device=True, allow_none=False):
    if t is None:
        if allow_none:
            return None
        raise ValueError(f"{what} is required")
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{what} must be a torch.Tensor")
    if t.dtype != dtype:
        raise TypeError(f"{what} must be {dtype}, got {t.dtype}")
    if device and t.device.type != "cuda":
        raise ValueError(f"{what} must be a device tensor")
    if not t.is_contiguous():
        raise ValueError(f"{what} must be contiguous")
    return ctypes.c_void_p(t.data_ptr()) if t.numel() else None


def _stream_handle(s):
    if s is None:
        return None
    if isinstance(s, torch.cuda.Stream):
        return ctypes.c_void_p(s.cuda_stream)
    return ctypes.c_void_p(int(s))


def _enum(table, v, what):
    if isinstance(v, str):
        if v not in table:
            raise ValueError(f"unknown {what} {v!r}")
        return table[v]
    return int(v)


# ------------------------------------------------------------------ entry points
def pbg_bucket_init(num_entities, num_partitions, num_relations, dim, op, cmp, loss,
                    margin=0.1, flags=0):
    L = library()
    ctx = ctypes.c_void_p()
    st = L.pbg_bucket_init(ctypes.byref(ctx), int(num_entities), int(num_partitions),
                           int(num_relations), int(dim), _enum(OPERATORS, op, "operator"),
                           _enum(COMPARATORS, cmp, "comparator"), _enum(LOSSES, loss, "loss"),
                           float(margin), int(flags))
    if st != 0:
        msg = L.pbg_last_error(ctx).decode() if ctx.value else "pbg_bucket_init failed"
        if ctx.value:
            L.pbg_free(ctx)
        raise PbgError(st, msg)
    ctx._flags = int(flags)   # the layouts some outputs take depend on them
    ctx._R = int(num_relations)
    return ctx


def pbg_free(ctx):
    if ctx is not None and ctx.value:
        library().pbg_free(ctx)
        ctx.value = None
        ctx._bound = None


def pbg_last_error(ctx) -> str:
    return library().pbg_last_error(ctx).decode()


def pbg_partition_rows(ctx, p) -> int:
    return int(library().pbg_partition_rows(ctx, int(p)))


def pbg_relation_param_floats(ctx) -> int:
    return int(library().pbg_relation_param_floats(ctx))


def _keep(ctx, key, *tensors):
    """The library keeps raw pointers to bound buffers: hold the tensors for as
    long as the context lives, so that they cannot be freed under it."""
    bound = getattr(ctx, "_bound", None)
    if bound is None:
        bound = {}
        ctx._bound = bound
    bound[key] = tensors


def pbg_bind_partition(ctx, p, emb, adagrad, where=MEM_DEVICE):
    on_dev = where == MEM_DEVICE
    if not on_dev and not (emb.is_pinned() and adagrad.is_pinned()):
        raise ValueError("host partitions must be in page-locked (pinned) memory")
    _check(ctx, library().pbg_bind_partition(ctx, int(p), _ptr(emb, torch.float32, "emb", on_dev),
                                             _ptr(adagrad, torch.float32, "adagrad", on_dev), int(where)))
    _keep(ctx, ("partition", int(p)), emb, adagrad)


def pbg_set_entity_types(ctx, type_entities, type_partitioned, rel_src_type, rel_dst_type):
    """Host sequences: entities per type, partitioned flags per type, and the
    source and destination type of every relation."""
    import numpy as np
    n = np.ascontiguousarray(type_entities, dtype=np.int64)
    part = np.ascontiguousarray(type_partitioned, dtype=np.int32)
    rs = np.ascontiguousarray(rel_src_type, dtype=np.int32)
    rd = np.ascontiguousarray(rel_dst_type, dtype=np.int32)
    if part.size != n.size or rs.size != getattr(ctx, "_R", rs.size) or rd.size != rs.size:
        raise ValueError("one partitioned flag per type and one source and destination type per relation")
    _check(ctx, library().pbg_set_entity_types(ctx, int(n.size), n.ctypes.data, part.ctypes.data, rs.ctypes.data,
                                               rd.ctypes.data))
    bound = getattr(ctx, "_bound", None)
    if bound is not None:   # the tables are unbound
        for k in [k for k in bound if isinstance(k, tuple) and k[0] in ("partition", "table")]:
            del bound[k]


def pbg_bind_type_partition(ctx, t, p, emb, adagrad, where=MEM_DEVICE):
    on_dev = where == MEM_DEVICE
    if not on_dev and not (emb.is_pinned() and adagrad.is_pinned()):
        raise ValueError("host partitions must be in page-locked (pinned) memory")
    _check(ctx, library().pbg_bind_type_partition(ctx, int(t), int(p), _ptr(emb, torch.float32, "emb", on_dev),
                                                  _ptr(adagrad, torch.float32, "adagrad", on_dev), int(where)))
    _keep(ctx, ("table", int(t), int(p)), emb, adagrad)


def pbg_type_partition_rows(ctx, t, p) -> int:
    return int(library().pbg_type_partition_rows(ctx, int(t), int(p)))


def pbg_set_relation_weights(ctx, weights):
    """weights: host sequence of R floats, or None for weight 1 everywhere."""
    import numpy as np
    if weights is None:
        _check(ctx, library().pbg_set_relation_weights(ctx, None))
        return
    w = np.ascontiguousarray(weights, dtype=np.float32)
    if w.size != getattr(ctx, "_R", w.size):
        raise ValueError("one weight per relation")
    _check(ctx, library().pbg_set_relation_weights(ctx, w.ctypes.data))


def pbg_bind_relations(ctx, params, adagrad):
    _check(ctx, library().pbg_bind_relations(ctx, _ptr(params, torch.float32, "params", allow_none=True),
                                             _ptr(adagrad, torch.float32, "adagrad", allow_none=True)))
    _keep(ctx, "relations", params, adagrad)


def pbg_set_streams(ctx, compute_stream=None, copy_stream=None):
    _check(ctx, library().pbg_set_streams(ctx, _stream_handle(compute_stream), _stream_handle(copy_stream)))


def pbg_bucket_edges(ctx, src, rel, dst, offsets, src_local, rel_out, dst_local):
    n = src.numel()
    _check(ctx, library().pbg_bucket_edges(
        ctx, _ptr(src, torch.int64, "src"), _ptr(rel, torch.int32, "rel", allow_none=True),
        _ptr(dst, torch.int64, "dst"), n, _ptr(offsets, torch.int64, "offsets"),
        _ptr(src_local, torch.int32, "src_local", allow_none=n == 0),
        _ptr(rel_out, torch.int32, "rel_out", allow_none=True),
        _ptr(dst_local, torch.int32, "dst_local", allow_none=n == 0)))


def _neg(chunk_size, num_uniform, chunks_per_step, first_chunk, chunking="consecutive"):
    return NegConfig(int(chunk_size), int(num_uniform), int(chunks_per_step), _enum(CHUNKINGS, chunking, "chunking"),
                     int(first_chunk))


def pbg_train_bucket(ctx, i, j, src_local, rel, dst_local, chunk_size, num_uniform,
                     chunks_per_step, lr, seed, first_chunk=0, chunking="consecutive") -> float:
    n = src_local.numel()
    if dst_local.numel() != n or (rel is not None and rel.numel() != n):
        raise ValueError("edge arrays differ in length")
    neg = _neg(chunk_size, num_uniform, chunks_per_step, first_chunk, chunking)
    loss = ctypes.c_double(0.0)
    _check(ctx, library().pbg_train_bucket(
        ctx, int(i), int(j), _ptr(src_local, torch.int32, "src_local", allow_none=n == 0),
        _ptr(rel, torch.int32, "rel", allow_none=True),
        _ptr(dst_local, torch.int32, "dst_local", allow_none=n == 0), n, ctypes.byref(neg),
        float(lr), int(seed) & 0xFFFFFFFFFFFFFFFF, ctypes.byref(loss)))
    return loss.value


def pbg_get_step_losses(ctx):
    n = ctypes.c_int64(0)
    _check(ctx, library().pbg_get_step_losses(ctx, None, 0, ctypes.byref(n)))
    buf = (ctypes.c_double * max(n.value, 1))()
    _check(ctx, library().pbg_get_step_losses(ctx, buf, n.value, ctypes.byref(n)))
    return [buf[k] for k in range(n.value)]


def pbg_train_epoch(ctx, offsets, src_local, rel, dst_local, chunk_size, num_uniform,
                    chunks_per_step, lr, seed, max_resident, chunking="consecutive") -> float:
    for t, name in ((src_local, "src_local"), (dst_local, "dst_local")):
        if t.numel() and not t.is_pinned():
            raise ValueError(f"{name} must be in page-locked host memory")
    if offsets.device.type != "cpu":
        raise ValueError("offsets must be a host tensor")
    neg = _neg(chunk_size, num_uniform, chunks_per_step, 0, chunking)
    loss = ctypes.c_double(0.0)
    _check(ctx, library().pbg_train_epoch(
        ctx, _ptr(offsets, torch.int64, "offsets", device=False),
        _ptr(src_local, torch.int32, "src_local", device=False, allow_none=True),
        _ptr(rel, torch.int32, "rel", device=False, allow_none=True),
        _ptr(dst_local, torch.int32, "dst_local", device=False, allow_none=True),
        ctypes.byref(neg), float(lr), int(seed) & 0xFFFFFFFFFFFFFFFF, int(max_resident),
        ctypes.byref(loss)))
    return loss.value


def pbg_score_edges(ctx, i, j, src_local, rel, dst_local, scores):
    n = src_local.numel()
    _check(ctx, library().pbg_score_edges(
        ctx, int(i), int(j), _ptr(src_local, torch.int32, "src_local", allow_none=n == 0),
        _ptr(rel, torch.int32, "rel", allow_none=True),
        _ptr(dst_local, torch.int32, "dst_local", allow_none=n == 0), n,
        _ptr(scores, torch.float32, "scores", allow_none=n == 0)))


def pbg_group_by_relation(ctx, src, rel, dst, src_out, rel_out, dst_out):
    n = src.numel()
    if rel.numel() != n or dst.numel() != n:
        raise ValueError("edge arrays differ in length")
    _check(ctx, library().pbg_group_by_relation(
        ctx, _ptr(src, torch.int32, "src", allow_none=n == 0), _ptr(rel, torch.int32, "rel", allow_none=n == 0),
        _ptr(dst, torch.int32, "dst", allow_none=n == 0), n,
        _ptr(src_out, torch.int32, "src_out", allow_none=n == 0), _ptr(rel_out, torch.int32, "rel_out", allow_none=n == 0),
        _ptr(dst_out, torch.int32, "dst_out", allow_none=n == 0)))


def pbg_score_edges_noalloc(ctx, i, j, src_local, rel, dst_local, scores):
    n = src_local.numel()
    _check(ctx, library().pbg_score_edges_noalloc(
        ctx, int(i), int(j), _ptr(src_local, torch.int32, "src_local", allow_none=n == 0),
        _ptr(rel, torch.int32, "rel", allow_none=True),
        _ptr(dst_local, torch.int32, "dst_local", allow_none=n == 0), n,
        _ptr(scores, torch.float32, "scores", allow_none=n == 0)))


def pbg_rank_eval(ctx, src, rel, dst, known_src, known_rel, known_dst, ranks):
    n, nk = src.numel(), known_src.numel()
    mrr, hits = ctypes.c_double(0.0), ctypes.c_double(0.0)
    _check(ctx, library().pbg_rank_eval(
        ctx, _ptr(src, torch.int32, "src", allow_none=n == 0), _ptr(rel, torch.int32, "rel", allow_none=True),
        _ptr(dst, torch.int32, "dst", allow_none=n == 0), n,
        _ptr(known_src, torch.int32, "known_src", allow_none=nk == 0),
        _ptr(known_rel, torch.int32, "known_rel", allow_none=True),
        _ptr(known_dst, torch.int32, "known_dst", allow_none=nk == 0), nk,
        _ptr(ranks, torch.int32, "ranks", allow_none=n == 0), ctypes.byref(mrr), ctypes.byref(hits)))
    return mrr.value, hits.value


def pbg_rank_sampled(ctx, src, rel, dst, cand, ranks):
    n, nc = src.numel(), cand.numel()
    mrr, hits = ctypes.c_double(0.0), ctypes.c_double(0.0)
    _check(ctx, library().pbg_rank_sampled(
        ctx, _ptr(src, torch.int32, "src", allow_none=n == 0), _ptr(rel, torch.int32, "rel", allow_none=True),
        _ptr(dst, torch.int32, "dst", allow_none=n == 0), n, _ptr(cand, torch.int32, "cand", allow_none=nc == 0),
        nc, _ptr(ranks, torch.int32, "ranks", allow_none=n == 0), ctypes.byref(mrr), ctypes.byref(hits)))
    return mrr.value, hits.value


def pbg_get_stats(ctx) -> dict:
    s = Stats()
    _check(ctx, library().pbg_get_stats(ctx, ctypes.byref(s)))
    return s.as_dict()


def pbg_sample_negatives(ctx, i, j, first_chunk, n_chunks, num_uniform, seed, out):
    _check(ctx, library().pbg_sample_negatives(
        ctx, int(i), int(j), int(first_chunk), int(n_chunks), int(num_uniform),
        int(seed) & 0xFFFFFFFFFFFFFFFF, _ptr(out, torch.int32, "out", allow_none=True)))


def pbg_inspect_step(ctx, i, j, src_local, rel, dst_local, chunk_size, num_uniform, chunks_per_step, seed,
                     first_chunk=0, scores=None, dscores=None, row_loss=None, pos=None, chunking="consecutive",
                     n_chunks=None) -> float:
    """n_chunks: chunks of the call (consecutive chunking: ceil(n / chunk_size)).
    pos holds nch * chunk_size floats, twice that with F_RECIPROCAL."""
    n = src_local.numel()
    if dst_local.numel() != n or (rel is not None and rel.numel() != n):
        raise ValueError("edge arrays differ in length")
    nch = -(-n // int(chunk_size)) if n_chunks is None else int(n_chunks)
    N = int(chunk_size) + int(num_uniform)
    psides = 2 if getattr(ctx, "_flags", 0) & F_RECIPROCAL else 1   # positive scores per edge
    for t, want, name in ((scores, nch * 2 * chunk_size * N, "scores"), (dscores, nch * 2 * chunk_size * N, "dscores"),
                          (row_loss, nch * 2 * chunk_size, "row_loss"), (pos, nch * psides * chunk_size, "pos")):
        if t is not None and t.numel() != want:
            raise ValueError(f"{name} must hold {want} floats")
    neg = _neg(chunk_size, num_uniform, chunks_per_step, first_chunk, chunking)
    loss = ctypes.c_double(0.0)
    _check(ctx, library().pbg_inspect_step(
        ctx, int(i), int(j), _ptr(src_local, torch.int32, "src_local", allow_none=n == 0),
        _ptr(rel, torch.int32, "rel", allow_none=True),
        _ptr(dst_local, torch.int32, "dst_local", allow_none=n == 0), n, ctypes.byref(neg),
        int(seed) & 0xFFFFFFFFFFFFFFFF, _ptr(scores, torch.float32, "scores", allow_none=True),
        _ptr(dscores, torch.float32, "dscores", allow_none=True),
        _ptr(row_loss, torch.float32, "row_loss", allow_none=True),
        _ptr(pos, torch.float32, "pos", allow_none=True), ctypes.byref(loss)))
    return loss.value
