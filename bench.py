"""Benchmark of the bucket training step on one MI355X.

Workload: the social-network-shaped graph (LiveJournal node and edge counts:
4,847,571 nodes, 68,993,773 directed edges, Zipf(1.05) out- and in-degree, one
relation, one partition), dim 128, translation operator, cos comparator,
ranking loss (margin 0.1), chunks of 1000 edges with 1000 uniform + in-chunk
negatives per side, 40 chunks per step, row-wise Adagrad lr 0.1.  Inputs are
seeded synthetic data drawn on the device and resident in HBM before timing.

A bench step is one training step: 40 chunks (40,000 edges) through gather,
score contraction, loss epilogue, backward contractions, operator backward,
sort and Adagrad.  W warm-up steps run first, then K timed steps bracketed by
device synchronisation; the steps walk consecutive chunks of the bucket
(wrapping around after the last one).

Prints one JSON line with the metric, the roofline figure of the dominant
kernel (the score contraction with its fused loss epilogue, timed with HIP
events on the compute stream) and the CPU oracle timed on a bounded sample.
The line also carries the bf16-input leg of the same workload and, under
"big_bucket", one whole bucket (3, 7) of the partitioned
large-knowledge-graph-shaped run (9,375,000 edges, two resident partitions of
7,576,046 rows, d = 100, diagonal, dot, ranking): the one-GPU share of a
bucket-parallel run.
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

N_NODES, N_EDGES, DIM = 4_847_571, 68_993_773, 128
C, U, S = 1000, 1000, 40
LR, MARGIN, SEED = 0.1, 0.1, 20190002
PEAK_FP32_MFMA = 157.3   # TFLOP/s, MI355X dense fp32 matrix
PEAK_BF16_MFMA = 2516.6  # TFLOP/s, MI355X dense bf16 matrix
PEAK_HBM = 8000.0        # GB/s
SPLIT_PIECES = 6         # bf16 piece products per float32 product in the score contraction


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=400)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--cpu-sample-chunks", type=int, default=400,
                    help="chunks of the same bucket the CPU oracle is timed on")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-bf16", action="store_true", help="skip the bf16-input leg")
    ap.add_argument("--no-big-bucket", action="store_true",
                    help="skip the second workload of the default line (one bucket of the partitioned graph)")
    ap.add_argument("--row", choices=["bucketing", "knowledge_graph", "knowledge_graph_reciprocal", "big_bucket",
                                      "epoch", "tiny", "negatives", "library_gemm"],
                    help="measure another row of the hot path instead of the default training step: "
                         "edge bucketing of the follower graph, the knowledge-graph pass and filtered "
                         "rank evaluation, one bucket of the large partitioned graph, the follower-graph "
                         "epoch with partition swapping, or the tiny social graph; library_gemm times the "
                         "vendor GEMMs at the score shape and large square shapes for context")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a plain 1 GiB device-to-device copy five times (reference kernel of known "
                         "size for scaling hardware byte counters) and exit")
    return ap.parse_args()


def calibrate_copy():
    """A plain copy of known size: 2^28 float32 read and written per launch."""
    import torch
    torch.cuda.set_device(0)
    src = torch.ones(1 << 28, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": src.numel() * 4, "copy_bytes_written": dst.numel() * 4,
                      "launches": 5}))


def train_range(pbg, ctx, src, dst, step0, nsteps, total_steps):
    """Trains steps [step0, step0 + nsteps) of the bucket, wrapping around."""
    loss = 0.0
    s = step0 % total_steps
    left = nsteps
    while left > 0:
        take = min(left, total_steps - s)
        lo = s * S * C
        hi = min(N_EDGES, (s + take) * S * C)
        loss += pbg.pbg_train_bucket(ctx, 0, 0, src[lo:hi], None, dst[lo:hi], C, U, S, LR, SEED,
                                     first_chunk=s * S)
        left -= take
        s = 0
    return loss


def host_cpu():
    """What the oracle's timing ran on: CPU model, cores this process may use
    (its affinity set) and the threads torch's CPU kernels use."""
    import torch
    model = None
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"cpu_model": model, "affinity_cores": len(os.sched_getaffinity(0)),
            "threads": torch.get_num_threads()}


def cpu_baseline(src_h, dst_h, emb_h, chunks):
    """The oracle, as it stands, on the first `chunks` chunks of the bucket."""
    import numpy as np
    import torch
    from oracle import pbg_oracle as O
    from paper_1903_12287_amd import synth
    m = chunks * C
    model = O.Model.create(N_NODES, 1, 1, DIM, "translation", "cos", "ranking", MARGIN,
                           [emb_h], synth.identity_relation_params("translation", 1, DIM))
    t0 = time.perf_counter()
    O.train_bucket(model, 0, 0, src_h[:m], None, dst_h[:m], C, U, S, LR, SEED)
    dt = time.perf_counter() - t0
    return {"value": m / dt, "unit": "edges/s", "cores": torch.get_num_threads(), "kind": "oracle", **host_cpu(),
            "sample": f"first {chunks} chunks ({m} edges) of the same bucket from the same initial "
                      f"state, fp64 numpy/torch-CPU oracle, {dt:.1f} s"}


def run_leg(pbg, torch, flags, emb0, relp0, src, dst, args, total_steps, timing=None, steps=None):
    """Warm-up + timed steps from a copy of the initial state; returns the
    wall time of the timed steps and the library's stats for them.  `timing`:
    the library's event flag (score-only events by default, which add two
    events per step; all phases add seven)."""
    if timing is None:
        timing = pbg.F_SCORE_TIMING
    if steps is None:
        steps = args.steps
    dev = emb0.device
    emb = emb0.clone()
    relp = relp0.clone()
    G = torch.zeros(N_NODES, dtype=torch.float32, device=dev)
    relG = torch.zeros_like(relp)
    ctx = pbg.pbg_bucket_init(N_NODES, 1, 1, DIM, "translation", "cos", "ranking", MARGIN, flags | timing)
    try:
        pbg.pbg_bind_partition(ctx, 0, emb, G)
        pbg.pbg_bind_relations(ctx, relp, relG)
        pbg.pbg_set_streams(ctx, torch.cuda.current_stream(), None)
        train_range(pbg, ctx, src, dst, 0, args.warmup, total_steps)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        train_range(pbg, ctx, src, dst, args.warmup, steps, total_steps)
        torch.cuda.synchronize()
        dt = time.perf_counter() - t0
        st = pbg.pbg_get_stats(ctx)
    finally:
        pbg.pbg_free(ctx)
    del emb, G
    return dt, st


def measured_traffic(name):
    """HBM bytes per step of a kernel group ("score", "gather", "adagrad") from
    the committed rocprofv3 FETCH_SIZE / WRITE_SIZE runs, or None when a source
    of the group has changed since they were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "kernel_hbm_traffic.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path)).get(name)
    if rec is None:
        return None
    for rel, sha in rec["sources"].items():
        if hashlib.sha256(open(os.path.join(ROOT, rel), "rb").read()).hexdigest() != sha:
            return None
    return rec["hbm_read_bytes_per_step"] + rec["hbm_write_bytes_per_step"]


def hbm_rate(st, bytes_key, ms_key, traffic):
    """Achieved HBM rate of a memory-bound phase: algorithmic bytes and, when
    the counters match the sources, measured bytes, over the phase time."""
    sec = st[ms_key] / 1e3
    if sec <= 0:
        return None
    steps = max(1, st["steps"])
    out = {"bound": "hbm", "peak": PEAK_HBM, "unit": "GB/s",
           "achieved_effective": st[bytes_key] / sec / 1e9,
           "frac_effective": st[bytes_key] / sec / 1e9 / PEAK_HBM,
           "algorithmic_bytes_per_step": st[bytes_key] / steps}
    if traffic is not None:
        out["traffic_per_step"] = traffic
        out["achieved_measured"] = traffic * steps / sec / 1e9
        out["frac_measured"] = out["achieved_measured"] / PEAK_HBM
    return out


def roofline(st, kernel, traffic=None, pieces=None, issued=1.0):
    """Dominant kernel: the score contraction with its fused loss epilogue.
    Algorithmic flops per launch: 2 sides x 2 C N d per chunk (a third of the
    12 C N d of the three contractions), one launch per step.  The kernel
    issues v_mfma_f32_16x16x32_bf16 in both precisions; a float32 contraction
    issues `pieces` exact bf16 piece products per product, so its ceiling is
    the bf16 matrix peak over `pieces` (frac), and its rate against the fp32
    matrix peak is given beside it (fp32_peak_frac).  `issued`: the share of
    the algorithmic products the kernel computes (with cos, side 1's in-chunk
    block comes transposed from side 0's tiles)."""
    launches = max(1, st["steps"])
    timed = max(1, st.get("score_timed_steps") or launches)   # launches the events bracketed
    flops = st["score_flops"] / 3.0 / launches                   # per launch
    avg_ms = st["score_ms"] / timed
    achieved = flops / (avg_ms / 1e3) / 1e12 if avg_ms > 0 else None
    peak = PEAK_BF16_MFMA / (pieces or 1)
    out = {"kernel": kernel, "bound": "mfma", "achieved": achieved, "peak": peak,
           "unit": "TFLOP/s", "frac": achieved / peak if achieved else None, "traffic": traffic,
           "avg_launch_ms": avg_ms, "flops_per_launch": flops, "timed_launches": timed}
    if pieces and achieved:
        out["peak_note"] = (f"bf16 matrix peak {PEAK_BF16_MFMA} / {pieces} exact bf16 piece products "
                            "per float32 product (the instruction the kernel issues)")
        out["fp32_peak"] = PEAK_FP32_MFMA
        out["fp32_peak_frac"] = achieved / PEAK_FP32_MFMA
        out["executed_tflops"] = pieces * issued * achieved
    if issued != 1.0:
        out["issued_share"] = issued
    return out


def phases(st):
    return {k: st[k] / max(1, st["steps"]) for k in
            ("gather_ms", "score_ms", "epilogue_ms", "backward_ms", "opbwd_ms", "update_ms")}


def main():
    args = parse()
    if args.calibrate_copy:
        calibrate_copy()
        return
    if args.row:
        if args.gpus != 1:
            print("bench.py runs on one GPU only", file=sys.stderr)
            sys.exit(2)
        print(json.dumps(ROWS[args.row]()))
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); the multi-GPU path is not "
              "built", file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_1903_12287_amd import pbg, synth
    if not os.path.exists(pbg.LIB_PATH):
        from paper_1903_12287_amd import build as _b
        _b.build()
    torch.cuda.set_device(0)
    dev = torch.device("cuda")
    t_gen = time.perf_counter()
    src, dst, emb0 = synth.social_network_device(N_NODES, N_EDGES, DIM, SEED)
    relp0 = torch.from_numpy(synth.identity_relation_params("translation", 1, DIM)).to(dev)
    torch.cuda.synchronize()
    print(f"# workload drawn on device in {time.perf_counter() - t_gen:.1f} s", file=sys.stderr)
    total_steps = -(-N_EDGES // (S * C))

    # the phase breakdown comes from a separate run with events around every
    # kernel group (they add to each step, so the timed run records only the
    # two around the score contraction).  It runs first: after the host-side
    # preparation the GPU takes some 40 ms of this work to reach its loaded
    # clock (the score contraction runs ~15 % slower at first), more than a
    # few warm-up steps cover, and the phase run spans that time.
    phase_steps = 100
    _, stp = run_leg(pbg, torch, 0, emb0, relp0, src, dst, args, total_steps, pbg.F_PHASE_TIMING, phase_steps)
    dt, st = run_leg(pbg, torch, 0, emb0, relp0, src, dst, args, total_steps)
    print(f"# fp32: {st['edges'] / dt:.4g} edges/s", file=sys.stderr)
    out = {
        "metric": "trained edges/sec on 1 MI355X",
        "value": st["edges"] / dt,
        "unit": "edges/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": dt * 1e3 / args.steps,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded, drawn on device; LiveJournal-shaped counts)",
        "config": {"workload": "social_network", "nodes": N_NODES, "edges": N_EDGES, "dim": DIM,
                   "operator": "translation", "comparator": "cos", "loss": "ranking",
                   "chunk": C, "uniform_negatives": U, "chunks_per_step": S,
                   "edges_per_step": S * C, "partitions": 1},
        "roofline": roofline(st, "score_split_kernel3<EPI_LOSS_BITS, 6> (float32 score + ranking epilogue)",
                             measured_traffic("score"), pieces=SPLIT_PIECES,
                             issued=1.0 - (128 * (C // 128)) ** 2 / (2.0 * C * (C + U))),
        # from the phase-timing run of phase_steps steps
        "phases_ms_per_step": phases(stp),
        "phase_steps": phase_steps,
        "backward_contractions_tflops": (2 * stp["score_flops"] / 3.0) / (stp["backward_ms"] / 1e3) / 1e12
        if stp["backward_ms"] > 0 else None,
        # the gather (gather_op_kernel) and the entity Adagrad update
        # (seg_update_local + seg_update_span) against HBM peak
        "gather_hbm": hbm_rate(stp, "gather_bytes", "gather_ms", measured_traffic("gather")),
        "adagrad_hbm": hbm_rate(stp, "update_bytes", "update_ms", measured_traffic("adagrad")),
    }
    if not args.no_bf16:
        _, st16p = run_leg(pbg, torch, pbg.F_BF16_SCORE, emb0, relp0, src, dst, args, total_steps,
                           pbg.F_PHASE_TIMING, phase_steps)
        dt16, st16 = run_leg(pbg, torch, pbg.F_BF16_SCORE, emb0, relp0, src, dst, args, total_steps)
        print(f"# bf16: {st16['edges'] / dt16:.4g} edges/s", file=sys.stderr)
        out["bf16"] = {"value": st16["edges"] / dt16, "unit": "edges/s",
                       "ms_per_step": dt16 * 1e3 / args.steps, "dtype": "bf16 inputs, f32 accumulate",
                       "roofline": roofline(st16, "gemm_bf16_kernel<128,GA_KC,EPI_LOSS_BITS,1> "
                                                  "(score + ranking epilogue)"),
                       "phases_ms_per_step": phases(st16p)}
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(src.cpu().numpy(), dst.cpu().numpy(), emb0.cpu().numpy(),
                                           args.cpu_sample_chunks)
    if not args.no_big_bucket:
        # the one-GPU share of the partitioned run: one whole bucket at its real shape
        del src, dst, emb0
        torch.cuda.empty_cache()
        out["big_bucket"] = big_bucket_legs(with_cpu=False)
    print(json.dumps(out))


# ---------------------------------------------------------------------------
# Other rows of the hot path (bench.py --row ...).  Each prints one JSON line
# with its throughput, the roofline of its dominant kernel and the oracle
# timed on a bounded sample on the host.
# ---------------------------------------------------------------------------
def _median_time(fn, reps=3):
    import torch
    times = []
    for _ in range(reps):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        fn()
        torch.cuda.synchronize()
        times.append(time.perf_counter() - t0)
    times.sort()
    return times[len(times) // 2]


def _cores():
    import torch
    return torch.get_num_threads()





def row_bucketing():
    """Edge bucketing of the follower-graph-shaped graph (41,652,230 nodes,
    1,468,365,182 edges, Zipf 1.2 sources / 0.9 destinations, 8 partitions)."""
    import numpy as np
    import torch
    from oracle import pbg_oracle as O
    from paper_1903_12287_amd import pbg, synth
    n, E, P = 41_652_230, 1_468_365_182, 8
    torch.cuda.set_device(0)
    src, dst = synth.zipf_edges_device(n, E, 1.2, 0.9, synth.device_generator(20190005))
    dev = torch.device("cuda")
    offsets = torch.empty(P * P + 1, dtype=torch.int64, device=dev)
    sl = torch.empty(E, dtype=torch.int32, device=dev)
    dl = torch.empty(E, dtype=torch.int32, device=dev)
    ctx = pbg.pbg_bucket_init(n, P, 1, 100, "linear", "dot", "logistic")
    try:
        pbg.pbg_set_streams(ctx, torch.cuda.current_stream(), None)
        pbg.pbg_bucket_edges(ctx, src, None, dst, offsets, sl, None, dl)
        dt = _median_time(lambda: pbg.pbg_bucket_edges(ctx, src, None, dst, offsets, sl, None, dl))
    finally:
        pbg.pbg_free(ctx)
    alg_bytes = E * (8 + 8 + 4 + 4)          # read two int64 ids, write two int32 local ids
    m = 30_000_000
    hs, hd = src[:m].cpu().numpy(), dst[:m].cpu().numpy()
    t0 = time.perf_counter()
    O.bucket_edges(hs, np.zeros(m, np.int32), hd, n, P)
    ct = time.perf_counter() - t0
    return {"metric": "edges bucketed/sec on 1 MI355X", "value": E / dt, "unit": "edges/s",
            "ms": dt * 1e3, "dtype": "int64 -> int32",
            "config": {"workload": "follower_graph", "nodes": n, "edges": E, "partitions": P},
            "roofline": {"bound": "hbm", "achieved": alg_bytes / dt / 1e9, "peak": PEAK_HBM, "unit": "GB/s",
                         "frac": alg_bytes / dt / 1e9 / PEAK_HBM, "traffic": None,
                         "note": "algorithmic bytes = 24 per edge (two int64 ids in, two int32 local ids out); "
                                 "the call also makes one stable radix pass over 8-byte key/position pairs"},
            "cpu_baseline": {"value": m / ct, "unit": "edges/s", "cores": _cores(), "kind": "oracle", **host_cpu(),
                             "sample": f"first {m} edges, numpy stable argsort, {ct:.1f} s"}}


def row_knowledge_graph(reciprocal=False):
    """Knowledge-graph-shaped graph (15,000 entities, 1,345 relations, 483,000
    training + 50,000 held-out triples, d = 400, complex_diagonal, dot,
    softmax): one training pass and the filtered rank evaluation of the
    held-out triples against all entities on both sides.  reciprocal: with
    reciprocal predicates (a second parameter row per relation for the source
    side, Sec. 5.4's recipe for this model)."""
    import numpy as np
    import torch
    from oracle import pbg_oracle as O
    from paper_1903_12287_amd import pbg, synth
    torch.cuda.set_device(0)
    w = synth.knowledge_graph()
    rng = synth.rng_for(w.seed + 1)
    emb0 = synth.init_embeddings(w.n, w.d, rng)
    rel0 = synth.identity_relation_params(w.op, 2 * w.R if reciprocal else w.R, w.d)
    dev = torch.device("cuda")
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.int32)).to(dev)
    src, rel, dst = t(w.src), t(w.rel), t(w.dst)
    out = {"metric": "trained edges/sec on 1 MI355X", "unit": "edges/s", "dtype": "f32",
           "config": {"workload": "knowledge_graph", "entities": w.n, "relations": w.R, "train": w.E,
                      "held_out": len(w.held_src), "dim": w.d, "operator": w.op, "comparator": w.cmp,
                      "loss": w.loss, "chunk": w.C, "uniform_negatives": w.U, "chunks_per_step": w.S,
                      "reciprocal_predicates": reciprocal}}
    emb = torch.from_numpy(emb0.copy()).to(dev)
    G = torch.zeros(w.n, dtype=torch.float32, device=dev)
    relp = torch.from_numpy(rel0.copy()).to(dev)
    relG = torch.zeros_like(relp)
    ctx = pbg.pbg_bucket_init(w.n, 1, w.R, w.d, w.op, w.cmp, w.loss, w.margin,
                              pbg.F_PHASE_TIMING | (pbg.F_RECIPROCAL if reciprocal else 0))
    try:
        pbg.pbg_bind_partition(ctx, 0, emb, G)
        pbg.pbg_bind_relations(ctx, relp, relG)
        pbg.pbg_set_streams(ctx, torch.cuda.current_stream(), None)
        pbg.pbg_train_bucket(ctx, 0, 0, src, rel, dst, w.C, w.U, w.S, w.lr, w.seed)   # warm-up pass
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        pbg.pbg_train_bucket(ctx, 0, 0, src, rel, dst, w.C, w.U, w.S, w.lr, w.seed + 1)
        torch.cuda.synchronize()
        dt = time.perf_counter() - t0
        st = pbg.pbg_get_stats(ctx)
        out["value"] = w.E / dt
        out["ms_per_pass"] = dt * 1e3
        out["roofline"] = roofline(st, "score_split_kernel<EPI_SOFTMAX_EXP, 6> (score)", pieces=SPLIT_PIECES)
        out["phases_ms_per_step"] = phases(st)
        # filtered ranks of the held-out triples, known = train + held-out
        hs, hr, hd = t(w.held_src), t(w.held_rel), t(w.held_dst)
        ks, kr, kd = (t(np.concatenate([w.src, w.held_src])), t(np.concatenate([w.rel, w.held_rel])),
                      t(np.concatenate([w.dst, w.held_dst])))
        ranks = torch.empty(2 * len(w.held_src), dtype=torch.int32, device=dev)
        pbg.pbg_rank_eval(ctx, hs, hr, hd, ks, kr, kd, ranks)
        et = _median_time(lambda: pbg.pbg_rank_eval(ctx, hs, hr, hd, ks, kr, kd, ranks))
        mrr, hits = pbg.pbg_rank_eval(ctx, hs, hr, hd, ks, kr, kd, ranks)
        flops = 2.0 * 2.0 * len(w.held_src) * w.n * w.d
        out["rank_eval"] = {"value": len(w.held_src) / et, "unit": "held-out triples/s (both sides)",
                            "ms": et * 1e3, "mrr": mrr, "hits10": hits,
                            "roofline": {"bound": "mfma", "achieved": flops / et / 1e12,
                                         "peak": PEAK_BF16_MFMA / SPLIT_PIECES, "unit": "TFLOP/s",
                                         "frac": flops / et / 1e12 / (PEAK_BF16_MFMA / SPLIT_PIECES),
                                         "fp32_peak_frac": flops / et / 1e12 / PEAK_FP32_MFMA,
                                         "traffic": None,
                                         "note": "2 sides x 2 x held-out x entities x dim flops of candidate "
                                                 "scores, whole call time"}}
        # raw ranks against 10,000 candidates drawn by prevalence (the
        # large-graph evaluation), the same held-out triples
        cand_h = synth.prevalence_candidates(w.src, w.dst, w.n, 10_000, synth.rng_for(w.seed + 2))
        cand = t(cand_h)
        pbg.pbg_rank_sampled(ctx, hs, hr, hd, cand, ranks)
        st_ = _median_time(lambda: pbg.pbg_rank_sampled(ctx, hs, hr, hd, cand, ranks))
        smrr, shits = pbg.pbg_rank_sampled(ctx, hs, hr, hd, cand, ranks)
        sflops = 2.0 * 2.0 * len(w.held_src) * len(cand_h) * w.d
        out["rank_sampled"] = {"value": len(w.held_src) / st_, "unit": "held-out triples/s (both sides)",
                               "ms": st_ * 1e3, "candidates": len(cand_h), "mrr": smrr, "hits10": shits,
                               "roofline": {"bound": "mfma", "achieved": sflops / st_ / 1e12,
                                            "peak": PEAK_BF16_MFMA / SPLIT_PIECES, "unit": "TFLOP/s",
                                            "frac": sflops / st_ / 1e12 / (PEAK_BF16_MFMA / SPLIT_PIECES),
                                            "fp32_peak_frac": sflops / st_ / 1e12 / PEAK_FP32_MFMA,
                                            "traffic": None,
                                            "note": "2 sides x 2 x held-out x candidates x dim flops of "
                                                    "candidate scores, whole call time"}}
        emb_h = emb.cpu().numpy()
        relp_h = relp.cpu().numpy()
    finally:
        pbg.pbg_free(ctx)
    model = O.Model.create(w.n, 1, w.R, w.d, w.op, w.cmp, w.loss, w.margin, [emb0.astype(np.float64)],
                           rel0.astype(np.float64), reciprocal=reciprocal)
    m = 10 * w.C
    c0 = time.perf_counter()
    O.train_bucket(model, 0, 0, w.src[:m], w.rel[:m], w.dst[:m], w.C, w.U, w.S, w.lr, w.seed)
    ct = time.perf_counter() - c0
    out["cpu_baseline"] = {"value": m / ct, "unit": "edges/s", "cores": _cores(), "kind": "oracle", **host_cpu(),
                           "sample": f"first 10 chunks ({m} edges), one step, fp64, {ct:.1f} s"}
    emodel = O.Model.create(w.n, 1, w.R, w.d, w.op, w.cmp, w.loss, w.margin, [emb_h.astype(np.float64)],
                            relp_h.astype(np.float64), reciprocal=reciprocal)
    k = 100
    c0 = time.perf_counter()
    O.rank_eval(emodel, w.held_src[:k], w.held_rel[:k], w.held_dst[:k], np.concatenate([w.src, w.held_src]),
                np.concatenate([w.rel, w.held_rel]), np.concatenate([w.dst, w.held_dst]))
    ct = time.perf_counter() - c0
    out["rank_eval"]["cpu_baseline"] = {"value": k / ct, "unit": "held-out triples/s", "cores": _cores(),
                                        "kind": "oracle", **host_cpu(), "sample": f"first {k} held-out triples, {ct:.1f} s"}
    c0 = time.perf_counter()
    O.rank_sampled(emodel, w.held_src[:k], w.held_rel[:k], w.held_dst[:k], cand_h)
    ct = time.perf_counter() - c0
    out["rank_sampled"]["cpu_baseline"] = {"value": k / ct, "unit": "held-out triples/s", "cores": _cores(),
                                           "kind": "oracle", **host_cpu(), "sample": f"first {k} held-out triples, {ct:.1f} s"}
    return out


def _big_bucket_tensors(torch, synth):
    n, P, i, j, R, E, d = 121_216_723, 16, 3, 7, 5_000, 9_375_000, 100
    ps = -(-n // P)
    gen = synth.device_generator(20190004)
    src, _ = synth.zipf_device(ps, 1.0, E, gen)
    dst, _ = synth.zipf_device(ps, 1.0, E, gen)
    rel, _ = synth.zipf_device(R, 1.3, E, gen)
    emb_i = synth.init_embeddings_device(ps, d, gen)
    emb_j = synth.init_embeddings_device(ps, d, gen)
    return (n, P, i, j, R, E, d, ps, src.to(torch.int32), rel.to(torch.int32), dst.to(torch.int32),
            emb_i, emb_j)


def big_bucket_legs(with_cpu=True, phase_steps=20):
    """Bucket (3, 7) of a large partitioned knowledge-graph-shaped run
    (121,216,723 entities in 16 partitions of 7,576,046 rows, 9,375,000 edges,
    5,000 relations Zipf 1.3, d = 100, diagonal, dot, ranking 0.1): one pass
    in fp32 and one with bf16 score inputs, both partitions resident in HBM,
    each after a 10-step warm-up; the phase breakdown from a separate run of
    `phase_steps` steps with events around every kernel group."""
    import numpy as np
    import torch
    from oracle import pbg_oracle as O
    from paper_1903_12287_amd import pbg, synth
    torch.cuda.set_device(0)
    n, P, i, j, R, E, d, ps, src, rel, dst, emb_i0, emb_j0 = _big_bucket_tensors(torch, synth)
    relp0 = torch.ones(R, d, dtype=torch.float32, device="cuda")
    Cb, Ub, Sb = 1000, 1000, 40
    out = {"metric": "trained edges/sec on 1 MI355X", "unit": "edges/s", "dtype": "f32",
           "config": {"workload": "big_bucket", "entities": n, "partitions": P, "bucket": [i, j],
                      "rows_per_partition": ps, "edges": E, "relations": R, "dim": d, "operator": "diagonal",
                      "comparator": "dot", "loss": "ranking", "chunk": Cb, "uniform_negatives": Ub,
                      "chunks_per_step": Sb}}

    def leg(flags, timing, m):
        emb_i, emb_j, relp = emb_i0.clone(), emb_j0.clone(), relp0.clone()
        Gi = torch.zeros(ps, device="cuda")
        Gj = torch.zeros(ps, device="cuda")
        relG = torch.zeros_like(relp)
        ctx = pbg.pbg_bucket_init(n, P, R, d, "diagonal", "dot", "ranking", 0.1, flags | timing)
        try:
            pbg.pbg_bind_partition(ctx, i, emb_i, Gi)
            pbg.pbg_bind_partition(ctx, j, emb_j, Gj)
            pbg.pbg_bind_relations(ctx, relp, relG)
            pbg.pbg_set_streams(ctx, torch.cuda.current_stream(), None)
            w = 10 * Sb * Cb
            pbg.pbg_train_bucket(ctx, i, j, src[:w], rel[:w], dst[:w], Cb, Ub, Sb, 0.1, 1)   # warm-up
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            pbg.pbg_train_bucket(ctx, i, j, src[:m], rel[:m], dst[:m], Cb, Ub, Sb, 0.1, 20190004)
            torch.cuda.synchronize()
            dt = time.perf_counter() - t0
            st = pbg.pbg_get_stats(ctx)
        finally:
            pbg.pbg_free(ctx)
        return dt, st

    for flags, key in ((0, None), (pbg.F_BF16_SCORE, "bf16")):
        # the phase run first, as in the default line (it brings the GPU to its loaded clock)
        _, stp = leg(flags, pbg.F_PHASE_TIMING, phase_steps * Sb * Cb)
        dt, st = leg(flags, pbg.F_SCORE_TIMING, E)
        res = {"value": E / dt, "ms_per_pass": dt * 1e3, "ms_per_step": dt * 1e3 / max(1, st["steps"]),
               "roofline": roofline(st, "score contraction with the ranking epilogue",
                                    pieces=None if flags else SPLIT_PIECES),
               "phases_ms_per_step": phases(stp), "phase_steps": phase_steps,
               "gather_hbm": hbm_rate(stp, "gather_bytes", "gather_ms", None),
               "adagrad_hbm": hbm_rate(stp, "update_bytes", "update_ms", None)}
        if key:
            res["dtype"] = "bf16 inputs, f32 accumulate"
            out[key] = res
        else:
            out.update(res)
        print(f"# big bucket {key or 'fp32'}: {E / dt:.4g} edges/s", file=sys.stderr, flush=True)
    if with_cpu:
        # oracle: the first 10 chunks from the same initial state, partitions i and j only
        m = 10 * Cb
        model = O.Model(n, P, R, d, "diagonal", "dot", "ranking", 0.1)
        model.emb = {i: emb_i0.cpu().numpy().astype(np.float64), j: emb_j0.cpu().numpy().astype(np.float64)}
        model.G = {i: np.zeros(ps), j: np.zeros(ps)}
        model.rel = np.ones((R, d))
        model.relG = np.zeros((R, d))
        hs, hr, hd = src[:m].cpu().numpy(), rel[:m].cpu().numpy(), dst[:m].cpu().numpy()
        c0 = time.perf_counter()
        O.train_bucket(model, i, j, hs, hr, hd, Cb, Ub, Sb, 0.1, 20190004)
        ct = time.perf_counter() - c0
        out["cpu_baseline"] = {"value": m / ct, "unit": "edges/s", "cores": _cores(), "kind": "oracle",
                               **host_cpu(), "sample": f"first 10 chunks ({m} edges) of the bucket, fp64, "
                                                       f"{ct:.1f} s"}
    return out


def row_big_bucket():
    return big_bucket_legs(with_cpu=True)


def row_epoch():
    """Follower-graph-shaped partitioned epoch (41,652,230 nodes,
    1,468,365,182 edges, 8 partitions, d = 100, linear, dot, logistic): every
    non-empty bucket in inside-out order, partitions in page-locked host memory
    swapped through 3 HBM slots on a copy stream.  Edges are bucketed on the
    device first (not timed)."""
    import numpy as np
    import torch
    from oracle import pbg_oracle as O
    from paper_1903_12287_amd import pbg, synth
    torch.cuda.set_device(0)
    n, E, P, d = 41_652_230, 1_468_365_182, 8, 100
    Ce, Ue, Se = 1000, 1000, 40
    gen = synth.device_generator(20190005)
    src, dst = synth.zipf_edges_device(n, E, 1.2, 0.9, gen)
    dev = torch.device("cuda")
    offsets = torch.empty(P * P + 1, dtype=torch.int64, device=dev)
    sl = torch.empty(E, dtype=torch.int32, device=dev)
    dl = torch.empty(E, dtype=torch.int32, device=dev)
    ctx = pbg.pbg_bucket_init(n, P, 1, d, "linear", "dot", "logistic", 0.1, pbg.F_PHASE_TIMING)
    try:
        pbg.pbg_set_streams(ctx, torch.cuda.current_stream(), None)
        pbg.pbg_bucket_edges(ctx, src, None, dst, offsets, sl, None, dl)
        del src, dst
        off_h = offsets.cpu()
        sl_h = torch.empty(E, dtype=torch.int32, pin_memory=True)
        dl_h = torch.empty(E, dtype=torch.int32, pin_memory=True)
        sl_h.copy_(sl)
        dl_h.copy_(dl)
        del sl, dl
        rows = [pbg.pbg_partition_rows(ctx, p) for p in range(P)]
        embs, Gs = [], []
        for p in range(P):
            e = torch.empty(rows[p], d, dtype=torch.float32, pin_memory=True)
            e.copy_(synth.init_embeddings_device(rows[p], d, gen))
            embs.append(e)
            Gs.append(torch.zeros(rows[p], dtype=torch.float32, pin_memory=True))
            pbg.pbg_bind_partition(ctx, p, embs[p], Gs[p], pbg.MEM_PINNED_HOST)
        relp = torch.eye(d, dtype=torch.float32, device=dev).reshape(1, d * d).contiguous()
        relG = torch.zeros_like(relp)
        pbg.pbg_bind_relations(ctx, relp, relG)
        copy = torch.cuda.Stream()
        pbg.pbg_set_streams(ctx, torch.cuda.current_stream(), copy)
        torch.cuda.synchronize()
        emb0_h = embs[0].numpy().copy()
        print(f"# epoch inputs ready: {E} edges in {P * P} buckets, {P} pinned partitions", file=sys.stderr)
        t0 = time.perf_counter()
        loss = pbg.pbg_train_epoch(ctx, off_h, sl_h, None, dl_h, Ce, Ue, Se, 0.1, 20190005, 3)
        torch.cuda.synchronize()
        dt = time.perf_counter() - t0
        st = pbg.pbg_get_stats(ctx)
    finally:
        pbg.pbg_free(ctx)
    m = Se * Ce
    b00 = int(off_h[1])
    model = O.Model(n, P, 1, d, "linear", "dot", "logistic", 0.1)
    model.emb = {0: emb0_h.astype(np.float64)}
    model.G = {0: np.zeros(rows[0])}
    model.rel = np.eye(d).reshape(1, d * d)
    model.relG = np.zeros((1, d * d))
    c0 = time.perf_counter()
    O.train_bucket(model, 0, 0, sl_h[:min(m, b00)].numpy(), None, dl_h[:min(m, b00)].numpy(), Ce, Ue, Se, 0.1,
                   20190005)
    ct = time.perf_counter() - c0
    return {"metric": "trained edges/sec on 1 MI355X, whole epoch incl. partition swaps and edge transfers",
            "value": E / dt, "unit": "edges/s", "seconds": dt, "dtype": "f32", "loss": loss,
            "config": {"workload": "follower_graph_epoch", "nodes": n, "edges": E, "partitions": P,
                       "buckets": P * P, "dim": d, "operator": "linear", "comparator": "dot",
                       "loss": "logistic", "chunk": Ce, "uniform_negatives": Ue, "chunks_per_step": Se,
                       "max_resident": 3},
            "partition_loads": st["partition_loads"], "copy_ms": st["copy_ms"],
            "compute_ms": sum(st[k] for k in ("gather_ms", "score_ms", "epilogue_ms", "backward_ms",
                                               "opbwd_ms", "update_ms")),
            "roofline": roofline(st, "score contraction with the logistic epilogue", pieces=SPLIT_PIECES),
            "phases_ms_per_step": phases(st),
            "cpu_baseline": {"value": min(m, b00) / ct, "unit": "edges/s", "cores": _cores(), "kind": "oracle", **host_cpu(),
                             "sample": f"first {min(m, b00)} edges of bucket (0, 0), fp64, {ct:.1f} s"}}


def row_tiny():
    """Tiny social graph (10,000 nodes, 100,000 edges, d = 32, identity, dot,
    ranking 0.1, C = U = 100): one full pass, and the oracle's full pass."""
    import numpy as np
    import torch
    from oracle import pbg_oracle as O
    from paper_1903_12287_amd import pbg, synth
    torch.cuda.set_device(0)
    w = synth.tiny_social()
    emb0 = synth.init_embeddings(w.n, w.d, synth.rng_for(w.seed + 1))
    dev = torch.device("cuda")
    src = torch.from_numpy(w.src.astype(np.int32)).to(dev)
    dst = torch.from_numpy(w.dst.astype(np.int32)).to(dev)
    emb = torch.from_numpy(emb0.copy()).to(dev)
    G = torch.zeros(w.n, device=dev)
    ctx = pbg.pbg_bucket_init(w.n, 1, 1, w.d, w.op, w.cmp, w.loss, w.margin)
    try:
        pbg.pbg_bind_partition(ctx, 0, emb, G)
        pbg.pbg_set_streams(ctx, torch.cuda.current_stream(), None)
        pbg.pbg_train_bucket(ctx, 0, 0, src, None, dst, w.C, w.U, w.S, w.lr, w.seed)
        dt = _median_time(lambda: pbg.pbg_train_bucket(ctx, 0, 0, src, None, dst, w.C, w.U, w.S, w.lr, w.seed))
    finally:
        pbg.pbg_free(ctx)
    model = O.Model.create(w.n, 1, 1, w.d, w.op, w.cmp, w.loss, w.margin, [emb0.astype(np.float64)])
    c0 = time.perf_counter()
    O.train_bucket(model, 0, 0, w.src, None, w.dst, w.C, w.U, w.S, w.lr, w.seed)
    ct = time.perf_counter() - c0
    return {"metric": "trained edges/sec on 1 MI355X", "value": w.E / dt, "unit": "edges/s",
            "ms_per_pass": dt * 1e3, "dtype": "f32",
            "config": {"workload": "tiny_social", "nodes": w.n, "edges": w.E, "dim": w.d, "operator": w.op,
                       "comparator": w.cmp, "loss": w.loss, "chunk": w.C, "uniform_negatives": w.U,
                       "chunks_per_step": w.S},
            "note": "the 1.3 MB table stays in cache and a pass is 25 steps of ~30 small launches: "
                    "launch latency bound, no roofline figure",
            "cpu_baseline": {"value": w.E / ct, "unit": "edges/s", "cores": _cores(), "kind": "oracle", **host_cpu(),
                             "sample": f"full pass ({w.E} edges), fp64, {ct:.1f} s"}}


def row_negatives():
    """Training speed against the number of negatives per edge, batched and
    unbatched (the comparison of Sec. 4.3 / Fig. 4), on the social-network
    graph (translation, cos, ranking, d = 128): batched, a chunk of B/2 edges
    is corrupted with its own entities and B/2 uniform draws (B negatives per
    edge, scored by contractions); unbatched, every edge is its own chunk with
    B uniform draws (chunk_size 1: one score row per edge).  Batched: 40 chunks
    a step, 50 steps; unbatched: 1,000 one-edge chunks a step (so that a step
    carries 1,000 edges, not 40), 10 steps.  Each point times whole steps after
    one warm-up call."""
    import torch
    from paper_1903_12287_amd import pbg, synth
    torch.cuda.set_device(0)
    dev = torch.device("cuda")
    src, dst, emb0 = synth.social_network_device(N_NODES, N_EDGES, DIM, SEED)
    relp0 = torch.zeros(DIM, dtype=torch.float32, device=dev)
    points = []
    for B in (10, 50, 100, 200, 500, 1000, 2000):
        for mode, c, u in (("batched", B // 2, B - B // 2), ("unbatched", 1, B)):
            steps, S_ = (50, 40) if mode == "batched" else (10, 1000)
            e_call = steps * S_ * c
            emb = emb0.clone()
            G = torch.zeros(N_NODES, dtype=torch.float32, device=dev)
            relp = relp0.clone()
            ctx = pbg.pbg_bucket_init(N_NODES, 1, 1, DIM, "translation", "cos", "ranking", MARGIN)
            try:
                pbg.pbg_bind_partition(ctx, 0, emb, G)
                pbg.pbg_bind_relations(ctx, relp, torch.zeros_like(relp))
                pbg.pbg_set_streams(ctx, torch.cuda.current_stream(), None)
                run = lambda: pbg.pbg_train_bucket(ctx, 0, 0, src[:e_call], None, dst[:e_call], c, u, S_, LR, SEED)
                run()
                torch.cuda.synchronize()
                t0 = time.perf_counter()
                run()
                torch.cuda.synchronize()
                dt = time.perf_counter() - t0
            finally:
                pbg.pbg_free(ctx)
            points.append({"negatives": B, "mode": mode, "chunk": c, "uniform": u, "chunks_per_step": S_,
                           "edges": e_call, "edges_per_s": e_call / dt})
            print(f"# {mode} B={B}: {e_call / dt:.4g} edges/s", file=sys.stderr, flush=True)
    best = max(p["edges_per_s"] for p in points if p["mode"] == "batched" and p["negatives"] == 1000)
    return {"metric": "trained edges/sec on 1 MI355X", "value": best, "unit": "edges/s", "dtype": "f32",
            "config": {"workload": "social_network negatives sweep", "nodes": N_NODES, "dim": DIM,
                       "operator": "translation", "comparator": "cos", "loss": "ranking"},
            "note": "value: batched, 1000 negatives per edge; points: every (negatives, mode)",
            "points": points}


def row_library_gemm():
    """Context for the matrix-peak fractions: what the vendor GEMM libraries
    (torch.bmm / torch.matmul on ROCm) reach on this GPU, at the score
    contraction's shape (80 chunk-sides of 1000 x 128 times 128 x 2000, the
    library writing S, no loss) and as large square products.  Not part of
    the hot path."""
    import torch
    torch.backends.cuda.matmul.allow_tf32 = False
    dev = torch.device("cuda")

    def timed(f, it):
        for _ in range(3):
            f()
        torch.cuda.synchronize()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(it):
            f()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / it

    out = []
    B, M, K, Nn = 2 * S, C, DIM, C + U
    for name, dt in (("f32", torch.float32), ("bf16", torch.bfloat16)):
        q = torch.randn(B, M, K, device=dev, dtype=dt)
        nt = torch.randn(B, Nn, K, device=dev, dtype=dt).transpose(1, 2).contiguous()
        ms = timed(lambda: torch.bmm(q, nt), 20)
        fl = 2.0 * B * M * Nn * K
        peak = PEAK_FP32_MFMA if dt == torch.float32 else PEAK_BF16_MFMA
        out.append({"op": "bmm", "dtype": name, "shape": [B, M, K, Nn], "us": ms * 1e3,
                    "tflops": fl / ms / 1e9, "peak": peak, "frac": fl / ms / 1e9 / peak})
        del q, nt
    for sz in (4096, 8192):
        for name, dt in (("bf16", torch.bfloat16), ("f32", torch.float32)):
            a = torch.randn(sz, sz, device=dev, dtype=dt)
            b = torch.randn(sz, sz, device=dev, dtype=dt)
            ms = timed(lambda: a @ b, 10)
            fl = 2.0 * sz ** 3
            peak = PEAK_FP32_MFMA if dt == torch.float32 else PEAK_BF16_MFMA
            out.append({"op": "matmul", "dtype": name, "shape": [sz, sz, sz], "us": ms * 1e3,
                        "tflops": fl / ms / 1e9, "peak": peak, "frac": fl / ms / 1e9 / peak})
            del a, b
    return {"row": "library_gemm", "unit": "TFLOP/s", "results": out}


ROWS = {"bucketing": row_bucketing, "knowledge_graph": row_knowledge_graph,
        "knowledge_graph_reciprocal": lambda: row_knowledge_graph(reciprocal=True), "big_bucket": row_big_bucket,
        "epoch": row_epoch, "tiny": row_tiny, "negatives": row_negatives, "library_gemm": row_library_gemm}


if __name__ == "__main__":
    main()
