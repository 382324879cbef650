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


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=400)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--cpu-sample-chunks", type=int, default=400,
                    help="chunks of the same bucket the CPU oracle is timed on")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-bf16", action="store_true", help="skip the bf16-input leg")
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
    return {"value": m / dt, "unit": "edges/s", "cores": torch.get_num_threads(), "kind": "oracle",
            "sample": f"first {chunks} chunks ({m} edges) of the same bucket from the same initial "
                      f"state, fp64 numpy/torch-CPU oracle, {dt:.1f} s"}


def run_leg(pbg, torch, flags, emb0, relp0, src, dst, args, total_steps):
    """Warm-up + timed steps from a copy of the initial state; returns the
    wall time of the timed steps and the library's stats for them."""
    dev = emb0.device
    emb = emb0.clone()
    relp = relp0.clone()
    G = torch.zeros(N_NODES, dtype=torch.float32, device=dev)
    relG = torch.zeros_like(relp)
    ctx = pbg.pbg_bucket_init(N_NODES, 1, 1, DIM, "translation", "cos", "ranking", MARGIN,
                              flags | pbg.F_PHASE_TIMING)
    try:
        pbg.pbg_bind_partition(ctx, 0, emb, G)
        pbg.pbg_bind_relations(ctx, relp, relG)
        pbg.pbg_set_streams(ctx, torch.cuda.current_stream(), None)
        train_range(pbg, ctx, src, dst, 0, args.warmup, total_steps)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        train_range(pbg, ctx, src, dst, args.warmup, args.steps, total_steps)
        torch.cuda.synchronize()
        dt = time.perf_counter() - t0
        st = pbg.pbg_get_stats(ctx)
    finally:
        pbg.pbg_free(ctx)
    del emb, G
    return dt, st


def measured_traffic(kernel_source_rel):
    """HBM bytes per launch of the score kernel from the committed rocprofv3
    counter runs, or None when the kernel source has changed since they were
    taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "score_kernel_hbm_traffic.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    src = open(os.path.join(ROOT, kernel_source_rel), "rb").read()
    if rec.get("source_sha256") != hashlib.sha256(src).hexdigest():
        return None
    return rec["hbm_read_bytes_per_launch"] + rec["hbm_write_bytes_per_launch"]


def roofline(st, peak, kernel, traffic=None):
    """Dominant kernel: the score contraction with its fused loss epilogue.
    Algorithmic flops per launch: 2 sides x 2 C N d per chunk (a third of the
    12 C N d of the three contractions), one launch per step."""
    launches = max(1, st["steps"])
    flops = st["score_flops"] / 3.0
    achieved = flops / (st["score_ms"] / 1e3) / 1e12 if st["score_ms"] > 0 else None
    return {"kernel": kernel, "bound": "mfma", "achieved": achieved, "peak": peak,
            "unit": "TFLOP/s", "frac": achieved / peak if achieved else None, "traffic": traffic,
            "avg_launch_ms": st["score_ms"] / launches, "flops_per_launch": flops / launches}


def phases(st):
    return {k: st[k] / max(1, st["steps"]) for k in
            ("gather_ms", "score_ms", "epilogue_ms", "backward_ms", "opbwd_ms", "update_ms")}


def main():
    args = parse()
    if args.calibrate_copy:
        calibrate_copy()
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
        "roofline": roofline(st, PEAK_FP32_MFMA,
                             "gemm_f32_kernel<128,true,true,EPI_LOSS_BITS> (score + ranking epilogue)",
                             measured_traffic("paper_1903_12287_amd/csrc/kernels_gemm.hip")),
        "phases_ms_per_step": phases(st),
        "backward_contractions_tflops": (2 * st["score_flops"] / 3.0) / (st["backward_ms"] / 1e3) / 1e12
        if st["backward_ms"] > 0 else None,
        "gather_gbps_effective": st["gather_bytes"] / (st["gather_ms"] / 1e3) / 1e9
        if st["gather_ms"] > 0 else None,
    }
    if not args.no_bf16:
        dt16, st16 = run_leg(pbg, torch, pbg.F_BF16_SCORE, emb0, relp0, src, dst, args, total_steps)
        print(f"# bf16: {st16['edges'] / dt16:.4g} edges/s", file=sys.stderr)
        out["bf16"] = {"value": st16["edges"] / dt16, "unit": "edges/s",
                       "ms_per_step": dt16 * 1e3 / args.steps, "dtype": "bf16 inputs, f32 accumulate",
                       "roofline": roofline(st16, PEAK_BF16_MFMA,
                                            "gemm_bf16_kernel<8,LOSS> (score + ranking epilogue)"),
                       "phases_ms_per_step": phases(st16)}
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(src.cpu().numpy(), dst.cpu().numpy(), emb0.cpu().numpy(),
                                           args.cpu_sample_chunks)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
