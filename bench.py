#!/usr/bin/env python3
"""Throughput of the NN-select + encode serving path on one MI355X.

One step = one tav2_select_encode call over one ranking request's batch of
candidates with every input already resident in HBM: exact top-k over the
user's lifelong sequence for every candidate, token assembly, feature encoding,
the causal encoder and the pooled head.  The default workload is one request
with a 16384-action lifelong sequence (d = 256, bf16), 1000 candidates and
k = 256, encoded by 2 layers of d_model 256 / 4 heads / FFN 1024.

Prints one JSON line: candidates/s (whole job), the dominant kernel's
roofline position, and the CPU oracle's throughput on a bounded sample.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "candidates scored/sec at L=16k (NN-select+encode); % MFMA / HBM roofline"
METRIC_SELECT = "candidates NN-selected/sec at L=16k over int8 codes (fused dequant + L2 norm)"
PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3       # MI355X fp32 vector
PEAK_HBM_GBS = 8000.0         # MI355X HBM3E


def site_work(w, total, valid_tokens, max_len, launches_per_step):
    """Algorithmic work of one launch of each kernel site.

    Returns {site: (kind, amount)} with kind 'flop' or 'byte'.  Only the work the
    method defines is counted: valid tokens only, causal attention over
    T (T + 1) / 2 query-key pairs, scores 2 L d per candidate, the top-k's read
    of the score rows.
    """
    dm, ff, d, H = w.d_model, w.d_ffn, w.d, w.n_heads
    dh = dm // H
    per = {}
    M = valid_tokens
    per["gemm_ffn1"] = ("flop", 2.0 * M * ff * dm)
    per["gemm_ffn2_ln2"] = ("flop", 2.0 * M * ff * dm)
    per["gemm_qkv"] = ("flop", 2.0 * M * 3 * dm * dm)
    per["gemm_oproj_ln1"] = ("flop", 2.0 * M * dm * dm)
    per["gemm_embed"] = ("flop", 2.0 * M * d * dm)
    per["gemm_pool"] = ("flop", 2.0 * M * dm * dm)
    per["gemm_cand"] = ("flop", 2.0 * total * d * dm)
    T = w.T
    per["attention"] = ("flop", 4.0 * H * dh * total * T * (T + 1) / 2.0)
    # the fused encoder: input projection (token half per token, candidate half per
    # candidate), all layers (causal attention over valid positions) and the head
    Tv = valid_tokens / max(total, 1)
    per["encoder_fused"] = ("flop", 2.0 * valid_tokens * d * dm + 2.0 * total * d * dm
                            + w.n_layers * (2.0 * M * (3 * dm * dm + dm * dm + 2 * ff * dm)
                                            + 4.0 * H * dh * total * Tv * (Tv + 1) / 2.0)
                            + 2.0 * M * dm * dm)
    per["score_bf16"] = ("flop", 2.0 * total * max_len * d)
    per["score_f32"] = ("flop", 2.0 * total * max_len * d)
    # int8 storage: the score rows written dominate (d = 32 codes per row)
    per["score_i8"] = ("byte", 4.0 * total * max_len + max_len * d * w.R + 2.0 * total * d)
    per["topk"] = ("byte", 4.0 * total * max_len)
    out = {}
    for site, (kind, amount) in per.items():
        n = launches_per_step.get(site)
        if n:
            out[site] = (kind, amount / n)
    return out


TRAFFIC_FILES = {"encoder_fused": "encoder_fused_{workload}_traffic.md"}
KERNEL_SOURCES = {"encoder_fused": "paper_2506_02267_amd/csrc/encoder_fused.hip"}


def measured_traffic(site, workload):
    """HBM bytes per launch of `site` from the committed counter summary, or None.

    The summary (profiles/) records FETCH_SIZE + WRITE_SIZE per dispatch scaled by
    a plain copy of known size, and the SHA-256 of the kernel source it was taken
    on; a different source (the kernel changed since) gives None.
    """
    import hashlib
    name = TRAFFIC_FILES.get(site)
    if name is None:
        return None
    path = os.path.join(ROOT, "profiles", name.format(workload=workload))
    src = os.path.join(ROOT, KERNEL_SOURCES[site])
    if not (os.path.exists(path) and os.path.exists(src)):
        return None
    sha = hashlib.sha256(open(src, "rb").read()).hexdigest()
    fields = {}
    for line in open(path):
        if line.startswith("<!-- ") and ":" in line:
            key, val = line[5:].split("-->")[0].split(":", 1)
            fields[key.strip()] = val.strip()
    if fields.get("kernel_sha256") != sha or "hbm_bytes_per_launch" not in fields:
        return None
    return float(fields["hbm_bytes_per_launch"])


def cpu_baseline_select(inp, k):
    """The oracle's NN search, untuned, over every candidate of the workload."""
    import oracle
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count() or 1
    t0 = time.perf_counter()
    oracle.nn_select_batch(inp.seq, inp.cand, inp.cand_offset, k)
    t_sel = time.perf_counter() - t0
    return {"value": inp.total / t_sel, "unit": "candidates/s", "cores": int(threads),
            "kind": "oracle",
            "sample": f"NN search of all {inp.total} candidates ({t_sel:.2f} s), numpy"}


def cpu_baseline(inp, W, k, budget_s):
    """The oracle, untuned, on a bounded sample of the same workload."""
    import oracle
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        threads = os.cpu_count() or 1
    total = inp.total
    T = inp.w.T
    t0 = time.perf_counter()
    idx, _ = oracle.nn_select_batch(inp.seq, inp.cand, inp.cand_offset, k)
    t_sel = time.perf_counter() - t0
    creq = inp.cand_request()
    n, t_enc, chunk = 0, 0.0, 8
    while n < total and (t_enc < budget_s or n == 0):
        ids = np.arange(n, min(total, n + chunk))
        t1 = time.perf_counter()
        tok_emb, tok_act, tok_time, valid = oracle.gather_tokens(inp.seq, inp.rt, creq[ids],
                                                                 idx[ids], T)
        oracle.encode(tok_emb, tok_act, tok_time, valid, inp.cand[ids], W)
        t_enc += time.perf_counter() - t1
        n += ids.size
    per_cand = t_sel / total + t_enc / n
    return {"value": 1.0 / per_cand, "unit": "candidates/s", "cores": int(threads),
            "kind": "oracle",
            "sample": (f"NN select of all {total} candidates ({t_sel:.2f} s) + gather and "
                       f"encode of the first {n} candidates ({t_enc:.2f} s), float64 numpy, "
                       f"scaled per candidate")}


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="single_bf16",
                    help="tiny_f32 | single_bf16 | ragged_bf16 | mixed_bf16 | stress_bf16 | "
                         "select_i8 (the NN search alone over int8 codes)")
    ap.add_argument("--cpu-budget", type=float, default=15.0,
                    help="seconds of oracle encoder work in the CPU baseline sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--graph", action="store_true",
                    help="time replays of one step captured as a HIP graph (the roofline "
                         "figure still comes from an eager pass)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="after the timed region, copy 256 MiB device to device three times "
                         "(a plain copy of known size for scaling memory counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: the path runs on one MI355X and this build has no "
              "multi-GPU mode (candidates would shard across GPUs with no exchange).",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import synth
    from paper_2506_02267_amd import tav2 as T

    w = synth.BY_NAME[args.workload]
    inp = synth.make_inputs(w)
    select_only = w.dtype == "i8"
    W = None if select_only else synth.make_weights(w)
    dt = {"bf16": T.BF16, "i8": T.I8}.get(w.dtype, T.F32)
    seq = T.DeviceSeq.from_host(inp.seq, dt)
    rt = T.DeviceSeq.from_host(inp.rt, dt) if inp.rt is not None else None
    cands = T.DeviceCands.from_host(inp.cand, inp.cand_offset, dt)
    if select_only:
        # one step = tav2_nn_select over the whole batch (outputs and workspace reused)
        out_idx = torch.empty((inp.total, w.k), dtype=torch.int32, device="cuda")
        out_score = torch.empty((inp.total, w.k), dtype=torch.float32, device="cuda")
        ws = T.Workspace(torch.device("cuda"))

        def call():
            T.nn_select(seq, cands, w.k, out_idx, out_score, ws)
    else:
        call = T.SelectEncode(seq, rt, cands, w.k, T.DeviceWeights(W))
    stream = torch.cuda.current_stream()
    total = inp.total
    lengths = inp.seq.length.astype(np.int64)
    per_req_valid = np.minimum(w.k, lengths) + (w.rt_len if inp.rt is not None else 0)
    counts = np.diff(inp.cand_offset)
    valid_tokens = int(np.sum(per_req_valid * counts))

    for _ in range(args.warmup):
        call()
    torch.cuda.synchronize()

    # which kernel dominates: one profiled pass over every launch site
    T.profile_enable(True)
    prof_steps = 3
    for _ in range(prof_steps):
        call()
    torch.cuda.synchronize()
    sites = T.profile_report()
    T.profile_enable(False)
    dominant = max(sites, key=lambda s: sites[s][1])
    launches = {s: c // prof_steps for s, (c, _) in sites.items()}

    # timed region: events only around the dominant kernel's launches
    T.profile_enable(True, dominant)
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(args.steps):
        call()
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    dom = T.profile_report()
    T.profile_enable(False)
    ms = ev0.elapsed_time(ev1)
    if args.graph:
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            call()
        for _ in range(args.warmup):
            graph.replay()
        torch.cuda.synchronize()
        ev0.record(stream)
        for _ in range(args.steps):
            graph.replay()
        ev1.record(stream)
        torch.cuda.synchronize()
        ms = ev0.elapsed_time(ev1)
    ms_per_step = ms / args.steps
    value = total * args.steps / (ms / 1000.0)

    if args.copy_calibration:
        src = torch.empty(64 << 20, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        src.fill_(1.0)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()

    work = site_work(w, total, valid_tokens, int(lengths.max()), launches)
    cnt, dom_ms = dom.get(dominant, (0, 0.0))
    avg_s = dom_ms / max(cnt, 1) / 1000.0
    kind, amount = work.get(dominant, ("flop", 0.0))
    if kind == "flop":
        peak = PEAK_BF16_TFLOPS if w.dtype in ("bf16", "i8") else PEAK_F32_TFLOPS
        achieved = amount / avg_s / 1e12 if avg_s > 0 else 0.0
        roof = {"bound": "mfma" if w.dtype == "bf16" else "alu", "achieved": round(achieved, 2),
                "peak": peak, "unit": "TFLOP/s", "frac": round(achieved / peak, 4),
                "traffic": None}
    else:
        achieved = amount / avg_s / 1e9 if avg_s > 0 else 0.0
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4), "traffic": None}
    roof["traffic"] = measured_traffic(dominant, w.name)
    roof["kernel"] = dominant
    roof["avg_launch_us"] = round(avg_s * 1e6, 2)
    roof["work_per_launch"] = amount

    # stage breakdown for the log (stderr)
    print(f"[bench] {w.name}: {ms_per_step:.3f} ms/step, wall {wall:.2f} s for {args.steps} steps",
          file=sys.stderr)
    for s, (c, t) in sorted(sites.items(), key=lambda kv: -kv[1][1]):
        per_launch = t / max(c, 1)
        extra = ""
        if s in work:
            k_, a_ = work[s]
            extra = (f" {a_ / (per_launch / 1e3) / 1e12:.1f} TFLOP/s" if k_ == "flop"
                     else f" {a_ / (per_launch / 1e3) / 1e9:.0f} GB/s")
        print(f"[bench]   {s:16s} {c // prof_steps:3d}/step {t / prof_steps:9.3f} ms/step"
              f" {per_launch * 1e3:9.1f} us/launch{extra}", file=sys.stderr)

    cpu = None
    if not args.no_cpu_baseline:
        cpu = (cpu_baseline_select(inp, w.k) if select_only
               else cpu_baseline(inp, W, w.k, args.cpu_budget))

    config = {"workload": w.name, "requests": w.R, "L": w.L if w.L else list(w.L_range),
              "d": w.d, "candidates": total, "k": w.k}
    if args.graph:
        config["launch"] = "hip_graph"
    if not select_only:
        config.update({"rt_len": w.rt_len, "T": w.T, "d_model": w.d_model, "heads": w.n_heads,
                       "d_ffn": w.d_ffn, "layers": w.n_layers})
    line = {"metric": METRIC_SELECT if select_only else METRIC, "value": round(value, 1),
            "unit": "candidates/s", "n_gpus": 1,
            "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4),
            "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
            "dtype": "bf16" if w.dtype in ("bf16", "i8") else "f32",
            "data": ("synthetic (seeded int8 codes of random unit rows, 1/8-grid candidates)"
                     if select_only else
                     "synthetic (seeded 1/8-grid embeddings, N(0,0.02) weights)"),
            "config": config, "roofline": roof, "cpu_baseline": cpu}
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
