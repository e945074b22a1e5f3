"""Benchmark of the spike-gated INT8 projection on one MI355X.

Workload (default): the 22-block decode stack of the 874M spiking decoder --
per block a TCAM projection 1536 -> 1536 and an FFN down projection
6144 -> 1536, per-block spike rate r_l ~ U[0.05, 0.20], 1000 tokens of
fresh Bernoulli spikes, independent INT8 weights per projection (~260 MB).

A step is one pass of the whole 1000-token stream through all 44
projections: one launch of the stream kernel, in which every (token,
projection) pair is an independent batch-1 projection (compaction, active-
column gather, INT32 sums, one FP32 scale per output).  Tokens rotate over
DEFAULT_SETS address-distinct copies of the weights so that a column read by
one token is not still cached when the next token on the same copy reads it:
the figure is HBM bandwidth, not cache bandwidth (a one-copy "warm" figure is
reported beside it).

Headline value: active-column INT8 bytes per second (sum over tokens and
projections of |A| * N bytes, the only weight bytes the method needs),
against the MI355X HBM peak of 8 TB/s.  Also reported: the per-token
latency of the 44 projections run in stream order (graph replay, median and
p99), and the CPU oracle on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0      # MI355X HBM3E, published
DEFAULT_SETS = 32          # rotated weight copies (8.3 GB)
DEFAULT_TOKENS = 1000
METRIC = "active-column INT8 GB/s (% HBM peak) + per-token 22-layer spike-proj latency"


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def active_bytes(masks: np.ndarray, Ks, N: int) -> np.ndarray:
    """|A| * N per (token, projection) from the packed masks."""
    from paper_2606_03026_amd import workloads as wl
    out = np.empty((masks.shape[0], len(Ks)), dtype=np.int64)
    off = 0
    for j, K in enumerate(Ks):
        w = wl.words_per_row(K)
        bits = wl.unpack_bits(masks[:, off:off + w], K)
        out[:, j] = bits.sum(axis=1) * N
        off += w
    return out


def cpu_baseline(host, masks, Ks, budget_s: float, threads: int):
    """The oracle, as it stands, on the first tokens of the same stream until
    about budget_s seconds of CPU work are done."""
    import oracle
    offs = np.cumsum([0] + [(K + 63) // 64 for K in Ks])
    done_bytes, t0, tokens = 0, time.perf_counter(), 0
    for t in range(masks.shape[0]):
        for j, (W, s) in enumerate(host):
            m = masks[t:t + 1, offs[j]:offs[j + 1]]
            oracle.spike_forward(W, s, m, threads=threads)
            done_bytes += int(np.unpackbits(m.view(np.uint8), bitorder="little")[:Ks[j]].sum()) * W.shape[1]
        tokens += 1
        if time.perf_counter() - t0 >= budget_s:
            break
    el = time.perf_counter() - t0
    return done_bytes / el / 1e9, tokens, el


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--tokens", type=int, default=DEFAULT_TOKENS)
    ap.add_argument("--sets", type=int, default=DEFAULT_SETS)
    ap.add_argument("--latency-tokens", type=int, default=1000)
    ap.add_argument("--cpu-budget", type=float, default=8.0, help="seconds per CPU-baseline leg")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-latency", action="store_true")
    args = ap.parse_args(argv)

    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported by this build "
              "(the projection shards without communication per output-channel range, but no "
              "multi-GPU path is built)", file=sys.stderr)
        return 2

    import torch
    from paper_2606_03026_amd import _binding as sp
    from paper_2606_03026_amd import workloads as wl

    torch.cuda.set_device(0)
    T, R = args.tokens, args.sets
    order = wl.stack_order()
    Ks = [wl.PROJ_SHAPES[j][0] for (_, j) in order]
    N = wl.RESIDUAL

    log(f"generating weights for {len(order)} projections and {T} tokens of spikes")
    host = [wl.stack_projection(l, j) for (l, j) in order]
    masks = wl.stack_token_masks(T)
    ab = active_bytes(masks, Ks, N)
    step_bytes = int(ab.sum())

    dev_w = [(torch.from_numpy(W).cuda(), torch.from_numpy(s).cuda()) for (W, s) in host]
    handles = [sp.spike_proj_create(W, s) for (W, s) in dev_w]
    copies = []
    for _ in range(R - 1):
        for (W, s) in dev_w:
            Wc, sc = W.clone(), s.clone()
            h = sp.spike_proj_create(Wc, sc)
            sp.spike_proj_reserve(h, 1)
            copies.append(h)
    dmasks = torch.from_numpy(masks.view(np.int64)).cuda()
    out = torch.empty((T, len(order) * N), dtype=torch.float32, device="cuda")
    stream_cold = sp.spike_stream_create(handles + copies, len(order), R, T)
    stream_warm = sp.spike_stream_create(handles, len(order), 1, T)
    torch.cuda.synchronize()
    log(f"weights resident: {R} sets x {sum(W.numel() for W, _ in dev_w) / 1e6:.1f} MB; "
        f"active bytes per step {step_bytes / 1e9:.3f} GB")

    def timed(stream_handle, steps, warmup):
        for _ in range(warmup):
            sp.spike_stream_forward(stream_handle, dmasks, out)
        torch.cuda.synchronize()
        start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        start.record()
        for _ in range(steps):
            sp.spike_stream_forward(stream_handle, dmasks, out)
        end.record()
        torch.cuda.synchronize()
        return start.elapsed_time(end) / 1e3

    el = timed(stream_cold, args.steps, args.warmup)
    ms_per_step = el / args.steps * 1e3
    gbs = step_bytes * args.steps / el / 1e9
    log(f"stream (cold, {R} sets): {ms_per_step:.3f} ms/step, {gbs:.1f} GB/s active-column")
    el_w = timed(stream_warm, max(3, args.steps // 2), 1)
    warm_gbs = step_bytes * max(3, args.steps // 2) / el_w / 1e9
    log(f"stream (warm, 1 set): {warm_gbs:.1f} GB/s")

    latency = None
    if not args.no_latency:
        words = masks.shape[1]
        static_mask = torch.zeros(words, dtype=torch.int64, device="cuda")
        static_out = torch.zeros(len(order) * N, device="cuda")
        sp.spike_stack_forward(handles, static_mask, 1, static_out)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            sp.spike_stack_forward(handles, static_mask, 1, static_out)
        nt = min(args.latency_tokens, T)
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(nt)]
        # Keep the device behind the host: a spin kernel at the head of every
        # chunk covers the time the host needs to enqueue the chunk, so no
        # token's start event can run ahead of its graph launch.
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        torch.cuda._sleep(1_000_000)
        b.record()
        torch.cuda.synchronize()
        cycles_per_ms = 1_000_000 / max(a.elapsed_time(b), 1e-3)
        chunk = 50
        for c0 in range(0, nt, chunk):
            torch.cuda._sleep(int(cycles_per_ms * 30))
            for t in range(c0, min(nt, c0 + chunk)):
                static_mask.copy_(dmasks[t])
                evs[t][0].record()
                g.replay()
                evs[t][1].record()
        torch.cuda.synchronize()
        lat = np.array([a.elapsed_time(b) * 1e3 for a, b in evs])[min(10, nt - 1):]
        lat_bytes = ab[:nt].sum(axis=1)[min(10, nt - 1):]
        latency = {"median_us": round(float(np.median(lat)), 2), "p99_us": round(float(np.percentile(lat, 99)), 2),
                   "tokens": int(lat.size), "gbs_median": round(float(np.median(lat_bytes / lat / 1e3)), 1),
                   "mode": "44 projections in stream order per token, graph replay, warm weights"}
        log(f"per-token latency: median {latency['median_us']} us, p99 {latency['p99_us']} us")

    cpu = None
    if not args.no_cpu:
        cores = min(len(os.sched_getaffinity(0)), 16)
        v1, tok1, el1 = cpu_baseline(host, masks, Ks, args.cpu_budget, 1)
        vn, tokn, eln = cpu_baseline(host, masks, Ks, args.cpu_budget, cores)
        cpu = {"value": round(vn, 3), "unit": "GB/s", "cores": cores, "kind": "oracle",
               "sample": f"first {tokn} tokens x 44 projections of the same stream ({eln:.1f} s)",
               "single_thread": {"value": round(v1, 3), "sample_tokens": tok1, "seconds": round(el1, 1)}}
        log(f"cpu oracle: {v1:.2f} GB/s on 1 thread, {vn:.2f} GB/s on {cores}")

    rec = {
        "metric": METRIC,
        "value": round(gbs, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int8",
        "data": "synthetic",
        "config": {"workload": "22-block decode stack, TCAM 1536->1536 + FFN down 6144->1536 per block, "
                               f"batch-1 per token, {T} tokens, rate U[0.05,0.20] per block, "
                               f"independent-token stream over {R} rotated weight copies",
                   "tokens": T, "projections_per_token": len(order), "weight_sets": R,
                   "active_bytes_per_step": step_bytes},
        "hbm_pct": round(100 * gbs / HBM_PEAK_GBS, 2),
        "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": None,
                     "kernel": "k_stream (one launch per step)"},
        "warm_gbs": round(warm_gbs, 1),
        "per_token_latency": latency,
        "cpu_baseline": cpu,
    }
    print(json.dumps(rec), flush=True)
    for s in (stream_cold, stream_warm):
        s.close()
    return 0


if __name__ == "__main__":
    sys.exit(main())
