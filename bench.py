"""Benchmark of the spike-gated INT8 projection on one MI355X.

Headline workload: the 22-block decode stack of the 874M spiking decoder --
per block a TCAM projection 1536 -> 1536 and an FFN down projection
6144 -> 1536, per-block spike rate r_l ~ U[0.05, 0.20], 1000 tokens of fresh
Bernoulli spikes, independent INT8 weights per projection (~260 MB).

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
p99); the single projection and the down-projection rate sweep at batch 1;
the 512-token prefill on the gather and on the matrix cores; the batched
decode stack (64 rows); and the CPU oracle on a bounded sample.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0      # MI355X HBM3E, published
INT8_PEAK_TOPS = 5000.0    # MI355X dense int8 matrix peak, published
DEFAULT_SETS = 32          # rotated weight copies of the decode stack (8.3 GB)
DEFAULT_TOKENS = 1000
METRIC = "active-column INT8 GB/s (% HBM peak) + per-token 22-layer spike-proj latency"
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "k_stream_decode_stack_traffic.json")
# The timed kernel: the stream kernel of gather.hpp at this launch shape
# (16 bytes per lane, 32-lane groups, 4 columns in flight, 256 threads,
# nontemporal loads).  The traffic record is keyed on both.
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2606_03026_amd", "csrc", f) for f in ("gather.hpp", "buffer.hpp")]
HEADLINE_SHAPE = (16, 32, 4, 256, True)


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def kernel_source_hash() -> str:
    """Hash of the device code the headline kernel is built from, and of its launch shape."""
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        h.update(open(p, "rb").read())
    h.update(repr(HEADLINE_SHAPE).encode())
    return h.hexdigest()[:16]


def active_counts(masks: np.ndarray, Ks) -> np.ndarray:
    """|A| per (row, projection) from masks packed projection after projection."""
    from paper_2606_03026_amd import workloads as wl
    out = np.empty((masks.shape[0], len(Ks)), dtype=np.int64)
    off = 0
    for j, K in enumerate(Ks):
        w = wl.words_per_row(K)
        out[:, j] = wl.unpack_bits(masks[:, off:off + w], K).sum(axis=1)
        off += w
    return out


class Timer:
    """HIP events on torch's current stream, which is the stream every
    binding call launches on."""

    def __init__(self, torch):
        self.torch = torch

    def __call__(self, fn, reps: int, warmup: int = 1) -> float:
        torch = self.torch
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(reps):
            fn()
        b.record()
        torch.cuda.synchronize()
        return a.elapsed_time(b) / 1e3 / reps


def graph_of(torch, fn):
    fn()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    return g


def make_handles(sp, torch, host, copies: int, max_B: int = 1):
    """Device weights and handles for (W, scale) pairs, plus `copies` - 1
    address-distinct device copies of all of them.  The first handles hold a
    workspace for max_B rows and the matrix-core copy of W (so that single
    calls take the faster path); the copies only feed streams and are
    gather-only (no second copy of their weights)."""
    dev = [(torch.from_numpy(W).cuda(), torch.from_numpy(s).cuda()) for (W, s) in host]
    base = [sp.spike_proj_create_reserved(W, s, max_B) for (W, s) in dev]
    extra = []
    for _ in range(copies - 1):
        for (W, s) in dev:
            extra.append(sp.spike_proj_create_reserved(W.clone(), s.clone(), 1, gather_only=True))
    return base, extra


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(host, masks, Ks, n_tokens: int, threads: int, passes: int = 5):
    """The oracle, as it stands, on the first n_tokens tokens of the same
    stream: one call per projection over all sampled rows.  Returns the
    median rate over `passes` passes, in active-column GB/s."""
    import oracle
    offs = np.cumsum([0] + [(K + 63) // 64 for K in Ks])
    sample = masks[:n_tokens]
    active_bytes = int(active_counts(sample, Ks).sum()) * host[0][0].shape[1]
    times = []
    for _ in range(passes):
        t0 = time.perf_counter()
        for j, (W, s) in enumerate(host):
            oracle.spike_forward(W, s, sample[:, offs[j]:offs[j + 1]], threads=threads)
        times.append(time.perf_counter() - t0)
    return active_bytes / float(np.median(times)) / 1e9, float(np.median(times))


def bench_decode_stack(sp, torch, wl, timer, args):
    T, R = args.tokens, args.sets
    order = wl.stack_order()
    Ks = [wl.PROJ_SHAPES[j][0] for (_, j) in order]
    N = wl.RESIDUAL
    log(f"decode stack: weights for {len(order)} projections, {T} tokens of spikes, {R} weight sets")
    host = [wl.stack_projection(l, j) for (l, j) in order]
    masks = wl.stack_token_masks(T)
    counts = active_counts(masks, Ks)
    step_bytes = int(counts.sum()) * N
    handles, copies = make_handles(sp, torch, host, R)
    dmasks = torch.from_numpy(masks.view(np.int64)).cuda()
    out = torch.empty((T, len(order) * N), dtype=torch.float32, device="cuda")
    cold = sp.spike_stream_create(handles + copies, len(order), R, T)
    warm = sp.spike_stream_create(handles, len(order), 1, T)
    for st in (cold, warm):
        sp.spike_stream_tune(st, sp.SPIKE_TUNE_SHAPE, sp.SPIKE_SHAPE(*HEADLINE_SHAPE))
    torch.cuda.synchronize()

    sec = timer(lambda: sp.spike_stream_forward(cold, dmasks, out), args.steps, args.warmup)
    gbs = step_bytes / sec / 1e9
    log(f"stream cold: {sec * 1e3:.3f} ms/step, {gbs:.1f} GB/s active-column ({100 * gbs / HBM_PEAK_GBS:.1f}% of HBM)")
    sec_w = timer(lambda: sp.spike_stream_forward(warm, dmasks, out), max(3, args.steps // 2), 1)
    warm_gbs = step_bytes / sec_w / 1e9
    log(f"stream warm (one weight set, {R}x fewer bytes than the cold copies): {warm_gbs:.1f} GB/s")
    # the same stream summing in exact 16-bit partials (paper Sec. 2.3), for comparison
    sp.spike_stream_tune(cold, sp.SPIKE_TUNE_SHAPE, sp.SPIKE_SHAPE(*HEADLINE_SHAPE[:4], NT=True, I16=True))
    sec16 = timer(lambda: sp.spike_stream_forward(cold, dmasks, out), max(3, args.steps // 2), 1)
    sp.spike_stream_tune(cold, sp.SPIKE_TUNE_SHAPE, sp.SPIKE_SHAPE(*HEADLINE_SHAPE))
    i16_gbs = step_bytes / sec16 / 1e9
    log(f"stream cold with 16-bit partial sums: {i16_gbs:.1f} GB/s ({100 * i16_gbs / HBM_PEAK_GBS:.1f}% of HBM)")
    res = {"sec": sec, "gbs": gbs, "warm_gbs": warm_gbs, "i16_gbs": i16_gbs, "step_bytes": step_bytes,
           "host": host, "masks": masks, "Ks": Ks}

    if not args.no_latency:
        static_mask = torch.zeros(masks.shape[1], dtype=torch.int64, device="cuda")
        static_out = torch.zeros(len(order) * N, device="cuda")
        g = graph_of(torch, lambda: sp.spike_stack_forward(handles, static_mask, 1, static_out))
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
        for c0 in range(0, nt, 50):
            torch.cuda._sleep(int(cycles_per_ms * 30))
            for t in range(c0, min(nt, c0 + 50)):
                static_mask.copy_(dmasks[t])
                evs[t][0].record()
                g.replay()
                evs[t][1].record()
        torch.cuda.synchronize()
        skip = min(10, nt - 1)
        lat = np.array([x.elapsed_time(y) * 1e3 for x, y in evs])[skip:]
        tok_bytes = counts[:nt].sum(axis=1)[skip:] * N
        res["latency"] = {"median_us": round(float(np.median(lat)), 2),
                          "p99_us": round(float(np.percentile(lat, 99)), 2), "tokens": int(lat.size),
                          "gbs_median": round(float(np.median(tok_bytes / lat / 1e3)), 1),
                          "mode": "44 batch-1 projections in stream order per token (HIP graph replay), "
                                  "one weight set (260 MB of matrix-core weights, more than the 256 MB "
                                  "Infinity Cache, so each token reads them from HBM)"}
        log(f"per-token latency: median {res['latency']['median_us']} us, p99 {res['latency']['p99_us']} us")
    for s in (cold, warm):
        s.close()
    return res


MALL_BYTES = 256 << 20  # MI355X Infinity Cache


def bench_batch1(sp, torch, timer, name, W, scale, mask_sets, copies: int, warm_sets: int, calls: int):
    """One projection at batch 1, for each (label, rate, masks) of mask_sets:
    mean latency of `calls` dependent calls (graph replay, one weight copy),
    and the stream rate over all masks, cold and warm.  Cold: mask i reads
    copy i % copies, and `copies` is chosen so that the active-column bytes
    read between two uses of a copy exceed the Infinity Cache.  Warm:
    `warm_sets` copies, whose bytes stay in the caches."""
    K, N = W.shape
    handles, extra = make_handles(sp, torch, [(W, scale)], copies)
    all_h = handles + extra
    h = handles[0]
    results = []
    for label, p, masks in mask_sets:
        nm = masks.shape[0]
        counts = active_counts(masks, [K])[:, 0]
        dm = torch.from_numpy(masks.view(np.int64)).cuda()
        out = torch.empty((nm, N), device="cuda")
        n = min(calls, nm)
        g = graph_of(torch, lambda: [sp.spike_proj_forward(h, dm[i], 1, out[i]) for i in range(n)])
        sec = timer(g.replay, 3, 1) / n
        del g
        rates = {}
        for kind, hs in (("cold", all_h), ("warm", all_h[:warm_sets])):
            st = sp.spike_stream_create(hs, 1, len(hs), nm)
            sec_s = timer(lambda: sp.spike_stream_forward(st, dm, out), 5, 1)
            st.close()
            rates[kind] = round(counts.sum() * N / sec_s / 1e9, 1)
        bytes_per = float(counts.mean()) * N
        r = {"K": K, "N": N, "p": p, "active_bytes_mean": round(bytes_per), "call_us": round(sec * 1e6, 2),
             "call_gbs": round(bytes_per / sec / 1e9, 1), "stream_masks": nm, "stream_gbs_cold": rates["cold"],
             "stream_hbm_frac_cold": round(rates["cold"] / HBM_PEAK_GBS, 4), "stream_cold_copies": copies,
             "cold_reuse_distance_bytes": int(bytes_per * copies), "stream_gbs_warm": rates["warm"],
             "stream_warm_copies": warm_sets}
        log(f"{name} {label}: {r['call_us']} us per dependent call ({r['call_gbs']} GB/s); stream over {nm} masks: "
            f"cold {r['stream_gbs_cold']} GB/s ({100 * r['stream_hbm_frac_cold']:.1f}% of HBM), "
            f"warm {r['stream_gbs_warm']} GB/s")
        results.append(r)
    for x in all_h:
        x.close()
    return results


def cold_copies(bytes_per_mask: float, n_masks: int) -> int:
    """Weight copies for a cold stream: the active bytes read between two
    uses of one copy are at least twice the Infinity Cache."""
    return int(min(n_masks, max(32, np.ceil(2 * MALL_BYTES / bytes_per_mask))))


def bench_dense(sp, torch, wl, timer, batches=(1, 2)):
    """The continuous-input projections (row-major INT8 weights, FP32
    activations): attention 1536->1536, FFN up 1536->6144 and the vocabulary
    head 1536->57344.  Per call: `calls` launches in one graph, each on the
    next of `copies` weight copies, with copies * weight bytes >= 2x the
    Infinity Cache, so every call streams its weights from HBM.  Bytes per
    call: weights + scales + activations in + outputs."""
    res = {}
    for kind in wl.DENSE_SHAPES:
        d = wl.dense_projection(kind, B=max(batches))
        M, K = d["Q"].shape
        copies = int(max(1, np.ceil(2 * MALL_BYTES / (M * K))))
        Qs = [torch.from_numpy(d["Q"]).cuda() for _ in range(copies)]
        s = torch.from_numpy(d["scale"]).cuda()
        x = torch.from_numpy(d["x"]).cuda()
        y = torch.empty((max(batches), M), dtype=torch.float32, device="cuda")
        calls = max(copies, 64)
        for B in batches:
            g = graph_of(torch, lambda: [sp.dense_proj_forward(Qs[i % copies], s, x, B, y) for i in range(calls)])
            sec = timer(g.replay, 3, 1) / calls
            del g
            byts = M * K + 4 * M + 4 * B * (K + M)
            plan = sp.dense_proj_plan(K, M, B)
            r = {"K": K, "M": M, "B": B, "bytes_per_call": byts, "call_us": round(sec * 1e6, 2),
                 "gbs": round(byts / sec / 1e9, 1), "hbm_frac": round(byts / sec / 1e9 / HBM_PEAK_GBS, 4),
                 "weight_copies": copies,
                 "kernel": "register" if plan["kernel"] == sp.DENSE_KERNEL_REGISTER else "staged",
                 "launches_per_call": -(-B // plan["rows_per_launch"])}
            log(f"dense {kind} {K}->{M} B={B}: {r['call_us']} us per call, {r['gbs']} GB/s "
                f"({100 * r['hbm_frac']:.1f}% of HBM), {r['kernel']} kernel")
            res[f"{kind}_{K}x{M}_b{B}"] = r
        del Qs
        torch.cuda.empty_cache()
    return res


def bench_quantize(sp, torch, wl, timer):
    """The exporter's symmetric per-channel INT8 quantization on the model's
    largest matrices: FFN down [1536][6144] into the column-major spike
    layout and the vocabulary head [57344][1536] into the row-major dense
    layout.  Algorithmic bytes: W read once (4 B/element), Q written once
    (1 B/element), scales written.  The row-major export of rows of at most
    4096 values runs in one pass (those bytes move); the column-major one
    reads W twice (scale pass, then quantize pass), so 9 B/element move."""
    res = {}
    for name, (M, K), layout in (("down_col", (1536, 6144), sp.SPIKE_LAYOUT_COL_MAJOR),
                                 ("head_row", (wl.VOCAB, 1536), sp.SPIKE_LAYOUT_ROW_MAJOR)):
        rng = np.random.default_rng([42, 14, M, K])
        W = torch.from_numpy(rng.normal(0.0, 0.02, size=(M, K)).astype(np.float32)).cuda()
        Q = torch.empty(M * K, dtype=torch.int8, device="cuda")
        s = torch.empty(M, dtype=torch.float32, device="cuda")
        g = graph_of(torch, lambda: [sp.spike_quantize_int8(W, layout, Q, s) for _ in range(10)])
        sec = timer(g.replay, 3, 1) / 10
        del g
        algo = 5 * M * K + 4 * M
        one_pass = layout == sp.SPIKE_LAYOUT_ROW_MAJOR and K % 4 == 0 and K <= 4096
        moved = (5 if one_pass else 9) * M * K + 4 * M
        r = {"M": M, "K": K, "layout": "col" if layout == sp.SPIKE_LAYOUT_COL_MAJOR else "row",
             "passes": 1 if one_pass else 2,
             "call_us": round(sec * 1e6, 2), "algorithmic_gbs": round(algo / sec / 1e9, 1),
             "moved_gbs": round(moved / sec / 1e9, 1), "hbm_frac_moved": round(moved / sec / 1e9 / HBM_PEAK_GBS, 4)}
        log(f"quantize {name} [{M}][{K}]: {r['call_us']} us, {r['algorithmic_gbs']} GB/s algorithmic, "
            f"{r['moved_gbs']} GB/s moved ({100 * r['hbm_frac_moved']:.1f}% of HBM)")
        res[name] = r
        del W, Q, s
        torch.cuda.empty_cache()
    return res


def bench_head_verify(sp, torch, wl, timer):
    """The vocabulary head 1536 -> 57,344 with candidate verification (paper
    Sec. 5): INT8-activation head over all rows + top-K selection, gate and
    FP32 recompute of K rows, per token, against the FP32-activation dense
    head over all rows (the paper's baseline configuration).  Cold weights:
    calls rotate over copies whose bytes exceed 2x the Infinity Cache."""
    d = wl.dense_projection("head", B=1)
    V, K = d["Q"].shape
    copies = int(max(1, np.ceil(2 * MALL_BYTES / (V * K))))
    Qs = [torch.from_numpy(d["Q"]).cuda() for _ in range(copies)]
    s = torch.from_numpy(d["scale"]).cuda()
    x = torch.from_numpy(d["x"][0]).cuda()
    logits = torch.empty(V, dtype=torch.float32, device="cuda")
    cand = torch.empty(64, dtype=torch.int32, device="cuda")
    cl = torch.empty(64, dtype=torch.float32, device="cuda")
    res = torch.empty(2, dtype=torch.int32, device="cuda")
    calls = max(copies, 64)
    out = {"V": V, "K": K, "weight_copies": copies}
    for k, thr, label in ((64, float("inf"), "k64_always_verify"), (64, 0.0, "k64_never_verify"),
                          (16, 0.5, "k16_gate_0.5")):
        g = graph_of(torch, lambda: [sp.head_verify_forward(Qs[i % copies], s, x, k, thr, logits, cand, cl, res)
                                     for i in range(calls)])
        sec = timer(g.replay, 3, 1) / calls
        del g
        out[label] = {"call_us": round(sec * 1e6, 2),
                      "weight_gbs": round(V * K / sec / 1e9, 1),
                      "hbm_frac": round(V * K / sec / 1e9 / HBM_PEAK_GBS, 4)}
        log(f"head verify {label}: {out[label]['call_us']} us per token ({out[label]['weight_gbs']} GB/s of weights)")
    y = torch.empty((1, V), dtype=torch.float32, device="cuda")
    xb = x.view(1, K)
    g = graph_of(torch, lambda: [sp.dense_proj_forward(Qs[i % copies], s, xb, 1, y) for i in range(calls)])
    out["fp32_activation_head_us"] = round(timer(g.replay, 3, 1) / calls * 1e6, 2)
    del g, Qs
    torch.cuda.empty_cache()
    log(f"head with FP32 activations (dense kernel): {out['fp32_activation_head_us']} us per token")
    return out


def write_traffic_record(fetch_csv: str, write_csv: str, steps: int, warmup: int, tokens: int) -> int:
    """Assemble the HBM-traffic record of the headline stream kernel from two
    rocprofv3 --pmc runs of `bench.py --only-stream --copy-probe` (one with
    FETCH_SIZE, one with WRITE_SIZE; KiB per dispatch).  Each counter is
    scaled by what it reads for the 1 GiB copy of --copy-probe.  Of the
    headline shape's stream dispatches, the first warmup + steps are the cold
    (rotated-copies) ones and the rest the warm (one weight set) ones."""
    import csv
    from paper_2606_03026_amd import workloads as wl

    V, LG, U, BLOCK, NT = HEADLINE_SHAPE
    headline = f"spk::k_stream<spk::Shape<{V}, {LG}, {U}, {BLOCK}, {str(NT).lower()}, false>"

    def rows(path, counter):
        out = [r for r in csv.DictReader(open(path)) if r["Counter_Name"] == counter]
        out.sort(key=lambda r: int(r["Dispatch_Id"]))
        copy = max((r for r in out if r["Kernel_Name"].startswith("__amd_rocclr_copyBuffer")),
                   key=lambda r: float(r["Counter_Value"]))
        stream = [float(r["Counter_Value"]) for r in out if headline in r["Kernel_Name"]]
        return float(copy["Counter_Value"]), stream

    gib_kib = float(1 << 20)
    f_copy, fetch = rows(fetch_csv, "FETCH_SIZE")
    w_copy, write = rows(write_csv, "WRITE_SIZE")
    n_cold = warmup + steps
    f_scale, w_scale = gib_kib / f_copy, gib_kib / w_copy
    fetch_bytes = float(np.mean(fetch[:n_cold])) * 1024 * f_scale
    write_bytes = float(np.mean(write[:n_cold])) * 1024 * w_scale
    order = wl.stack_order()
    Ks = [wl.PROJ_SHAPES[j][0] for (_, j) in order]
    algo = int(active_counts(wl.stack_token_masks(tokens), Ks).sum()) * wl.RESIDUAL
    cmd = ("rocprofv3 --pmc {c} -d gpurun_out/pmc_{c} -o pmc --output-format csv -- python3 -u bench.py "
           f"--only-stream --copy-probe --steps {steps} --warmup {warmup} --no-cpu")
    rec = {
        "kernel": f"k_stream<Shape{HEADLINE_SHAPE}, buffer loads> on the {tokens}-token 22-block decode stream",
        "kernel_source_hash": kernel_source_hash(),
        "command_fetch": cmd.format(c="FETCH_SIZE"),
        "command_write": cmd.format(c="WRITE_SIZE"),
        "command_record": (f"python3 bench.py --traffic-record gpurun_out/pmc_FETCH_SIZE/pmc_counter_collection.csv "
                           f"gpurun_out/pmc_WRITE_SIZE/pmc_counter_collection.csv --steps {steps} --warmup {warmup}"),
        "calibration": {"kernel": "__amd_rocclr_copyBuffer, 1 GiB read + 1 GiB written (bench.py --copy-probe)",
                        "fetch_kib": f_copy, "write_kib": w_copy,
                        "fetch_scale": round(f_scale, 4), "write_scale": round(w_scale, 4)},
        "raw_kib_per_launch": {"fetch_cold": [round(v, 1) for v in fetch[:n_cold]],
                               "fetch_warm": [round(v, 1) for v in fetch[n_cold:]],
                               "write": [round(v, 1) for v in write]},
        "fetch_bytes_per_launch": round(fetch_bytes),
        "write_bytes_per_launch": round(write_bytes),
        "hbm_bytes_per_launch": round(fetch_bytes + write_bytes),
        "algorithmic_active_bytes_per_launch": algo,
        "fetch_over_algorithmic": round(fetch_bytes / algo, 4),
    }
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(rec, f, indent=1)
    print(json.dumps({k: rec[k] for k in ("hbm_bytes_per_launch", "fetch_over_algorithmic", "kernel_source_hash")}))
    return 0


def bench_prefill(sp, torch, wl, timer):
    d = wl.prefill_projection()
    B, K, N = d["masks"].shape[0], d["K"], d["N"]
    h = make_handles(sp, torch, [(d["W"], d["scale"])], 1, max_B=B)[0][0]
    dm = torch.from_numpy(d["masks"].view(np.int64)).cuda()
    out = torch.empty((B, N), device="cuda")
    r = {"B": B, "K": K, "N": N}
    for name, path in (("gather", sp.SPIKE_PATH_GATHER), ("mfma", sp.SPIKE_PATH_MFMA)):
        sp.spike_proj_tune(h, sp.SPIKE_TUNE_PATH, path)
        sec = timer(lambda: sp.spike_proj_forward(h, dm, B, out), 20, 2)
        r[f"{name}_us"] = round(sec * 1e6, 2)
    ops = 2.0 * B * K * N
    r["mfma_tops"] = round(ops / (r["mfma_us"] * 1e-6) / 1e12, 1)
    r["mfma_util"] = round(r["mfma_tops"] / INT8_PEAK_TOPS, 4)
    r["speedup_mfma_vs_gather"] = round(r["gather_us"] / r["mfma_us"], 2)
    log(f"prefill 512x6144->1536: gather {r['gather_us']} us, matrix cores {r['mfma_us']} us "
        f"({r['mfma_tops']} TOPS dense, {100 * r['mfma_util']:.1f}% of int8 peak)")
    return r


def bench_batched_stack(sp, torch, wl, timer, steps: int = 16, B: int = 64):
    """B = 64 rows through the 22-block stack for `steps` decode steps of
    structured spikes.  All steps are captured in one graph (each step reads
    its own masks), replayed, and the time divided by the steps: one fused
    matrix-core launch per step, 44 launches per step in stream order on the
    matrix cores, and the same on the gather."""
    order = wl.stack_order()
    host = [wl.batched_stack_projection(l, j) for (l, j) in order]
    bits = [wl.batched_stack_bits(l, j, B=B, n_steps=steps) for (l, j) in order]
    handles = make_handles(sp, torch, host, 1, max_B=B)[0]
    per_step = [np.concatenate([wl.pack_bits(b[s]).reshape(-1) for b in bits]) for s in range(steps)]
    union = sum(int(b.any(axis=1).sum(axis=1).mean()) * 1536 for b in bits)  # mean union columns per step
    dm = [torch.from_numpy(m.view(np.int64)).cuda() for m in per_step]
    out = torch.empty(sum(B * h.N for h in handles), device="cuda")
    r = {"B": B, "steps": steps, "union_bytes_per_step": union}
    for name, path, fn in (("fused", sp.SPIKE_PATH_AUTO, sp.spike_stack_forward_fused),
                           ("mfma", sp.SPIKE_PATH_AUTO, sp.spike_stack_forward),
                           ("gather", sp.SPIKE_PATH_GATHER, sp.spike_stack_forward)):
        for h in handles:
            sp.spike_proj_tune(h, sp.SPIKE_TUNE_PATH, path)
        g = graph_of(torch, lambda: [fn(handles, dm[s], B, out) for s in range(steps)])
        t = timer(g.replay, 5, 1) / steps
        del g
        r[f"{name}_step_us"] = round(t * 1e6, 1)
        r[f"{name}_union_gbs"] = round(union / t / 1e9, 1)
    r["mfma_tops_fused"] = round(sum(2.0 * B * h.K * h.N for h in handles) / (r["fused_step_us"] * 1e-6) / 1e12, 1)
    log(f"batched stack B={B}: one fused matrix-core launch per step {r['fused_step_us']} us/step "
        f"({r['fused_union_gbs']} GB/s on union bytes, {r['mfma_tops_fused']} dense TOPS); in stream order "
        f"(44 launches): matrix cores {r['mfma_step_us']} us/step, gather {r['gather_step_us']} us/step")
    return r


def crossover_sweep(sp, torch, timer):
    """Per-call time of the gather and of the matrix cores over K in {1536,
    6144}, spike rate p and batch B (N = 1536): each cell is 20 dependent
    calls captured in one graph, replayed 5 times.  Prints one JSON row per
    cell; the data behind the automatic path choice."""
    from paper_2606_03026_amd import workloads as wl
    rows = []
    for K in (1536, 6144):
        N = 1536
        rng = np.random.default_rng([42, 7, K])
        W = rng.integers(-127, 127, size=(K, N), dtype=np.int8, endpoint=True)
        s = rng.uniform(1e-3, 1e-2, N).astype(np.float32)
        h = make_handles(sp, torch, [(W, s)], 1, max_B=512)[0][0]
        for p in (0.02, 0.05, 0.10, 0.20, 0.40):
            for B in (1, 2, 3, 4, 5, 6, 8, 12, 16, 24, 32, 64, 128, 256, 512):
                bits = rng.random((B, K)) < p
                dm = torch.from_numpy(wl.pack_bits(bits).view(np.int64)).cuda()
                out = torch.empty((B, N), device="cuda")
                t = {}
                for name, path in (("gather", sp.SPIKE_PATH_GATHER), ("mfma", sp.SPIKE_PATH_MFMA)):
                    sp.spike_proj_tune(h, sp.SPIKE_TUNE_PATH, path)
                    g = graph_of(torch, lambda: [sp.spike_proj_forward(h, dm, B, out) for _ in range(20)])
                    t[name] = timer(g.replay, 5, 1) / 20
                    del g
                rows.append({"K": K, "N": N, "p": p, "B": B, "gather_us": round(t["gather"] * 1e6, 2),
                             "mfma_us": round(t["mfma"] * 1e6, 2)})
                print(json.dumps(rows[-1]), flush=True)
        h.close()
    return rows


def traffic_record():
    """HBM bytes per stream launch from the committed rocprofv3 PMC summary,
    if it was taken on the current kernel sources."""
    try:
        rec = json.load(open(TRAFFIC_FILE))
    except (OSError, ValueError):
        return None
    if rec.get("kernel_source_hash") != kernel_source_hash():
        return None
    return rec


def main(argv=None) -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--tokens", type=int, default=DEFAULT_TOKENS)
    ap.add_argument("--sets", type=int, default=DEFAULT_SETS)
    ap.add_argument("--latency-tokens", type=int, default=1000)
    ap.add_argument("--batch1-masks", type=int, default=8000, help="masks per batch-1 stream (configs 1-2)")
    ap.add_argument("--cpu-tokens", type=int, default=100, help="tokens of the stream in the CPU-baseline sample")
    ap.add_argument("--no-cpu", action="store_true")
    ap.add_argument("--no-latency", action="store_true")
    ap.add_argument("--only-stream", action="store_true", help="time only the headline stream (for profiling)")
    ap.add_argument("--crossover", action="store_true",
                    help="only the per-call gather vs matrix-core sweep over (K, p, B), one JSON row per cell")
    ap.add_argument("--only-mfma", action="store_true",
                    help="time only the matrix-core workloads, prefill and batched stack (for profiling)")
    ap.add_argument("--copy-probe", action="store_true",
                    help="run a 1 GiB device copy first (reference for the PMC byte counters)")
    ap.add_argument("--only-dense", action="store_true",
                    help="time only the continuous-input projections, the quantizer and the head verification "
                         "(for profiling)")
    ap.add_argument("--traffic-record", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="write the stream kernel's HBM-traffic record from two rocprofv3 --pmc CSVs (no GPU)")
    args = ap.parse_args(argv)

    if args.traffic_record:
        return write_traffic_record(*args.traffic_record, args.steps, args.warmup, args.tokens)

    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the projection shards without communication per output-channel range, but no "
              "multi-GPU path is implemented)", file=sys.stderr)
        return 2

    import torch
    from paper_2606_03026_amd import _binding as sp
    from paper_2606_03026_amd import workloads as wl

    torch.cuda.set_device(0)
    timer = Timer(torch)
    if args.copy_probe:
        src = torch.ones(1 << 28, dtype=torch.int32, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        log("copy probe: 1 GiB read + 1 GiB written")
        del src, dst

    if args.crossover:
        crossover_sweep(sp, torch, timer)
        return 0
    if args.only_mfma:
        res = {"prefill_512x6144x1536": bench_prefill(sp, torch, wl, timer),
               "batched_stack_b64": bench_batched_stack(sp, torch, wl, timer)}
        print(json.dumps({"workloads": res}), flush=True)
        return 0
    if args.only_dense:
        print(json.dumps({"workloads": {"dense": bench_dense(sp, torch, wl, timer),
                                        "quantize": bench_quantize(sp, torch, wl, timer),
                                        "head_verify": bench_head_verify(sp, torch, wl, timer)}}), flush=True)
        return 0
    if args.only_stream:
        args.no_latency = True
    main_res = bench_decode_stack(sp, torch, wl, timer, args)
    gbs = main_res["gbs"]

    extra = {}
    if not args.only_stream:
        nm = args.batch1_masks
        d = wl.single_projection(n_masks=nm)
        copies = cold_copies(0.10 * d["K"] * d["N"], nm)
        extra["single_1536x1536_b1"] = bench_batch1(sp, torch, timer, "1536x1536", d["W"], d["scale"],
                                                    [("p=0.10", d["p"], d["masks"])], copies, 32, 1000)[0]
        downs = [wl.down_sweep(p, n_masks=nm) for p in wl.DOWN_SWEEP_RATES]
        copies = cold_copies(min(wl.DOWN_SWEEP_RATES) * downs[0]["K"] * downs[0]["N"], nm)
        extra["down_6144x1536_b1"] = bench_batch1(sp, torch, timer, "6144x1536", downs[0]["W"], downs[0]["scale"],
                                                  [(f"p={x['p']}", x["p"], x["masks"]) for x in downs], copies, 32,
                                                  200)
        del downs
        extra["prefill_512x6144x1536"] = bench_prefill(sp, torch, wl, timer)
        extra["batched_stack_b64"] = bench_batched_stack(sp, torch, wl, timer)
        extra["dense"] = bench_dense(sp, torch, wl, timer)
        extra["quantize"] = bench_quantize(sp, torch, wl, timer)
        extra["head_verify"] = bench_head_verify(sp, torch, wl, timer)

    cpu = None
    if not args.no_cpu:
        affinity = len(os.sched_getaffinity(0))
        threads = min(affinity, 16)  # at most the 16 host cores that serve one GPU
        host, masks, Ks = main_res["host"], main_res["masks"], main_res["Ks"]
        nt = args.cpu_tokens
        v1, t1 = cpu_baseline(host, masks, Ks, nt, 1)
        vn, tn = cpu_baseline(host, masks, Ks, nt, threads)
        best_multi = vn >= v1
        cpu = {"value": round(max(v1, vn), 3), "unit": "GB/s", "cores": threads if best_multi else 1,
               "kind": "oracle",
               "sample": (f"first {nt} tokens x 44 projections of the same stream, one oracle call per projection "
                          f"over the {nt} rows, median of 5 passes; 1 thread: {v1:.3f} GB/s ({t1:.2f} s per pass), "
                          f"{threads} threads: {vn:.3f} GB/s ({tn:.2f} s per pass); host CPU {cpu_model()}, "
                          f"{affinity} cores in the process affinity mask")}
        log(f"cpu oracle: {v1:.3f} GB/s on 1 thread, {vn:.3f} GB/s on {threads} ({cpu_model()})")

    traffic = traffic_record()
    rec = {
        "metric": METRIC,
        "value": round(gbs, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(main_res["sec"] * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int8",
        "data": "synthetic",
        "config": {"workload": "22-block decode stack, TCAM 1536->1536 + FFN down 6144->1536 per block, "
                               f"batch-1 per token, {args.tokens} tokens, rate U[0.05,0.20] per block, "
                               f"independent-token stream over {args.sets} rotated weight copies",
                   "tokens": args.tokens, "projections_per_token": 44, "weight_sets": args.sets,
                   "active_bytes_per_step": main_res["step_bytes"]},
        "hbm_pct": round(100 * gbs / HBM_PEAK_GBS, 2),
        "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(gbs / HBM_PEAK_GBS, 4),
                     "traffic": None if traffic is None else traffic["hbm_bytes_per_launch"],
                     "kernel": f"k_stream<Shape{HEADLINE_SHAPE}> (one launch per step)",
                     "kernel_source_hash": kernel_source_hash()},
        "warm_one_set_gbs": round(main_res["warm_gbs"], 1),
        "int16_partials_cold_gbs": round(main_res["i16_gbs"], 1),
        "per_token_latency": main_res.get("latency"),
        "workloads": extra,
        "cpu_baseline": cpu,
    }
    print(json.dumps(rec), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
