"""Benchmark of the fused S^4R decode step on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload llama8b_128k] [--gpus 1] [--no-extra]

A step is one call of s4r_decode_step: one layer, all heads, the whole batch
(latent scoring of every cached token, top-k selection, sparse
reconstruction with RoPE, attention).  The main line is the Llama-3.1-8B-shaped
layer at 128k context (B=4, 32/8 heads, d_h=128, rank 160, 4 sinks, window
128, top-k 2048, bf16 storage), seeded synthetic data drawn in latent
coordinates (workloads.latent_state), inputs resident in HBM.  The same run
then measures every other workload and reports each under "configs": the tiny
fp32 layer, the Llama 32k layer at batch 1, the Qwen2.5-7B-shaped 128k layer
at batch 8, the paper's efficiency setting (Qwen3-4B shape at 120k, W = W_q =
4, k = 0.2 L - W, with its dense and full-reconstruction comparators) and the
32-layer sustained run (16 warm-up + 256 timed steps, the new token appended
in every layer).

Timing: W untimed steps, then K timed steps between two device
synchronisations, measured with HIP events on the launch stream.  Steps
rotate over independent copies of the coefficient caches (at least 4, and at
least three times the 256 MB Infinity Cache in total) so that no step finds
its coefficients in that cache.  A second pass with the library's per-kernel
event hook gives the average duration of each kernel; the latent-score stream
over C^K is the roofline entry.  The CPU oracle is timed on a bounded sample
(one sequence of the same workload, repeated for ~10 s; ~5 s for the other
workloads) for the cpu_baseline entries.

Prints ONE JSON line on stdout.
"""

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0          # MI355X HBM3E
BF16_PEAK_TFLOPS = 2500.0       # MI355X dense bf16 MFMA
N_REPLICAS = 4
SHAPES = {"llama8b_32k": "Llama-3.1-8B-shaped", "llama8b_128k": "Llama-3.1-8B-shaped",
          "qwen7b_128k": "Qwen2.5-7B-shaped", "qwen3_4b_120k": "Qwen3-4B-shaped (the paper's efficiency setting)",
          "qwen3_4b_120k_w32": "Qwen3-4B-shaped (the paper's default W = W_q = 32)",
          "tiny_fp32": "tiny"}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def algorithmic(wl, m, windowed=False):
    """Bytes the method must move per step and MFMA flops of the reconstruction
    (windowed: the older query rows' softmax read from the window state and
    the newest row's written, instead of their coefficient rows; above five
    rows their fp64 running sum read and written and the leaving row read)."""
    B, L, R, Dp, es = wl.batch, wl.L, wl.R, wl.Dp, (2 if wl.dtype == "bf16" else 4)
    ck = B * L * R * es                       # C^K streamed once (latent scoring)
    gather = 2 * B * m * R * es               # selected rows of C^K and C^V
    bases = 2 * B * Dp * R * es               # B^K and B^V
    sinks = 2 * B * wl.n_sink * Dp * es
    q = B * wl.n_q_heads * wl.head_dim * es
    out = B * wl.n_q_heads * wl.head_dim * 4
    qwin = B * wl.G * (wl.q_window - 1) * R * 4  # the window's earlier query coefficients (fp32)
    if windowed and wl.q_window > 5:
        qwin = B * wl.G * L * 24                   # running sum read and written (fp64), leaving row read, newest written
    elif windowed:
        qwin = B * wl.G * wl.q_window * L * 4     # older rows' softmax read, the newest row's written
    rec_flops = 2 * 2 * B * m * R * Dp        # K^ and V^ of every selected token
    return {"step_bytes": ck + gather + bases + sinks + q + out + qwin, "stream_bytes": ck, "rec_flops": rec_flops}


STREAM_SOURCES = ("stream.hip", "s4r_device.h", "s4r_internal.h")


def stream_kernel_sha():
    """Hash of the sources the latent-score stream kernel is compiled from."""
    h = hashlib.sha256()
    for f in STREAM_SOURCES:
        h.update(open(os.path.join(ROOT, "paper_2608_00528_amd", "csrc", f), "rb").read())
    return h.hexdigest()[:16]


def traffic_from_profile(workload):
    """HBM bytes per launch of the stream kernel from the committed rocprofv3
    counter summary, or None when it is absent or the kernel source changed."""
    path = os.path.join(ROOT, "profiles", f"score_stream_{workload}_traffic.txt")
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    if kv.get("kernel_source_sha256_16") != stream_kernel_sha():
        return None
    try:
        return float(kv["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def cpu_baseline(wl, st, budget_s=10.0, one_thread=True):
    """The oracle as it stands (numpy with its default BLAS threads) on one
    sequence of the workload, repeated for about budget_s seconds (and, with
    one_thread, again with one BLAS thread for half as long)."""
    from threadpoolctl import threadpool_info

    from oracle import decode
    cfg = dict(n_kv_heads=wl.n_kv_heads, window=wl.window, topk=wl.topk, pool_kernel=wl.pool_kernel,
               pool_mode=wl.pool_mode, group_agg=wl.group_agg, rope_theta=wl.rope_theta, dtype=wl.dtype)
    one = {k: st[k][:1] for k in ("q", "sink_k", "sink_v", "bases_k", "bases_v", "coef_k", "coef_v")}
    qwin = None if st.get("qwin_prev") is None else st["qwin_prev"][:1]
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    times = []
    t_end = time.perf_counter() + budget_s
    while True:
        t0 = time.perf_counter()
        decode.decode_step(cfg, wl.L, one["q"], one["sink_k"], one["sink_v"], one["bases_k"], one["bases_v"],
                           one["coef_k"], one["coef_v"], qwin_prev=qwin)
        times.append(time.perf_counter() - t0)
        if time.perf_counter() > t_end:
            break
    per_seq = float(np.median(times))
    src = ("one sequence of the same shape drawn on the host in latent coordinates (the oracle never reads a "
           "GPU-built state; its time does not depend on the values)" if wl.recipe == "raw"
           else f"sequence 0 of the {wl.name} workload (1 of {wl.batch})")
    sample = (f"float64 numpy oracle, {src}, {len(times)} runs in {sum(times):.1f} s, median per sequence x "
              f"{wl.batch} sequences; BLAS threads {threads}")
    res = {"value": round(per_seq * wl.batch * 1e6, 1), "unit": "us/step", "cores": threads, "kind": "oracle",
           "host_cpus": os.cpu_count(), "sample": sample}
    if not one_thread:
        return res
    # the same sample with one BLAS thread, for about half the budget
    from threadpoolctl import threadpool_limits
    times1 = []
    with threadpool_limits(limits=1):
        t_end = time.perf_counter() + budget_s / 2
        while True:
            t0 = time.perf_counter()
            decode.decode_step(cfg, wl.L, one["q"], one["sink_k"], one["sink_v"], one["bases_k"], one["bases_v"],
                               one["coef_k"], one["coef_v"], qwin_prev=qwin)
            times1.append(time.perf_counter() - t0)
            if time.perf_counter() > t_end:
                break
    per_seq1 = float(np.median(times1))
    res["value_1_thread"] = round(per_seq1 * wl.batch * 1e6, 1)
    res["sample"] += (f"; value_1_thread: the same with one BLAS thread, {len(times1)} runs in "
                      f"{sum(times1):.1f} s")
    return res


def copy_calibration(nbytes, reps):
    """A plain elementwise copy of known size (read nbytes, write nbytes), for
    scaling the FETCH_SIZE / WRITE_SIZE counters of a rocprofv3 --pmc run."""
    src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(reps):
        torch.neg(src, out=dst)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes_read": nbytes, "copy_calibration_bytes_written": nbytes,
                      "reps": reps, "kernel": "torch.neg (elementwise, float32)"}), flush=True)


EXTRA_SINGLE = ("tiny_fp32", "llama8b_32k", "qwen7b_128k", "qwen3_4b_120k", "qwen3_4b_120k_w32")
EXTRA_STEPS, EXTRA_WARMUP = 100, 10
PREFILL_ETA = 0.2                # the paper's sampling ratio (Section 4 implementation settings)
MALL_BYTES = 256 << 20          # MI355X Infinity Cache


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="llama8b_128k")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-comparator", action="store_true",
                    help="skip the dense Full-KV comparator (uncompressed bf16 KV of the same shape)")
    ap.add_argument("--no-extra", action="store_true",
                    help="measure the named workload only (by default the headline run also measures every "
                         "other workload and reports it under 'configs')")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="only run a plain copy of BYTES bytes (counter calibration) and exit")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures the single-GPU decode step only: this build runs on one GPU "
              f"(asked for --gpus {args.gpus}, WORLD_SIZE {world}).", file=sys.stderr)
        sys.exit(2)

    torch.cuda.set_device(0)
    if args.copy_calibration:
        copy_calibration(args.copy_calibration, 5)
        return

    import workloads as W

    wl = W.CONFIGS[args.workload]
    if wl.layers != 1:
        print(json.dumps(bench_sustained(args, wl, args.steps, args.warmup)), flush=True)
        return
    result = measure_single(args, wl, args.steps, args.warmup, full=True,
                            comparators=not args.no_comparator)
    if not args.no_extra and wl.name == W.HEADLINE:
        # every other workload, each with its own step counts, roofline entry and
        # CPU-oracle baseline (a shorter sample than the headline's)
        result["configs"] = {}
        for name in EXTRA_SINGLE:
            r = measure_single(args, W.CONFIGS[name], EXTRA_STEPS, EXTRA_WARMUP, full=False,
                               comparators=(name == "qwen3_4b_120k" and not args.no_comparator), cpu_budget=5.0)
            result["configs"][name] = summary_entry(r)
        torch.cuda.empty_cache()
        sw = W.CONFIGS["llama8b_32L_sustained"]
        r = bench_sustained(args, sw, sw.steps, 16, cpu_budget=5.0)
        result["configs"][sw.name] = summary_entry(r)
    print(json.dumps(result), flush=True)


def data_recipe(wl):
    """How the measured inputs were drawn (seeded, synthetic)."""
    if wl.recipe == "raw":
        extra = (f", {wl.outlier_channels} outlier key channels x{wl.outlier_scale:g}" if wl.outlier_channels else "")
        tail = ", Student-t (nu=3) coefficients" if wl.heavy_tail else ""
        return (f"raw pre-RoPE K/V drawn on the GPU: low rank (true rank {wl.r_true}) + {wl.noise:g} noise{tail}"
                f"{extra}, sinks x10, {wl.n_needles} needles at per-sequence positions; bases and coefficient caches "
                f"by the library's GPU prefill (hybrid sample eta={PREFILL_ETA}, token-wise normalisation, "
                f"truncated SVD, bulk projection)")
    return ("stored state drawn in latent coordinates: per-sequence orthonormal bases (QR of a Gaussian), "
            f"low-rank coefficient rows (true rank {wl.r_true}) + noise, sinks x10, {wl.n_needles} needles")


def summary_entry(r):
    """The per-workload entry of the headline line's 'configs' object."""
    keep = ("metric", "value", "unit", "steps", "warmup", "higher_is_better", "dtype", "data_recipe", "config",
            "achieved_step_GBps", "step_frac_of_hbm_peak", "algorithmic_bytes_per_step", "read_ceiling_GBps",
            "kernels_us", "kernels_us_per_layer", "roofline", "reconstruction_mfma", "comparator_full_kv",
            "cpu_baseline")
    return {k: r[k] for k in keep if k in r}


def replicas_for(bytes_per_replica):
    """Cache replicas to rotate over so that consecutive steps never find their
    coefficients in the Infinity Cache: at least 4 and at least 3x its size."""
    return int(max(N_REPLICAS, -(-3 * MALL_BYTES // max(1, bytes_per_replica))))


def measure_single(args, wl, steps, warmup, full, comparators, cpu_budget=10.0):
    """One single-layer workload: the fused step timed over `steps` steps
    after `warmup`, the per-kernel pass, the roofline entry of the latent-score
    stream and the CPU-oracle baseline; with `full`, also the per-step
    distribution, the graph replay and the read ceiling; with `comparators`,
    the dense Full-KV and full-reconstruction decodes of the same shape."""
    import paper_2608_00528_amd as s4r
    import workloads as W

    log(f"[bench] generating {wl.describe()} ({wl.recipe} recipe)")
    t0 = time.perf_counter()
    cap = ((wl.L + 15) // 16) * 16
    c = s4r.make_config(batch=wl.batch, n_q_heads=wl.n_q_heads, n_kv_heads=wl.n_kv_heads, head_dim=wl.head_dim,
                        rank=wl.rank, basis_groups=wl.basis_groups, n_sink=wl.n_sink, window=wl.window,
                        q_window=wl.q_window, topk=wl.topk, pool_kernel=wl.pool_kernel, pool_mode=wl.pool_mode,
                        group_agg=wl.group_agg, rope_theta=wl.rope_theta, dtype=wl.dtype, capacity=cap)
    dt = s4r.storage_dtype(c)

    def up(x):
        return torch.from_numpy(np.ascontiguousarray(x)).to(device="cuda", dtype=dt)

    if wl.recipe == "raw":
        # raw prompt K/V of the workload's recipe (low rank, outlier key
        # channels, sinks x10, needles) drawn on the GPU, then the prefill of
        # Section 3.1 on the GPU: hybrid sample (eta = 0.2), token-wise
        # normalisation, truncated SVD, bulk projection into the tiled caches
        raw = W.raw_kv_device(wl, seed=args.seed)
        pf = s4r.prefill(c, raw["S_k"], raw["S_v"], eta=PREFILL_ETA)
        q, sk, sv, bk, bv = raw["q"], pf["sink_k"], pf["sink_v"], pf["bases_k"], pf["bases_v"]
        qwin = None
        reps = [pf["coef_k"], pf["coef_v"]]
        del raw, pf
        # the CPU oracle's timing sample: one sequence of the same shape drawn
        # on the host (the oracle never reads a state built by the GPU)
        st = W.latent_state(wl.scaled(batch=1), seed=args.seed)
    else:
        st = W.latent_state(wl, seed=args.seed)
        # latent axes in the library's storage width (ranks rounded up to 32, zero columns)
        q, sk, sv = (up(st[k]) for k in ("q", "sink_k", "sink_v"))
        bk, bv = (up(s4r.pad_latent(st[k], wl.rank)) for k in ("bases_k", "bases_v"))
        qwin = None if st["qwin_prev"] is None else torch.from_numpy(
            s4r.pad_latent(st["qwin_prev"], wl.rank, wl.basis_groups)).to("cuda", torch.float32)
        reps = []
        for key in ("coef_k", "coef_v"):
            rm = np.zeros((wl.batch, cap, s4r.rank_stride(wl.rank) * wl.basis_groups))
            rm[:, :wl.L] = s4r.pad_latent(st[key], wl.rank, wl.basis_groups)
            reps.append(s4r.pack_coef(c, cap, up(rm)))
    torch.cuda.synchronize()
    log(f"[bench] generated in {time.perf_counter() - t0:.1f} s")
    n_rep = replicas_for(sum(t.numel() * t.element_size() for t in reps))
    replicas = [(reps[0], reps[1])] + [(reps[0].clone(), reps[1].clone()) for _ in range(n_rep - 1)]
    ws = s4r.alloc_workspace(c)
    out = torch.empty((wl.batch, wl.n_q_heads, wl.head_dim), dtype=torch.float32, device="cuda")
    m = s4r.num_selected(c, wl.L)
    torch.cuda.synchronize()

    # with a query window of several rows the step is the windowed one: the
    # older rows' softmax stays resident in the window state (set up once from
    # their coefficient rows; every replica holds the same cache), and only the
    # newest row is scored
    windowed = wl.q_window > 1
    state = None
    if windowed:
        state = s4r.alloc_window_state(c)
        s4r.window_state_init(c, wl.L, qwin, replicas[0][0], state, ws)

    def step(i):
        ck, cv = replicas[i % n_rep]
        if windowed:
            s4r.decode_step_windowed(c, wl.L, q, state, sk, sv, bk, bv, ck, cv, ws, out=out)
        else:
            s4r.decode_step(c, wl.L, q, sk, sv, bk, bv, ck, cv, ws, qwin_prev=qwin, out=out)

    for i in range(warmup):
        step(i)
    torch.cuda.synchronize()
    log(f"[bench] warmup done ({warmup} steps)")

    stream = torch.cuda.current_stream()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    e0.record(stream)
    for i in range(steps):
        step(i)
    e1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    ms_total = e0.elapsed_time(e1)
    ms_step = ms_total / steps
    log(f"[bench] {wl.name}: {steps} steps: {ms_step * 1e3:.2f} us/step (events), "
        f"wall {wall / steps * 1e6:.2f} us/step" + (" (windowed step)" if windowed else ""))
    stateless_us = None
    if windowed:
        # the same step recomputing every window row from qwin_prev, for reference
        ns = min(steps, 50)
        for i in range(5):
            s4r.decode_step(c, wl.L, q, sk, sv, bk, bv, *replicas[i % n_rep], ws, qwin_prev=qwin, out=out)
        e0.record(stream)
        for i in range(ns):
            s4r.decode_step(c, wl.L, q, sk, sv, bk, bv, *replicas[i % n_rep], ws, qwin_prev=qwin, out=out)
        e1.record(stream)
        torch.cuda.synchronize()
        stateless_us = e0.elapsed_time(e1) / ns * 1e3
        log(f"[bench] {wl.name}: stateless step (every window row scored): {stateless_us:.2f} us/step")

    result_extra = {}
    if full:
        result_extra = step_distribution_graph_ceiling(s4r, step, out, replicas, n_rep, steps)
    comparator = None
    if comparators and wl.dtype == "bf16" and wl.head_dim == 128:
        # the prefill's bulk projection is built for ranks up to 192
        comparator = run_comparators(s4r, W, args, wl, c, q, sk, sv, bk, bv, replicas[0], ws, out, ms_step,
                                     prefill=full and s4r.rank_stride(wl.rank) <= 192)

    # per-kernel pass (events between kernels), same steps again
    nk = min(steps, 200)
    s4r.timing_enable(nk)
    for i in range(nk):
        step(i)
    torch.cuda.synchronize()
    kms, nsteps = s4r.timing_read()
    kus = {k: v / nsteps * 1e3 for k, v in kms.items()}
    log(f"[bench] {wl.name} per-kernel us: " + ", ".join(f"{k}={v:.2f}" for k, v in kus.items()))

    alg = algorithmic(wl, m, windowed)
    stream_us = kus["score_stream"]
    achieved = alg["stream_bytes"] / (stream_us * 1e-6) / 1e9
    traffic = traffic_from_profile(wl.name)
    step_gbps = alg["step_bytes"] / (ms_step * 1e-3) / 1e9
    rec_tflops = alg["rec_flops"] / (kus["attn_split"] * 1e-6) / 1e12

    metric = "us per decode step (all heads, 1 layer) at 128k ctx; achieved HBM GB/s vs peak"
    if wl.name != W.HEADLINE:
        metric = f"us per decode step (all heads, 1 layer) at N={wl.N}; achieved HBM GB/s vs peak"
    result = {
        "metric": metric,
        "value": round(ms_step * 1e3, 3),
        "unit": "us/step",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if wl.dtype == "bf16" else "fp32",
        "data": "synthetic",
        "data_recipe": data_recipe(wl),
        "config": {
            "workload": (f"{wl.name}: {SHAPES.get(wl.name, 'single')} layer, B={wl.batch}, N={wl.N} "
                         f"(L={wl.L} non-sink), h_q/h_kv={wl.n_q_heads}/{wl.n_kv_heads}, d_h={wl.head_dim}, "
                         f"rank {wl.R}, s={wl.n_sink}, W={wl.window}, W_q={wl.q_window}, k={wl.topk}, m={m}, "
                         f"{wl.dtype} storage"),
            "batch": wl.batch, "context": wl.N, "rank": wl.R, "window": wl.window, "topk": wl.topk,
            "selected": m, "replicas": n_rep,
            **({"step": "windowed (the older query rows' softmax resident in the window state; "
                         "s4r_decode_step_windowed)"} if windowed else {}),
        },
        **result_extra,
        **({"stateless_us_per_step": round(stateless_us, 3)} if windowed else {}),
        "achieved_step_GBps": round(step_gbps, 1),
        "step_frac_of_hbm_peak": round(step_gbps / HBM_PEAK_GBPS, 4),
        "algorithmic_bytes_per_step": alg["step_bytes"],
        "kernels_us": {k: round(v, 3) for k, v in kus.items()},
        "roofline": {
            "kernel": "k_score_stream (latent scoring over C^K)",
            "bound": "hbm",
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBPS, 4),
            "traffic": traffic,
            "algorithmic_bytes_per_launch": alg["stream_bytes"],
            "avg_launch_us": round(stream_us, 3),
        },
        "reconstruction_mfma": {
            "kernel": "k_attn_tiles (reconstruction + attention on bf16 MFMA)" if wl.dtype == "bf16"
                      else "k_attn_split (reconstruction + attention, fp32 storage)",
            "flops": alg["rec_flops"],
            "avg_launch_us": round(kus["attn_split"], 3),
            "achieved_TFLOPs": round(rec_tflops, 2),
            "peak_TFLOPs": BF16_PEAK_TFLOPS,
            "frac": round(rec_tflops / BF16_PEAK_TFLOPS, 5),
        },
    }
    if comparator is not None:
        result["comparator_full_kv"] = comparator
    del replicas, ws
    if not args.no_cpu_baseline:
        log(f"[bench] timing the CPU oracle on a bounded sample of {wl.name}")
        result["cpu_baseline"] = cpu_baseline(wl, st, budget_s=cpu_budget, one_thread=full)
    del st
    torch.cuda.empty_cache()
    return result


def step_distribution_graph_ceiling(s4r, step, out, replicas, n_rep, steps):
    """Headline extras: per-step distribution, HIP-graph replay and the read
    ceiling over the same coefficient bytes."""
    stream = torch.cuda.current_stream()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    torch.cuda.synchronize()
    ev[0].record(stream)
    for i in range(steps):
        step(i)
        ev[i + 1].record(stream)
    torch.cuda.synchronize()
    per = np.array([ev[i].elapsed_time(ev[i + 1]) * 1e3 for i in range(steps)])
    p10, p50, p90 = (float(np.percentile(per, x)) for x in (10, 50, 90))
    log(f"[bench] per-step us: p10 {p10:.2f}  median {p50:.2f}  p90 {p90:.2f}")

    # the same steps replayed from a HIP graph (one captured step per cache
    # replica); the graph's output is checked against an eager step first
    graph_us = None
    try:
        ref_out = []
        for r in range(n_rep):
            step(r)
            ref_out.append(out.clone())
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            for r in range(n_rep):
                step(r)
        g.replay()
        torch.cuda.synchronize()
        if torch.equal(out, ref_out[n_rep - 1]):
            reps_g = max(1, steps // n_rep)
            g0 = torch.cuda.Event(enable_timing=True)
            g1 = torch.cuda.Event(enable_timing=True)
            g0.record(stream)
            for _ in range(reps_g):
                g.replay()
            g1.record(stream)
            torch.cuda.synchronize()
            graph_us = g0.elapsed_time(g1) * 1e3 / (reps_g * n_rep)
            log(f"[bench] graph replay: {graph_us:.2f} us/step")
        else:
            log("[bench] graph replay output differs from the eager step; graph timing not reported")
        del g
    except Exception as exc:   # capture unsupported here: report eager numbers only
        log(f"[bench] graph capture failed: {exc}")

    # achievable read bandwidth over the same bytes: the library's read
    # reference (one contiguous range per workgroup, non-temporal 16-byte
    # loads) over one C^K replica per launch, rotating replicas
    cks = [r[0] for r in replicas]
    sink = None
    for r in range(n_rep):
        sink = s4r.read_bandwidth(cks[r], sink)
    torch.cuda.synchronize()
    r0 = torch.cuda.Event(enable_timing=True)
    r1 = torch.cuda.Event(enable_timing=True)
    nrd = 4 * n_rep
    r0.record(stream)
    for i in range(nrd):
        s4r.read_bandwidth(cks[i % n_rep], sink)
    r1.record(stream)
    torch.cuda.synchronize()
    read_gbps = cks[0].numel() * cks[0].element_size() * nrd / (r0.elapsed_time(r1) * 1e-3) / 1e9
    log(f"[bench] read ceiling (contiguous non-temporal 16-byte stream over C^K): {read_gbps:.0f} GB/s")
    return {"step_us_p10_median_p90": [round(p10, 3), round(p50, 3), round(p90, 3)],
            "graph_replay_us_per_step": None if graph_us is None else round(graph_us, 3),
            "read_ceiling_GBps": round(read_gbps, 1)}


def run_comparators(s4r, W, args, wl, c, q, sk, sv, bk, bv, coef0, ws, out, ms_step, prefill):
    """The comparators on the same GPU: dense GQA decode over the uncompressed
    bf16 KV cache of the same shape (the paper's Full KV), full-reconstruction
    low-rank decoding over the same coefficient caches (Appendix B.1), and with
    `prefill` the prefill's bulk projection and basis construction."""
    stream = torch.cuda.current_stream()
    dc = W.dense_cache(wl, seed=args.seed)
    cd = s4r.make_config(batch=wl.batch, n_q_heads=wl.n_q_heads, n_kv_heads=wl.n_kv_heads,
                         head_dim=wl.head_dim, rank=wl.rank, n_sink=wl.n_sink, window=wl.window, topk=wl.topk,
                         rope_theta=wl.rope_theta, dtype=wl.dtype, capacity=((wl.N + 15) // 16) * 16)
    dk = torch.zeros((wl.batch, cd.capacity, wl.Dp), dtype=torch.bfloat16, device="cuda")
    dv = torch.zeros_like(dk)
    dk[:, :wl.N], dv[:, :wl.N] = dc["k"], dc["v"]
    del dc["k"], dc["v"]
    wsd = s4r.alloc_workspace(cd)
    outd = torch.empty_like(out)
    for _ in range(3):
        s4r.dense_decode(cd, wl.N, dc["q"], dk, dv, wsd, out=outd)
    torch.cuda.synchronize()
    nd = 20
    d0 = torch.cuda.Event(enable_timing=True)
    d1 = torch.cuda.Event(enable_timing=True)
    d0.record(stream)
    for _ in range(nd):
        s4r.dense_decode(cd, wl.N, dc["q"], dk, dv, wsd, out=outd)
    d1.record(stream)
    torch.cuda.synchronize()
    dense_us = d0.elapsed_time(d1) * 1e3 / nd
    dense_bytes = 2 * wl.batch * wl.N * wl.Dp * 2
    comparator = {
        "what": "dense GQA decode over the uncompressed bf16 KV cache of the same shape (Full KV), "
                "s4r_dense_decode: k_dense_decode + k_attn_combine",
        "us_per_step": round(dense_us, 2),
        "kv_bytes_per_step": dense_bytes,
        "achieved_GBps": round(dense_bytes / (dense_us * 1e-6) / 1e9, 1),
        "frac_of_hbm_peak": round(dense_bytes / (dense_us * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4),
        "s4r_step_speedup": round(dense_us / (ms_step * 1e3), 2),
    }
    log(f"[bench] {wl.name} dense Full-KV comparator: {dense_us:.1f} us/step "
        f"({comparator['achieved_GBps']:.0f} GB/s), S4R step {comparator['s4r_step_speedup']:.2f}x faster")
    if prefill:
        # the prefill's bulk projection C = S B of the same prompt (those rows as S)
        n_pf = cd.capacity
        cpf = s4r.make_config(batch=wl.batch, n_q_heads=wl.n_q_heads, n_kv_heads=wl.n_kv_heads,
                              head_dim=wl.head_dim, rank=wl.rank, n_sink=wl.n_sink, window=wl.window,
                              topk=wl.topk, rope_theta=wl.rope_theta, dtype=wl.dtype, capacity=n_pf)
        pk = torch.empty((wl.batch, n_pf, wl.R), dtype=torch.bfloat16, device="cuda")
        pv = torch.empty_like(pk)
        wspf = s4r.alloc_workspace(cpf)
        s4r.prefill_project(cpf, n_pf, dk, dv, bk, bv, pk, pv, wspf)
        torch.cuda.synchronize()
        p0 = torch.cuda.Event(enable_timing=True)
        p1 = torch.cuda.Event(enable_timing=True)
        npf = 5
        p0.record(stream)
        for _ in range(npf):
            s4r.prefill_project(cpf, n_pf, dk, dv, bk, bv, pk, pv, wspf)
        p1.record(stream)
        torch.cuda.synchronize()
        pf_us = p0.elapsed_time(p1) * 1e3 / npf
        pf_bytes = 2 * wl.batch * n_pf * (wl.Dp + wl.R) * 2
        comparator["prefill_projection"] = {
            "what": f"s4r_prefill_project: C = S B for K and V of {wl.batch} x {n_pf} prompt rows (Section 3.1)",
            "us": round(pf_us, 1), "bytes": pf_bytes,
            "achieved_GBps": round(pf_bytes / (pf_us * 1e-6) / 1e9, 1),
            "frac_of_hbm_peak": round(pf_bytes / (pf_us * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4),
        }
        log(f"[bench] prefill bulk projection: {pf_us:.1f} us "
            f"({comparator['prefill_projection']['achieved_GBps']:.0f} GB/s)")
        # the prefill's basis construction for the same prompt (sample, normalise,
        # Gram in fp64, eigenvectors), 20% of the rows sampled
        wsb = torch.empty(s4r.api.prefill_bases_workspace_size(cpf, n_pf, 0.2), dtype=torch.uint8, device="cuda")
        bkp, bvp = s4r.prefill_bases(cpf, n_pf, dk, dv, eta=0.2, center=True, ws=wsb)
        torch.cuda.synchronize()
        q0 = torch.cuda.Event(enable_timing=True)
        q1 = torch.cuda.Event(enable_timing=True)
        nq = 3
        q0.record(stream)
        for _ in range(nq):
            s4r.prefill_bases(cpf, n_pf, dk, dv, eta=0.2, center=True, bases_k=bkp, bases_v=bvp, ws=wsb)
        q1.record(stream)
        torch.cuda.synchronize()
        pb_ms = q0.elapsed_time(q1) / nq
        comparator["prefill_bases"] = {
            "what": f"s4r_prefill_bases: hybrid sample of {s4r.num_samples(n_pf, 0.2)} of {n_pf} rows, token-wise "
                    f"normalisation, centring, fp64 Gram and top-{wl.rank} eigenvectors for K and V of "
                    f"{wl.batch} sequences (Section 3.1.2)",
            "ms": round(pb_ms, 2),
        }
        log(f"[bench] prefill basis construction: {pb_ms:.2f} ms")
        del wsb, bkp, bvp, pk, pv, wspf
    del dk, dv, wsd
    torch.cuda.synchronize()
    # full-reconstruction low-rank decoding (Appendix B.1) over the same
    # coefficient caches: every one of the L tokens reconstructed
    ck0, cv0 = coef0
    outf = torch.empty_like(out)
    for _ in range(2):
        s4r.full_recon_decode(c, wl.L, q, sk, sv, bk, bv, ck0, cv0, ws, out=outf)
    torch.cuda.synchronize()
    f0 = torch.cuda.Event(enable_timing=True)
    f1 = torch.cuda.Event(enable_timing=True)
    nfr = 10
    f0.record(stream)
    for _ in range(nfr):
        s4r.full_recon_decode(c, wl.L, q, sk, sv, bk, bv, ck0, cv0, ws, out=outf)
    f1.record(stream)
    torch.cuda.synchronize()
    fr_us = f0.elapsed_time(f1) * 1e3 / nfr
    fr_flops = 2 * 2 * wl.batch * wl.L * wl.R * wl.Dp
    comparator["full_reconstruction"] = {
        "what": "full-reconstruction low-rank decoding (Appendix B.1): s4r_full_recon_decode, every non-sink "
                "token reconstructed on the matrix cores (k_attn_tiles over all tokens + k_attn_combine)",
        "us_per_step": round(fr_us, 2),
        "reconstruction_flops": fr_flops,
        "achieved_TFLOPs": round(fr_flops / (fr_us * 1e-6) / 1e12, 1),
        "frac_of_bf16_peak": round(fr_flops / (fr_us * 1e-6) / 1e12 / BF16_PEAK_TFLOPS, 4),
        "s4r_step_speedup": round(fr_us / (ms_step * 1e3), 2),
    }
    log(f"[bench] {wl.name} full-reconstruction comparator: {fr_us:.1f} us/step "
        f"({comparator['full_reconstruction']['achieved_TFLOPs']:.0f} TFLOP/s), "
        f"S4R step {comparator['full_reconstruction']['s4r_step_speedup']:.2f}x faster")
    return comparator


def bench_sustained(args, wl, steps, warmup, kernel_steps=8, cpu_budget=10.0):
    """Sustained multi-layer decode: every step runs all layers one after the
    other, each layer appending the new token's key/value coefficients (row
    L - 1) before scoring, so the context grows by one token per step.  Steps
    W..W+K-1 are timed as a whole; a further `kernel_steps` steps run with the
    per-kernel event hook for the roofline entry."""
    import paper_2608_00528_amd as s4r
    import workloads as W

    total = warmup + steps + kernel_steps
    L0 = wl.L - 1                       # the first step appends row L0 and runs at L = wl.L
    cap = ((L0 + total + 15) // 16) * 16
    c = s4r.make_config(batch=wl.batch, n_q_heads=wl.n_q_heads, n_kv_heads=wl.n_kv_heads, head_dim=wl.head_dim,
                        rank=wl.rank, basis_groups=wl.basis_groups, n_sink=wl.n_sink, window=wl.window,
                        q_window=wl.q_window, topk=wl.topk, pool_kernel=wl.pool_kernel, pool_mode=wl.pool_mode,
                        group_agg=wl.group_agg, rope_theta=wl.rope_theta, dtype=wl.dtype, capacity=cap)
    log(f"[bench] generating {wl.describe()}: {wl.layers} layers, {total} steps, capacity {cap}")
    t0 = time.perf_counter()
    layers, host0 = [], None
    for layer in range(wl.layers):
        st = W.sustained_layer(wl, args.seed, layer, L0, cap, total)
        if layer == 0:
            host0 = {k: st[k][:1].float().cpu().numpy().astype(np.float64)
                     for k in ("sink_k", "sink_v", "bases_k", "bases_v")}
            host0["coef_k"] = st["coef_k"][:1, :L0].float().cpu().numpy().astype(np.float64)
            host0["coef_v"] = st["coef_v"][:1, :L0].float().cpu().numpy().astype(np.float64)
            host0["q"] = st["q"][0, :1].float().cpu().numpy().astype(np.float64)
            host0["k_new"] = st["k_new"][0, :1].float().cpu().numpy().astype(np.float64)
            host0["v_new"] = st["v_new"][0, :1].float().cpu().numpy().astype(np.float64)
        for key in ("coef_k", "coef_v"):
            st[key] = s4r.pack_coef(c, cap, st[key])
        torch.cuda.synchronize()
        layers.append(st)
        if layer % 8 == 7:
            log(f"[bench] layer {layer + 1}/{wl.layers} resident ({time.perf_counter() - t0:.1f} s)")
    ws = s4r.alloc_workspace(c)
    outs = [torch.empty((wl.batch, wl.n_q_heads, wl.head_dim), dtype=torch.float32, device="cuda")
            for _ in range(wl.layers)]
    coef_bytes = sum(st[k].numel() * st[k].element_size() for st in layers for k in ("coef_k", "coef_v"))
    log(f"[bench] {coef_bytes / 1e9:.1f} GB of coefficients resident")

    def step(t):
        for layer, st in enumerate(layers):
            s4r.decode_step(c, L0 + t + 1, st["q"][t], st["sink_k"], st["sink_v"], st["bases_k"], st["bases_v"],
                            st["coef_k"], st["coef_v"], ws, k_new=st["k_new"][t], v_new=st["v_new"][t],
                            out=outs[layer])

    for t in range(warmup):
        step(t)
    torch.cuda.synchronize()
    log(f"[bench] warmup done ({warmup} steps)")
    stream = torch.cuda.current_stream()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for t in range(warmup, warmup + steps):
        step(t)
    e1.record(stream)
    torch.cuda.synchronize()
    ms_step = e0.elapsed_time(e1) / steps
    log(f"[bench] {steps} steps x {wl.layers} layers: {ms_step:.3f} ms/step, {1e3 / ms_step:.1f} steps/s")

    s4r.timing_enable(kernel_steps * wl.layers)
    for t in range(warmup + steps, total):
        step(t)
    torch.cuda.synchronize()
    kms, ncalls = s4r.timing_read()
    kus = {k: v / ncalls * 1e3 for k, v in kms.items()}
    log("[bench] per-layer kernel us: " + ", ".join(f"{k}={v:.2f}" for k, v in kus.items()))

    m = s4r.num_selected(c, wl.L)
    es = 2 if wl.dtype == "bf16" else 4
    L_mid = L0 + warmup + steps + kernel_steps // 2 + 1
    stream_bytes = wl.batch * L_mid * wl.R * es
    achieved = stream_bytes / (kus["score_stream"] * 1e-6) / 1e9
    layer_bytes = (stream_bytes + 2 * wl.batch * m * wl.R * es + 2 * wl.batch * wl.Dp * wl.R * es
                   + 2 * wl.batch * wl.n_sink * wl.Dp * es + wl.batch * wl.n_q_heads * wl.head_dim * (es + 4)
                   + 2 * wl.batch * wl.Dp * es + 2 * wl.batch * wl.R * es)
    step_gbps = layer_bytes * wl.layers / (ms_step * 1e-3) / 1e9
    result = {
        "metric": f"decode steps/s, {wl.layers} layers, sustained over {steps} steps",
        "value": round(1e3 / ms_step, 2),
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if wl.dtype == "bf16" else "fp32",
        "data": "synthetic",
        "config": {
            "workload": (f"{wl.name}: {wl.layers} Llama-3.1-8B-shaped layers, B={wl.batch}, N={wl.N} at the first "
                         f"timed step and +1 token per step, h_q/h_kv={wl.n_q_heads}/{wl.n_kv_heads}, "
                         f"d_h={wl.head_dim}, rank {wl.R}, s={wl.n_sink}, W={wl.window}, k={wl.topk}, "
                         f"{wl.dtype} storage, new token projected and appended in every layer of every step"),
            "batch": wl.batch, "context": wl.N, "layers": wl.layers, "rank": wl.R, "window": wl.window,
            "topk": wl.topk, "selected": m, "coefficient_GB": round(coef_bytes / 1e9, 2),
        },
        "achieved_step_GBps": round(step_gbps, 1),
        "step_frac_of_hbm_peak": round(step_gbps / HBM_PEAK_GBPS, 4),
        "kernels_us_per_layer": {k: round(v, 3) for k, v in kus.items()},
        "roofline": {
            "kernel": "k_score_stream (latent scoring over C^K)",
            "bound": "hbm",
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBPS, 4),
            "traffic": None,
            "algorithmic_bytes_per_launch": stream_bytes,
            "avg_launch_us": round(kus["score_stream"], 3),
        },
    }
    del layers, ws
    torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle on a bounded sample")
        result["cpu_baseline"] = cpu_baseline_sustained(wl, host0, L0 + 1, budget_s=cpu_budget)
    return result


def cpu_baseline_sustained(wl, one, L, budget_s=10.0):
    """The oracle on one sequence of one layer (append + decode step),
    repeated for about budget_s seconds, extrapolated to the whole step."""
    from threadpoolctl import threadpool_info

    from oracle import decode
    cfg = dict(n_kv_heads=wl.n_kv_heads, window=wl.window, topk=wl.topk, pool_kernel=wl.pool_kernel,
               pool_mode=wl.pool_mode, group_agg=wl.group_agg, rope_theta=wl.rope_theta, dtype=wl.dtype)
    ck = np.zeros((1, L, wl.R))
    cv = np.zeros((1, L, wl.R))
    ck[:, :L - 1], cv[:, :L - 1] = one["coef_k"], one["coef_v"]
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    times = []
    t_end = time.perf_counter() + budget_s
    while True:
        t0 = time.perf_counter()
        decode.decode_step(cfg, L, one["q"], one["sink_k"], one["sink_v"], one["bases_k"], one["bases_v"], ck, cv,
                           k_new=one["k_new"], v_new=one["v_new"])
        times.append(time.perf_counter() - t0)
        if time.perf_counter() > t_end:
            break
    per_seq = float(np.median(times))
    step_s = per_seq * wl.batch * wl.layers
    return {"value": round(1.0 / step_s, 5), "unit": "steps/s", "cores": threads, "kind": "oracle",
            "host_cpus": os.cpu_count(),
            "sample": (f"float64 numpy oracle, sequence 0 of layer 0 at L={L} (append + decode step), {len(times)} "
                       f"runs in {sum(times):.1f} s, median per sequence extrapolated x {wl.batch} sequences x "
                       f"{wl.layers} layers; BLAS threads {threads}")}


if __name__ == "__main__":
    main()
