"""Benchmark of the fused attention-forward hot path on one MI355X.

A step is one attn_fwd call over the whole workload (default: MHA, B=1, H=16,
S=131072, d=128, causal -- the long-context case whose K/V per head, 64 MiB,
far exceeds an XCD's 4 MB L2) with the swizzled head-first mapping -- under a
causal mask with each head's row blocks dispatched heaviest first, which keeps
every head on its XCD -- inputs already resident in HBM.  Prints ONE JSON line:

  value       attention TFLOP/s (FlashAttention flop convention) of the timed
              K back-to-back steps (warm: no cache flush between them), after
              a warm-up of at least --warmup steps and --warmup-s seconds
  headline_cold  the same variant launched alone after an L2 + MALL flush,
              --reps times interleaved with the other variants: median, min,
              max and IQR of the launch time
  roofline    the kernel against the dense bf16 MFMA peak (2.5 PFLOP/s):
              achieved = algorithmic flop per launch / average launch time
              (HIP events on the launch stream over the timed region);
              traffic = HBM bytes per launch from rocprofv3 FETCH_SIZE +
              WRITE_SIZE (scaled by a copy kernel of known size), read from
              the committed counter summary when it was taken on this kernel
              source, else null
  mfma_ceiling  the dense bf16 MFMA rate this chip sustains, measured live by
              a kernel of register-operand MFMAs only (attn_calib_mfma), with
              the shader clock it runs at; frac = value / that rate.  The
              published peak assumes the 2.4 GHz peak clock, which a sustained
              matrix-core load does not get
  per_mapping TFLOP/s of all four mappings (for causal workloads also each
              with the heavy-first block order) and of swizzled head-first with
              block-major order inside each XCD, interleaved, cold (L2 and MALL
              flushed before every launch) and warm, median over reps with min,
              max and IQR, plus the L2 hit rate from the counter summary
  small_workload  the small MHA case (B=1, H=4, S=256, d=64), which launch
              latency bounds: every mapping, --small-reps interleaved cold
              launches, median / min / IQR
  cpu_baseline  the fp64 CPU oracle on a time-bounded sample of the same
              workload's rows, in TFLOP/s of the same flop count

The warm-up is timed as well as counted: the power manager lowers the shader
clock for some tens of milliseconds after a matrix-core load starts, and the
K timed steps measure the settled rate.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
       python bench.py --profile [--workload NAME]   (kernel launches only, for rocprofv3)
"""

from __future__ import annotations

import argparse
import json
import os
import re
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
DEFAULT_WORKLOAD = "mha_b1_h16_s131072_d128_causal"
SMALL_WORKLOAD = "mha_b1_h4_s256_d64"
METRIC = "attention fwd TFLOP/s (% of bf16 MFMA peak) + L2 hit rate, per mapping"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0


def variants(causal: bool, d: int):
    """(name, mapping value) pairs measured per mapping."""
    import paper_2511_02132_amd as pa
    return pa.variants(causal, d)


def kernel_source_hash() -> str:
    from paper_2511_02132_amd.build import kernel_source_hash as h
    return h()


def counter_summary(workload: str):
    """Counter figures from profiles/, if they were taken on this kernel source."""
    path = os.path.join(ROOT, "profiles", "attn_fwd_%s_counters.md" % workload)
    if not os.path.exists(path):
        return None
    m = re.search(r"```json\n(.*?)\n```", open(path).read(), re.S)
    if not m:
        return None
    data = json.loads(m.group(1))
    if data.get("kernel_source_sha256") != kernel_source_hash():
        return None
    return data


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    p.add_argument("--warmup", type=int, default=10)
    p.add_argument("--warmup-s", type=float, default=2.0,
                   help="the warm-up also lasts at least this long (seconds)")
    p.add_argument("--workload", default=DEFAULT_WORKLOAD)
    p.add_argument("--reps", type=int, default=10, help="cold reps per mapping")
    p.add_argument("--small-reps", type=int, default=300,
                   help="cold reps per mapping of the small workload")
    p.add_argument("--no-small", action="store_true")
    p.add_argument("--cpu-seconds", type=float, default=12.0)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--profile", action="store_true",
                   help="kernel launches only, for rocprofv3: every mapping variant, a "
                        "one-workgroup launch and a copy of known size")
    p.add_argument("--profile-launches", type=int, default=2)
    return p.parse_args()


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU; there is no multi-GPU path (the forward would "
              "shard heads across GPUs with no exchange). Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import attn_inputs as ai
    import paper_2511_02132_amd as pa

    w = ai.WORKLOADS[args.workload]
    B, Hq, Hkv, Sq, Skv, d, causal = (w[k] for k in ("B", "Hq", "Hkv", "Sq", "Skv", "d", "causal"))
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    q_cpu, k_cpu, v_cpu = ai.workload_inputs(args.workload)
    q, k, v = q_cpu.to(dev), k_cpu.to(dev), v_cpu.to(dev)
    o = torch.empty_like(q)
    scale = ai.default_scale(d)
    flops = pa.attention_flops(B, Hq, Sq, Skv, d, causal)
    stream = torch.cuda.current_stream(dev)

    def step(mapping):
        pa.attn_fwd(q, k, v, o, causal=causal, scale=scale, mapping=mapping, stream=stream)

    if args.profile:
        # Each (mapping, order) is its own kernel symbol, so one run covers all.
        for _, m in variants(causal, d):
            for _ in range(args.profile_launches):
                step(m)
        # One workgroup (wid 0 runs on XCD 0): shows which counter instances belong to XCD 0.
        q1 = torch.zeros(1, 1, pa.block_m(128), 128, dtype=torch.bfloat16, device=dev)
        kv1 = torch.zeros(1, 1, 4096, 128, dtype=torch.bfloat16, device=dev)
        pa.attn_fwd(q1, kv1, kv1, causal=False, mapping=pa.SWIZZLED_HEAD_FIRST, stream=stream)
        # A plain copy of known size: scales FETCH_SIZE / WRITE_SIZE to bytes.
        src = torch.ones(256 * 2 ** 20, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(args.profile_launches):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"profile": args.workload, "variants": [n for n, _ in variants(causal, d)],
                          "copy_bytes_each_way": src.numel()}), flush=True)
        return

    # ---- headline: K back-to-back steps of the method (swizzled head-first)
    mapping = pa.method_variant(causal)
    headline_name = pa.variant_name(mapping)
    t_warm = time.perf_counter()
    n_warm = 0
    while n_warm < args.warmup or time.perf_counter() - t_warm < args.warmup_s:
        step(mapping)
        n_warm += 1
        if n_warm % 4 == 0:
            torch.cuda.synchronize()
    torch.cuda.synchronize()
    warm_s = time.perf_counter() - t_warm
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(args.steps):
        step(mapping)
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_per_step = ev0.elapsed_time(ev1) / args.steps
    value = flops / (ms_per_step * 1e-3) / 1e12
    print("headline: %.4f ms/step, %.1f TFLOP/s (wall %.3f s; warm-up %d launches, %.2f s)"
          % (ms_per_step, value, wall, n_warm, warm_s), file=sys.stderr, flush=True)

    # ---- compute ceiling: dense bf16 MFMA on register operands, after the
    # headline so that the clock has settled; the later half of the launches
    calib = pa.calib_mfma(dev, launches=8, stream=stream)
    settled = calib[len(calib) // 2:]
    ceiling = {"tflops": round(statistics.median(c["tflops"] for c in settled), 1),
               "clock_mhz": round(statistics.median(c["clock_mhz"] for c in settled)),
               "launches": len(settled)}
    ceiling["frac"] = round(value / ceiling["tflops"], 4)
    # dense bf16 peak at that clock: CUs x 4 SIMDs x 1024 flop per cycle
    n_cu = torch.cuda.get_device_properties(dev).multi_processor_count
    ceiling["peak_at_clock_tflops"] = round(n_cu * 4 * 1024 * ceiling["clock_mhz"] * 1e6 / 1e12, 1)
    ceiling["frac_of_peak_at_clock"] = round(value / ceiling["peak_at_clock_tflops"], 4)
    print("mfma ceiling: %s" % json.dumps(ceiling), file=sys.stderr, flush=True)

    # ---- per mapping: interleaved, cold (L2 + MALL flushed) and warm
    flush = torch.empty(512 * 2 ** 20, dtype=torch.uint8, device=dev)
    vs = variants(causal, d)
    cold, warm = timed_variants(torch, stream, flush, step, vs, args.reps, warm_too=True)
    counters = counter_summary(args.workload)
    per_mapping = {}
    for name, _ in vs:
        ent = {"cold": launch_stats(cold[name], flops), "warm": launch_stats(warm[name], flops)}
        ent["cold_tflops"] = ent["cold"]["tflops_median"]
        ent["warm_tflops"] = ent["warm"]["tflops_median"]
        if counters:
            c = counters["per_mapping"].get(name, {})
            ent["l2_hit_rate"] = c.get("l2_hit_rate")
        per_mapping[name] = ent
    headline_cold = dict(per_mapping[headline_name]["cold"])
    print("per mapping: %s" % json.dumps(per_mapping), file=sys.stderr, flush=True)

    # ---- the small workload: launch-latency bound, every mapping, many reps
    small = None
    if not args.no_small:
        small = small_workload(args, torch, dev, stream, flush, ai, pa)
        print("small workload: %s" % json.dumps(small), file=sys.stderr, flush=True)
    del flush

    # ---- roofline of the kernel (MFMA-bound contraction, bf16 peak)
    achieved = flops / (ms_per_step * 1e-3) / 1e12
    traffic = None
    if counters:
        t = counters["per_mapping"].get(headline_name, {})
        traffic = t.get("hbm_bytes_per_launch")
    roofline = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                "traffic": traffic,
                "work_per_launch": "%.6g flop = 4*B*Hq*Sq*Skv*d%s" % (
                    flops, " / 2 (causal)" if causal else "")}

    # ---- CPU baseline: the oracle on a time-bounded sample of rows
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(args, w, q_cpu, k_cpu, v_cpu, scale)

    out = {
        "metric": METRIC, "value": round(value, 2), "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": n_warm, "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic: Q,K,V ~ N(0,1) rounded to bf16, seeded",
        "timing": "value: K back-to-back launches (warm) after a warm-up of %d launches "
                  "(%.2f s); headline_cold: the same variant after an L2 + MALL flush, %d "
                  "interleaved reps" % (n_warm, warm_s, args.reps),
        "config": {"workload": args.workload, "B": B, "Hq": Hq, "Hkv": Hkv, "Sq": Sq, "Skv": Skv,
                   "d": d, "causal": causal, "mapping": headline_name,
                   "block_m": pa.block_m(d), "block_n": pa.block_n(d), "num_xcd": pa.num_xcd(),
                   "flop_convention": "4*B*Hq*Sq*Skv*d, halved when causal"},
        "roofline": roofline,
        "headline_cold": headline_cold,
        "mfma_ceiling": ceiling,
        "per_mapping": per_mapping,
        "small_workload": small,
        "cpu_baseline": cpu,
        "kernel_source_sha256": kernel_source_hash(),
    }
    print(json.dumps(out), flush=True)


def timed_variants(torch, stream, flush, step, vs, reps, warm_too=False):
    """Launch times (ms) of every variant, interleaved round-robin over reps:
    cold = one launch right after an L2 + MALL flush; warm = the launch that
    follows it (same inputs, caches as the cold launch left them)."""
    cold = {n: [] for n, _ in vs}
    warm = {n: [] for n, _ in vs}
    for _ in range(reps):
        for name, m in vs:
            flush.zero_()
            e = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
            e[0].record(stream)
            step(m)
            e[1].record(stream)
            if warm_too:
                step(m)
                e[2].record(stream)
            torch.cuda.synchronize()
            cold[name].append(e[0].elapsed_time(e[1]))
            if warm_too:
                warm[name].append(e[1].elapsed_time(e[2]))
    return cold, warm


def launch_stats(ms, flops):
    """Median, min, max and interquartile range of launch times (ms), and the
    median and best rate in TFLOP/s."""
    import numpy as np
    med = float(np.median(ms))
    q75, q25 = np.percentile(ms, [75, 25])
    return {"n": len(ms), "ms_median": round(med, 5), "ms_min": round(float(min(ms)), 5),
            "ms_max": round(float(max(ms)), 5), "ms_iqr": round(float(q75 - q25), 5),
            "tflops_median": round(flops / med / 1e9, 2),
            "tflops_best": round(flops / float(min(ms)) / 1e9, 2)}


def small_workload(args, torch, dev, stream, flush, ai, pa):
    """Every mapping on the small MHA workload (B1 H4 S256 d64, non-causal):
    launch-latency bound, so many interleaved cold reps."""
    w = ai.WORKLOADS[SMALL_WORKLOAD]
    qs, ks, vs_ = (t.to(dev) for t in ai.workload_inputs(SMALL_WORKLOAD))
    os_ = torch.empty_like(qs)
    sc = ai.default_scale(w["d"])
    fl = pa.attention_flops(w["B"], w["Hq"], w["Sq"], w["Skv"], w["d"], w["causal"])

    def st(m):
        pa.attn_fwd(qs, ks, vs_, os_, causal=w["causal"], scale=sc, mapping=m, stream=stream)

    vs = variants(w["causal"], w["d"])
    for _, m in vs:   # one untimed launch each
        st(m)
    torch.cuda.synchronize()
    cold, _ = timed_variants(torch, stream, flush, st, vs, args.small_reps)
    out = {"workload": SMALL_WORKLOAD, "flop": fl, "reps": args.small_reps,
           "note": "one launch of 8 workgroups; bound by launch latency, not by the MFMA rate",
           "per_mapping": {}}
    for name, _ in vs:
        st_ = launch_stats(cold[name], fl)
        out["per_mapping"][name] = {"us_median": round(st_["ms_median"] * 1e3, 2),
                                    "us_min": round(st_["ms_min"] * 1e3, 2),
                                    "us_iqr": round(st_["ms_iqr"] * 1e3, 2),
                                    "tflops_median": st_["tflops_median"]}
    return out


def cpu_model() -> str:
    """The host CPU's model name (first processor in /proc/cpuinfo), or "unknown"."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(args, w, q, k, v, scale):
    """Time the oracle on random rows of the workload for about args.cpu_seconds."""
    import numpy as np

    import attn_inputs as ai
    import oracle

    qb, kb, vb = (ai.bf16_bits(t) for t in (q, k, v))
    rng = np.random.default_rng(12345)
    total_flop, total_s, nrows = 0.0, 0.0, 0
    chunk = 64
    while total_s < args.cpu_seconds:
        rows = np.stack([rng.integers(0, w["B"], chunk), rng.integers(0, w["Hq"], chunk),
                         rng.integers(0, w["Sq"], chunk)], axis=1)
        t0 = time.perf_counter()
        oracle.attn_fwd_rows_f64(qb, kb, vb, rows, w["causal"], scale)
        total_s += time.perf_counter() - t0
        keys = np.minimum(rows[:, 2] + 1, w["Skv"]) if w["causal"] else np.full(chunk, w["Skv"])
        total_flop += float(np.sum(4.0 * keys * w["d"]))
        nrows += chunk
        chunk = min(chunk * 2, 4096)
    return {"value": round(total_flop / total_s / 1e12, 6), "unit": "TFLOP/s",
            "cores": oracle.max_threads(), "cpu_model": cpu_model(), "kind": "oracle",
            "sample": "%d uniformly drawn (b, hq, row) query rows of %s, %.1f GFLOP (4*|keys|*d "
                      "per row) in %.1f s, fp64 two-pass softmax" % (
                          nrows, args.workload, total_flop / 1e9, total_s)}


if __name__ == "__main__":
    main()
