"""Benchmark of the fused attention-forward hot path on one MI355X.

A step is one attn_fwd call over the whole workload (default: MHA, B=1, H=32,
S=8192, d=128, causal -- an 8B-class decoder layer) with the swizzled
head-first mapping -- under a causal mask with two dispatch-order options that
keep every head on its XCD: heavy-first blocks, and block-major order across
the heads of each XCD's piece (so the four WGs an XCD receives at a time cost
the same) -- inputs already resident in HBM.  Prints ONE JSON line:

  value       attention TFLOP/s (FlashAttention flop convention) of the timed
              K back-to-back steps
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
              flushed before every launch) and warm, median over reps, plus the
              L2 hit rate from the counter summary
  cpu_baseline  the fp64 CPU oracle on a time-bounded sample of the same
              workload's rows, in TFLOP/s of the same flop count

The default warm-up (60 steps, about 30 ms of work at the default workload)
outlasts the power manager's response to the start of a matrix-core load: the
shader clock dips for some tens of milliseconds before it settles, and the K
timed steps measure the settled rate.

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
DEFAULT_WORKLOAD = "mha_b1_h32_s8192_d128_causal"
METRIC = "attention fwd TFLOP/s (% of bf16 MFMA peak) + L2 hit rate, per mapping"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0


def variants(causal: bool):
    """(name, mapping value) pairs measured per mapping."""
    import paper_2511_02132_amd as pa
    return pa.variants(causal)


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
    p.add_argument("--steps", type=int, default=200)
    p.add_argument("--warmup", type=int, default=60)
    p.add_argument("--workload", default=DEFAULT_WORKLOAD)
    p.add_argument("--reps", type=int, default=10, help="cold reps per mapping")
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
    q, k, v = ai.workload_inputs(args.workload)
    q, k, v = q.to(dev), k.to(dev), v.to(dev)
    o = torch.empty_like(q)
    scale = ai.default_scale(d)
    flops = pa.attention_flops(B, Hq, Sq, Skv, d, causal)
    stream = torch.cuda.current_stream(dev)

    def step(mapping):
        pa.attn_fwd(q, k, v, o, causal=causal, scale=scale, mapping=mapping, stream=stream)

    if args.profile:
        # Each (mapping, order) is its own kernel symbol, so one run covers all.
        for _, m in variants(causal):
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
        print(json.dumps({"profile": args.workload, "variants": [n for n, _ in variants(causal)],
                          "copy_bytes_each_way": src.numel()}), flush=True)
        return

    # ---- headline: K back-to-back steps of the method (swizzled head-first)
    mapping = pa.method_variant(causal)
    headline_name = pa.variant_name(mapping)
    for _ in range(args.warmup):
        step(mapping)
    torch.cuda.synchronize()
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
    print("headline: %.4f ms/step, %.1f TFLOP/s (wall %.3f s)" % (ms_per_step, value, wall),
          file=sys.stderr, flush=True)

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

    # ---- per mapping: interleaved, cold (L2 + MALL flushed) and warm, median
    flush = torch.empty(512 * 2 ** 20, dtype=torch.uint8, device=dev)
    vs = variants(causal)
    cold = {n: [] for n, _ in vs}
    warm = {n: [] for n, _ in vs}
    for _ in range(args.reps):
        for name, m in vs:
            flush.zero_()
            e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
            e0.record(stream)
            step(m)
            e1.record(stream)
            step(m)
            e2.record(stream)
            torch.cuda.synchronize()
            cold[name].append(e0.elapsed_time(e1))
            warm[name].append(e1.elapsed_time(e2))
    del flush
    counters = counter_summary(args.workload)
    per_mapping = {}
    for name, _ in vs:
        cm, wm = statistics.median(cold[name]), statistics.median(warm[name])
        ent = {"cold_ms": round(cm, 5), "cold_tflops": round(flops / cm / 1e9, 2),
               "warm_ms": round(wm, 5), "warm_tflops": round(flops / wm / 1e9, 2),
               "cold_ms_min": round(min(cold[name]), 5), "cold_ms_max": round(max(cold[name]), 5),
               "cold_ms_iqr": round(float(np.subtract(*np.percentile(cold[name], [75, 25]))), 5)}
        if counters:
            c = counters["per_mapping"].get(name, {})
            ent["l2_hit_rate"] = c.get("l2_hit_rate")
        per_mapping[name] = ent
    print("per mapping: %s" % json.dumps(per_mapping), file=sys.stderr, flush=True)

    # ---- roofline of the kernel (MFMA-bound contraction, bf16 peak)
    achieved = flops / (ms_per_step * 1e-3) / 1e12
    traffic = None
    if counters:
        t = counters["per_mapping"].get(headline_name, {})
        traffic = t.get("hbm_bytes_per_launch")
    roofline = {"bound": "mfma", "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                "traffic": traffic}

    # ---- CPU baseline: the oracle on a time-bounded sample of rows
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(args, w, q, k, v, scale)

    out = {
        "metric": METRIC, "value": round(value, 2), "unit": "TFLOP/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic: Q,K,V ~ N(0,1) rounded to bf16, seeded",
        "config": {"workload": args.workload, "B": B, "Hq": Hq, "Hkv": Hkv, "Sq": Sq, "Skv": Skv,
                   "d": d, "causal": causal, "mapping": headline_name,
                   "block_m": pa.block_m(d), "block_n": pa.block_n(d), "num_xcd": pa.num_xcd(),
                   "flop_convention": "4*B*Hq*Sq*Skv*d, halved when causal"},
        "roofline": roofline,
        "mfma_ceiling": ceiling,
        "per_mapping": per_mapping,
        "cpu_baseline": cpu,
        "kernel_source_sha256": kernel_source_hash(),
    }
    print(json.dumps(out), flush=True)


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

    qb, kb, vb = (ai.bf16_bits(t.cpu()) for t in (q, k, v))
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
