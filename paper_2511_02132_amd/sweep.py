"""Mapping sweeps of the paper's sensitivity studies, on one MI355X.

* MHA (Section 4.3, Table "mha_sweep"): context 8K/32K/128K x batch 1/2/4/8 x
  heads (Hq = Hkv) 8/16/32/64/128, head dimension 128.
* GQA (Section 4.4): eight KV heads, Hq = 32/64/128, same contexts and batches.
* DeepSeek-V3 prefill (Section 4.5): 128 heads of dimension 56
  (``--family mha --heads 128 --d 56 --contexts 2048 8192 32768 131072``).
* Backward (Section 4.6, ``--pass bwd``): the gradient kernels of attn_bwd,
  timed after one forward that produced O and the log-sum-exp; the paper's
  study uses 128 heads, 8K/32K/128K and batches 1-2
  (``--family mha --heads 128 --batches 1 2 --pass bwd``).  TFLOP/s use the
  FlashAttention convention for the backward, 2.5x the forward's flops.

Every configuration runs every mapping (four of Sections 3.2-3.3, each with
and without the heavy-first block order when causal), interleaved within a
repetition, each launch after an L2 + MALL flush, timed with HIP events on the
launch stream; the median is reported, and each mapping relative to swizzled
head-first (the paper's normalisation).  Inputs are N(0,1) bf16 drawn on the
device with a seeded generator: the sweep only times the kernel, and the
largest MHA shape (B8, H128, 128K: 137 GB of Q, K, V, O) is drawn on the GPU
rather than on the host.

    python -m paper_2511_02132_amd.sweep --family mha [--reps 2] [--json OUT.jsonl]
    python -m paper_2511_02132_amd.sweep --family gqa --profile --manifest M.json
        (one launch per variant, for rocprofv3 --pmc; writes the launch order)
    Timed runs make one untimed launch per configuration first.
    python -m paper_2511_02132_amd.sweep --summarise --timing OUT.jsonl
        [--counters DIR --manifest M.json] --out profiles/FILE.md
"""

from __future__ import annotations

import argparse
import csv
import json
import math
import os
import re
import statistics
import sys
import time

MAPPING_NAMES = ["naive_block_first", "naive_head_first", "swizzled_head_first",
                 "swizzled_block_first"]
CONTEXTS = (8192, 32768, 131072)
BATCHES = (1, 2, 4, 8)
MHA_HEADS = (8, 16, 32, 64, 128)
GQA_QHEADS = (32, 64, 128)
GQA_KV_HEADS = 8
D = 128


def variants(causal: bool, d: int = D, backward: bool = False):
    import paper_2511_02132_amd as pa
    return pa.variants(causal, d, backward)


def configs(family: str, contexts, batches, heads, kv_heads=GQA_KV_HEADS):
    for S in contexts:
        for B in batches:
            for H in heads:
                if family == "mha":
                    yield {"B": B, "Hq": H, "Hkv": H, "S": S}
                else:
                    yield {"B": B, "Hq": H, "Hkv": kv_heads, "S": S}


def flops(c, causal, d=D):
    f = 4.0 * c["B"] * c["Hq"] * c["S"] * c["S"] * d
    return f / 2 if causal else f


def parse(argv=None):
    p = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    p.add_argument("--family", choices=("mha", "gqa"), default="mha")
    p.add_argument("--contexts", type=int, nargs="+", default=list(CONTEXTS))
    p.add_argument("--batches", type=int, nargs="+", default=list(BATCHES))
    p.add_argument("--heads", type=int, nargs="+", default=None,
                   help="query heads (default: the paper's list for the family)")
    p.add_argument("--kv-heads", type=int, default=GQA_KV_HEADS,
                   help="KV heads of the gqa family (1: one GPU's shard when heads are split by KV head)")
    p.add_argument("--non-causal", action="store_true")
    p.add_argument("--d", type=int, default=D, choices=(56, 64, 128), help="head dimension")
    p.add_argument("--pass", dest="which", choices=("fwd", "bwd"), default="fwd")
    p.add_argument("--reps", type=int, default=5,
                   help="interleaved timed launches per variant, at least")
    p.add_argument("--min-timed-ms", type=float, default=1500.0,
                   help="more reps (up to --max-reps) until each variant has about this much "
                        "timed launch time")
    p.add_argument("--max-reps", type=int, default=20)
    p.add_argument("--warmup-ms", type=float, default=1000.0,
                   help="untimed launches for this long before the first configuration: the "
                        "shader clock of a process's first few hundred milliseconds runs low")
    p.add_argument("--json", default=None, help="append one JSON line per configuration")
    p.add_argument("--profile", action="store_true")
    p.add_argument("--manifest", default=None)
    p.add_argument("--summarise", action="store_true")
    p.add_argument("--timing", nargs="*", default=[])
    p.add_argument("--counters", nargs="*", default=[],
                   help="counter directories of --profile runs, one per --manifests entry")
    p.add_argument("--manifests", nargs="*", default=[],
                   help="the manifests of those runs (summary mode; a later run's launch of a "
                        "configuration replaces an earlier one)")
    p.add_argument("--out", default=None)
    p.add_argument("--cmd", default="")
    p.add_argument("--note", default="", help="extra paragraph for the summary")
    a = p.parse_args(argv)
    if a.heads is None:
        a.heads = list(MHA_HEADS if a.family == "mha" else GQA_QHEADS)
    return a


def iqr(xs) -> float:
    """Interquartile range (linear interpolation between order statistics)."""
    ys = sorted(xs)

    def q(p):
        x = p * (len(ys) - 1)
        i = int(math.floor(x))
        j = min(i + 1, len(ys) - 1)
        return ys[i] + (ys[j] - ys[i]) * (x - i)
    return q(0.75) - q(0.25)


def compare(r, x, y):
    """+1 if variant x is faster than y in record r by more than the spread of
    either (the larger interquartile range of the two launch times), -1 if
    slower by more than that, 0 otherwise (within the spread).  Records
    without spreads compare medians."""
    mx, my = r["ms"][x], r["ms"][y]
    spread = max(r.get("ms_iqr", {}).get(x, 0.0), r.get("ms_iqr", {}).get(y, 0.0))
    if my - mx > spread:
        return 1
    if mx - my > spread:
        return -1
    return 0


def run(a):
    import torch

    import paper_2511_02132_amd as pa

    causal = not a.non_causal
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream(dev)
    flush = torch.empty(512 * 2 ** 20, dtype=torch.uint8, device=dev)
    gen = torch.Generator(device=dev)
    vs = variants(causal, a.d, a.which == "bwd")
    manifest = []
    out = open(a.json, "a") if a.json else None
    for ci, c in enumerate(configs(a.family, a.contexts, a.batches, a.heads, a.kv_heads)):
        gen.manual_seed(7919 * ci + 1)
        shape_q = (c["B"], c["Hq"], c["S"], a.d)
        shape_kv = (c["B"], c["Hkv"], c["S"], a.d)
        q = torch.randn(shape_q, generator=gen, device=dev, dtype=torch.bfloat16)
        k = torch.randn(shape_kv, generator=gen, device=dev, dtype=torch.bfloat16)
        v = torch.randn(shape_kv, generator=gen, device=dev, dtype=torch.bfloat16)
        o = torch.empty_like(q)
        scale = 1.0 / a.d ** 0.5
        times = {n: [] for n, _ in vs}
        reps = 1 if a.profile else a.reps
        if a.which == "bwd":
            do = torch.randn(shape_q, generator=gen, device=dev, dtype=torch.bfloat16)
            o, lse = pa.attn_fwd_lse(q, k, v, o, causal=causal, scale=scale, stream=stream)
            grads = (torch.empty_like(q), torch.empty_like(k), torch.empty_like(v),
                     torch.empty((c["B"], c["Hq"], c["S"]), dtype=torch.float32, device=dev))

        def launch(m):
            if a.which == "bwd":
                pa.attn_bwd(q, k, v, o, do, lse, *grads, causal=causal, scale=scale, mapping=m,
                            stream=stream)
            else:
                pa.attn_fwd(q, k, v, o, causal=causal, scale=scale, mapping=m, stream=stream)
        if not a.profile:
            # untimed launches: the first launch on fresh buffers runs slow, and
            # the shader clock runs low early in a process (a time, not a count)
            t_end = time.perf_counter() + (a.warmup_ms / 1e3 if ci == 0 else 0.0)
            while True:
                launch(vs[0][1])
                torch.cuda.synchronize()
                if time.perf_counter() >= t_end:
                    break
        if not a.profile:
            # reps from the duration of one launch: short configurations get more
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            launch(vs[0][1])
            e1.record(stream)
            torch.cuda.synchronize()
            est = max(e0.elapsed_time(e1), 1e-3)
            reps = min(max(a.reps, int(math.ceil(a.min_timed_ms / est))), max(a.max_reps, a.reps))
        for rep in range(reps):
            if not a.profile and est * len(vs) > 5000:
                print("  %s rep %d/%d" % (json.dumps(c), rep + 1, reps), file=sys.stderr, flush=True)
            for name, m in vs:
                flush.zero_()
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record(stream)
                launch(m)
                e1.record(stream)
                if a.profile:
                    manifest.append({"config": c, "variant": name})
                torch.cuda.synchronize()
                times[name].append(e0.elapsed_time(e1))
        f = flops(c, causal, a.d) * (2.5 if a.which == "bwd" else 1.0)
        rec = {"family": a.family, "pass": a.which, "causal": causal, **c, "d": a.d,
               "reps": reps,
               "ms": {n: round(statistics.median(t), 4) for n, t in times.items()},
               "ms_min": {n: round(min(t), 4) for n, t in times.items()},
               "ms_iqr": {n: round(iqr(t), 4) for n, t in times.items()},
               "tflops": {n: round(f / statistics.median(t) / 1e9, 1) for n, t in times.items()}}
        line = json.dumps(rec)
        print(line, flush=True)
        if out:
            out.write(line + "\n")
            out.flush()
        del q, k, v, o
        if a.which == "bwd":
            del do, lse, grads
        torch.cuda.empty_cache()
    if a.profile:
        # a plain copy of known size (256 MiB, twice): scales FETCH_SIZE / WRITE_SIZE to bytes
        src = torch.ones(256 * 2 ** 20, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(2):
            dst.copy_(src)
        torch.cuda.synchronize()
    if a.profile and a.manifest:
        with open(a.manifest, "w") as fm:
            json.dump(manifest, fm)


# ------------------------------------------------------------------ summary


def _variant_of(kernel_name: str):
    from paper_2511_02132_amd.rocprof_counters import variant_of

    return variant_of(kernel_name)


# gradient kernels: attn_bwd_dkdv_kernel<causal, mapping, order>, attn_bwd_dq_kernel<causal,
# mapping, order> (the dK/dV kernel carries only the block-major bit)
BWD_RE = re.compile(r"attn_bwd_(dkdv|dq)_kernel<(true|false), (\d), (\d)>")


L2_COUNTERS = ("TCC_HIT", "TCC_MISS", "TCC_READ", "TCC_WRITE")


def l2_by_launch(counters_dir: str, manifest_path: str):
    """{(B, Hq, Hkv, S, variant): l2 hit rate} from a --profile run under rocprofv3 --pmc."""
    return {k: v["TCC_HIT"] / max(v["TCC_HIT"] + v["TCC_MISS"], 1.0)
            for k, v in l2_counters_by_launch(counters_dir, manifest_path).items()}


def l2_read_bounds_by_launch(counters_dir: str, manifest_path: str):
    """{(B, Hq, Hkv, S, variant): [low, high]} bounds on the L2 hit rate of read
    requests alone, where the run also counted TCC_READ and TCC_WRITE."""
    from paper_2511_02132_amd.rocprof_counters import read_hit_bounds
    out = {}
    for k, v in l2_counters_by_launch(counters_dir, manifest_path).items():
        if v.get("TCC_READ"):
            out[k] = read_hit_bounds(v["TCC_HIT"], v["TCC_READ"], v.get("TCC_WRITE", 0.0))
    return out


def l2_counters_by_launch(counters_dir: str, manifest_path: str):
    """{(B, Hq, Hkv, S, variant): {counter: value}} of the L2 counters of each launch.

    For the backward, one manifest entry is one attn_bwd call: its dK/dV and
    dQ dispatches are summed (the D kernel is the same for every mapping)."""
    rows = {}
    with open(os.path.join(counters_dir, "run_counter_collection.csv")) as f:
        for r in csv.DictReader(f):
            name = r["Kernel_Name"]
            v = _variant_of(name)
            kind = "fwd"
            if v is None:
                m = BWD_RE.search(name)
                if m is None:
                    continue
                kind = m.group(1)
                from paper_2511_02132_amd.rocprof_counters import order_suffix
                v = MAPPING_NAMES[int(m.group(3))] + order_suffix(int(m.group(4)))
            d = rows.setdefault(int(r["Dispatch_Id"]), {"variant": v, "kind": kind})
            d[r["Counter_Name"]] = d.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    launches = [rows[k] for k in sorted(rows)]
    manifest = json.load(open(manifest_path))
    if any(rec["kind"] == "dkdv" for rec in launches):
        # backward run: drop the forward that made O and lse, and pair each dQ
        # dispatch with the dK/dV dispatch before it
        merged = []
        for rec in launches:
            if rec["kind"] == "fwd":
                continue
            if rec["kind"] == "dkdv":
                merged.append(dict(rec))
            else:
                prev = merged[-1]
                for key in L2_COUNTERS:
                    if key in rec:
                        prev[key] = prev.get(key, 0.0) + rec[key]
                prev["variant"] = rec["variant"]   # the dQ kernel carries every order bit
        launches = merged
    if len(launches) != len(manifest):
        raise ValueError("%d attention launches in the counters, %d in the manifest"
                         % (len(launches), len(manifest)))
    out = {}
    for rec, m in zip(launches, manifest):
        if rec["variant"] != m["variant"]:
            raise ValueError("launch order differs from the manifest")
        c = m["config"]
        vals = {key: rec[key] for key in L2_COUNTERS if key in rec}
        vals.setdefault("TCC_HIT", 0.0)
        vals.setdefault("TCC_MISS", 0.0)
        out[(c["B"], c["Hq"], c["Hkv"], c["S"], m["variant"])] = vals
    return out


def comparisons(recs, names, sh, causal):
    """Win / tie / loss counts of the paper's mapping against block-first, a
    win counting only when the gap exceeds the larger interquartile range of
    the two variants' launch times (compare)."""
    if not recs:
        return []
    spreads = "ms_iqr" in recs[0]
    out = ["", "Comparisons per configuration (%s):" % (
        "a win or a loss only where the gap of the medians exceeds the larger interquartile "
        "range of the two variants' launch times; otherwise a tie" if spreads else
        "medians only: these records carry no spread"), ""]
    pairs = [("swizzled_head_first", "naive_block_first", "same (increasing) block order")]
    if causal:
        pairs.append(("swizzled_head_first+heavy_first", "naive_block_first+heavy_first",
                      "same (heavy-first) block order"))
        pairs.append(("swizzled_head_first+heavy_first+paired",
                      "naive_block_first+heavy_first+paired", "same (paired) block order"))
    best_bf = [n for n in ("naive_block_first", "swizzled_block_first") + (
        ("naive_block_first+heavy_first", "swizzled_block_first+heavy_first",
         "naive_block_first+heavy_first+paired", "swizzled_block_first+heavy_first+paired")
        if causal else ()) if n in names]
    heads = [n for n in ("swizzled_head_first+heavy_first" if causal else "swizzled_head_first",
                         "swizzled_head_first+heavy_first+xcd_block_major" if causal else
                         "swizzled_head_first+xcd_block_major",
                         "swizzled_head_first+heavy_first+paired") if n in names]
    out += ["| comparison | wins | ties | losses | losses (ratio of medians) |", "|---|---|---|---|---|"]

    def row(label, res):
        w = sum(1 for x in res if x[0] > 0)
        t = sum(1 for x in res if x[0] == 0)
        lo = [x for x in res if x[0] < 0]
        det = ", ".join("%dK B%d H%d/%d %.3f" % (r["S"] // 1024, r["B"], r["Hq"], r["Hkv"], q)
                        for _, r, q in lo) or "-"
        out.append("| %s | %d | %d | %d | %s |" % (label, w, t, len(lo), det))

    for x, y, how in pairs:
        if x in names and y in names:
            row("%s vs %s (%s)" % (sh(x), sh(y), how),
                [(compare(r, x, y), r, r["ms"][y] / r["ms"][x]) for r in recs])
    for x in heads:
        res = []
        for r in recs:
            y = min(best_bf, key=lambda n: r["ms"][n])
            res.append((compare(r, x, y), r, r["ms"][y] / r["ms"][x]))
        row("%s vs the fastest block-first order of each configuration (%s)" % (
            sh(x), ", ".join(sh(n) for n in best_bf)), res)
    if spreads:
        worst = max(max(r["ms_iqr"][n] / r["ms"][n] for n in names) for r in recs)
        out += ["", "Largest interquartile range of a variant's launch times: %.1f%% of its "
                "median." % (100 * worst)]
    return out


def summarise(a):
    recs = {}
    for path in a.timing:   # a later file's record of a configuration replaces an earlier one
        with open(path) as f:
            for x in f:
                if x.strip():
                    r = json.loads(x)
                    recs[(r["S"], r["B"], r["Hq"], r["Hkv"])] = r
    recs = [recs[k] for k in sorted(recs)]
    manifests = a.manifests or ([a.manifest] if a.manifest else [])
    if len(manifests) != len(a.counters):
        raise SystemExit("--counters and --manifests must pair up")
    l2, l2r = {}, {}
    for cdir, man in zip(a.counters, manifests):
        l2.update(l2_by_launch(cdir, man))
        l2r.update(l2_read_bounds_by_launch(cdir, man))
    causal = recs[0]["causal"] if recs else True
    which = recs[0].get("pass", "fwd") if recs else "fwd"
    names = [n for n, _ in variants(causal, recs[0].get("d", D) if recs else D, which == "bwd")]
    short = {"naive_block_first": "NBF", "naive_head_first": "NHF", "swizzled_head_first": "SHF",
             "swizzled_block_first": "SBF"}

    def sh(n):
        parts = n.split("+")
        return short[parts[0]] + ("+hf" if "heavy_first" in parts else "") + \
            ("+bm" if "xcd_block_major" in parts else "") + ("+p" if "paired" in parts else "")

    import paper_2511_02132_amd as pa
    base = pa.variant_name(pa.method_variant(causal))
    if recs and base not in recs[0]["tflops"]:   # records taken before the block-major order
        base = "swizzled_head_first" + ("+heavy_first" if causal else "")
    names = [n for n in names if not recs or n in recs[0]["tflops"]]
    lines = ["# Mapping sweep: %s %s, d=%d, %s" % (
        recs[0]["family"].upper() if recs else "?", "backward" if which == "bwd" else "forward",
        recs[0].get("d", D) if recs else D, "causal" if causal else "non-causal"), ""]
    if which == "bwd":
        lines += ["TFLOP/s of the gradient kernels (D, dK/dV, dQ) in the FlashAttention "
                  "convention: 2.5x the forward's 4*B*Hq*S*S*d (halved when causal).", ""]
    lines += ["Each cell: TFLOP/s (median of the interleaved, L2+MALL-flushed launches), then "
              "relative to %s.  reps: timed launches per variant; max IQR: the largest "
              "interquartile range of a variant's launch times, relative to its median." % base]
    if l2:
        lines += ["Second table: L2 hit rate of one launch per variant (rocprofv3 TCC_HIT / "
                  "(TCC_HIT + TCC_MISS))."]
    if l2r:
        lines += ["Third table: bounds on the L2 hit rate of read requests alone (TCC_HIT, "
                  "TCC_READ, TCC_WRITE: between no write hitting and every write hitting)."]
    lines += ["", "Variants: NBF naive block-first, NHF naive head-first, SHF swizzled head-first "
              "(the method), SBF swizzled block-first; +hf = heavy-first block order, +bm = "
              "block-major order in groups of four heads inside each XCD's piece, +p = paired "
              "row blocks (one workgroup per pair NB-1-p, p of a head).", ""]
    if a.note:
        lines += [a.note, ""]
    if a.cmd:
        lines += ["Commands:", "", "```", a.cmd, "```", ""]
    hdr = "| S | B | Hq/Hkv | " + " | ".join(sh(n) for n in names) + " |"
    reps_col = bool(recs) and "reps" in recs[0]
    lines += [hdr[:-1] + ("| reps | max IQR |" if reps_col else "|"),
              "|" + "---|" * (3 + len(names) + (2 if reps_col else 0))]
    for r in recs:
        ref = r["tflops"][base]
        cells = ["%.0f (%.2f)" % (r["tflops"][n], r["tflops"][n] / ref) for n in names]
        if reps_col:
            cells += [str(r["reps"]), "%.1f%%" % (100 * max(r["ms_iqr"][n] / r["ms"][n]
                                                            for n in names))]
        lines.append("| %dK | %d | %d/%d | %s |" % (r["S"] // 1024, r["B"], r["Hq"], r["Hkv"],
                                                   " | ".join(cells)))
    if l2:
        lines += ["", hdr, "|" + "---|" * (3 + len(names))]
        for r in recs:
            cells = []
            for n in names:
                h = l2.get((r["B"], r["Hq"], r["Hkv"], r["S"], n))
                cells.append("-" if h is None else "%.1f%%" % (100 * h))
            lines.append("| %dK | %d | %d/%d | %s |" % (r["S"] // 1024, r["B"], r["Hq"], r["Hkv"],
                                                       " | ".join(cells)))
    if l2r:
        lines += ["", hdr, "|" + "---|" * (3 + len(names))]
        for r in recs:
            cells = []
            for n in names:
                b = l2r.get((r["B"], r["Hq"], r["Hkv"], r["S"], n))
                cells.append("-" if b is None else "%.1f..%.1f%%" % (100 * b[0], 100 * b[1]))
            lines.append("| %dK | %d | %d/%d | %s |" % (r["S"] // 1024, r["B"], r["Hq"], r["Hkv"],
                                                       " | ".join(cells)))
    # geometric-mean speed relative to the method, per variant
    lines += ["", "Geometric mean over the configurations, relative to %s:" % base, ""]
    for n in names:
        g = math.exp(sum(math.log(r["tflops"][n] / r["tflops"][base]) for r in recs) / len(recs))
        lines.append("- %s: %.3f" % (n, g))
    lines += comparisons(recs, names, sh, causal)
    text = "\n".join(lines) + "\n"
    if a.out:
        with open(a.out, "w") as f:
            f.write(text)
    print(text)


def main(argv=None):
    a = parse(argv)
    if a.summarise:
        summarise(a)
    else:
        run(a)


if __name__ == "__main__":
    sys.exit(main())
