"""Summarise rocprofv3 counter passes of ``bench.py --profile`` into profiles/.

Each pass directory holds one rocprofv3 run (``-d DIR -o run -f csv json``) of

    rocprofv3 --pmc <counters> -d DIR -o run -f csv json -- python3 bench.py --profile --workload W

Every (mapping, block order) of the attention kernel is its own kernel symbol
(``attn_fwd_kernel<d, stored d, causal, mapping, order>`` or, for d = 128,
``attn_fwd_pp_kernel<causal, mapping, order>``), so one run per pass
covers all variants.  The run also holds a one-workgroup launch (it can only
run on XCD 0) and a 256 MiB device copy, used to attribute counter instances
to XCDs and to scale FETCH_SIZE / WRITE_SIZE to bytes.

    python -m paper_2511_02132_amd.rocprof_counters --workload W --out FILE.md \\
        --cmd "<pass commands>" DIR_A DIR_B ...

The summary ends with a ```json block that bench.py reads (only when its
kernel_source_sha256 matches the current kernel sources).
"""

from __future__ import annotations

import argparse
import csv
import json
import os
import re
import sys
from collections import defaultdict

MAPPING_NAMES = ["naive_block_first", "naive_head_first", "swizzled_head_first",
                 "swizzled_block_first"]
# attn_fwd_kernel<d, stored d, causal, mapping, order> (4-wave kernel) and
# attn_fwd_pp_kernel<causal, mapping, order> (d = 128 two-group kernel); order
# bit 0 = heavy-first, bit 1 = block-major inside each XCD's piece, bit 2 =
# paired row blocks
KERNEL_RE = re.compile(r"attn_fwd_(?:kernel<\d+, \d+, |pp_kernel<)(true|false), (\d), (\d)>")


def order_suffix(order: int) -> str:
    return ("+heavy_first" if order & 1 else "") + ("+xcd_block_major" if order & 2 else "") + \
        ("+paired" if order & 4 else "")


def variant_of(kernel_name: str):
    m = KERNEL_RE.search(kernel_name)
    if not m:
        return None
    return MAPPING_NAMES[int(m.group(2))] + order_suffix(int(m.group(3)))


# backward kernels: attn_bwd_dkdv_kernel<causal, mapping, order>, attn_bwd_dq_kernel<...>
BWD_KERNEL_RE = re.compile(r"attn_bwd_(dkdv|dq)_kernel<(true|false), (\d), (\d)>")


def kernel_of(kernel_name: str):
    """Display name of an attention kernel: the forward's variant, 'dK/dV <variant>'
    or 'dQ <variant>' for the backward's gradient kernels, 'D' for its row-statistics
    kernel; None for any other kernel."""
    v = variant_of(kernel_name)
    if v is not None:
        return v
    m = BWD_KERNEL_RE.search(kernel_name)
    if m:
        # the dK/dV kernel carries only the block-major bit of the order
        return ("dK/dV " if m.group(1) == "dkdv" else "dQ ") + \
            MAPPING_NAMES[int(m.group(3))] + order_suffix(int(m.group(4)))
    if "attn_bwd_delta_kernel" in kernel_name:
        return "D"
    return None


def summarise_kernels(dirs):
    """{kernel display name: {counter: mean per dispatch}} over every dispatch of
    the passes in dirs, plus the copy-kernel scale factors of FETCH_SIZE and
    WRITE_SIZE (from a 256 MiB device copy in the run)."""
    acc = defaultdict(lambda: defaultdict(list))
    copy = defaultdict(list)
    for d in dirs:
        for did, kname, grid, cname, val in read_csv(d):
            k = kernel_of(kname)
            if k is not None:
                acc[k][cname].append(val)
            elif "copy" in kname.lower():
                copy[cname].append(val)
    copy_bytes = 256 * 2 ** 20
    fac = {c: copy_bytes / (sum(v) / len(v) * 1024) for c, v in copy.items()
           if c in ("FETCH_SIZE", "WRITE_SIZE") and v}
    out = {}
    for k, cs in acc.items():
        out[k] = {c: sum(v) / len(v) for c, v in cs.items()}
    return out, fac


def write_kernels_md(out: str, title: str, cmd: str, dirs, note: str = ""):
    """Per-kernel counter table (MFMA utilisation, LDS instructions per MFMA,
    LDS waits, L2 hits, HBM bytes) of the passes in dirs."""
    from paper_2511_02132_amd.build import BWD_KERNEL_SOURCES, kernel_source_hash

    res, fac = summarise_kernels(dirs)
    lines = ["# %s" % title, "", "Commands (run from the repository root; `cd /tmp` first, "
             "paths absolute in the run):", "", "```", cmd.strip(), "```", "",
             "Values are means per dispatch over the dispatches of each kernel in the run.", ""]
    if note:
        lines += [note, ""]
    if fac:
        lines.append("Copy-kernel scale factors (256 MiB device copy): %s." % ", ".join(
            "%s x%.4f" % (c, f) for c, f in sorted(fac.items())))
    lines += ["Kernel source sha256[:16]: forward kernels `%s`, backward kernels `%s`" % (
                  kernel_source_hash(), kernel_source_hash(BWD_KERNEL_SOURCES)), "",
              "| kernel | MFMA util % | MFMA instr | LDS instr | LDS / MFMA | LDS wait / LDS instr "
              "| VALU instr | L2 hit | HBM bytes read | HBM bytes written |",
              "|---|---|---|---|---|---|---|---|---|---|"]

    def f(v, fmt):
        return fmt % v if v is not None else "-"
    for k in sorted(res):
        e = res[k]
        mf, lds = e.get("SQ_INSTS_MFMA"), e.get("SQ_INSTS_LDS")
        hit, miss = e.get("TCC_HIT"), e.get("TCC_MISS")
        rd = e["FETCH_SIZE"] * 1024 * fac["FETCH_SIZE"] if "FETCH_SIZE" in e and "FETCH_SIZE" in fac \
            else None
        wr = e["WRITE_SIZE"] * 1024 * fac["WRITE_SIZE"] if "WRITE_SIZE" in e and "WRITE_SIZE" in fac \
            else None
        lines.append("| %s | %s | %s | %s | %s | %s | %s | %s | %s | %s |" % (
            k, f(e.get("MfmaUtil"), "%.1f"), f(mf, "%.3e"), f(lds, "%.3e"),
            f(lds / mf if lds is not None and mf else None, "%.2f"),
            f(e["SQ_WAIT_INST_LDS"] / lds if "SQ_WAIT_INST_LDS" in e and lds else None, "%.2f"),
            f(e.get("SQ_INSTS_VALU"), "%.3e"),
            f(100.0 * hit / (hit + miss) if hit is not None and miss is not None and hit + miss > 0
              else None, "%.1f%%"),
            f(rd, "%.3e"), f(wr, "%.3e")))
    data = {"kernel_source_sha256": kernel_source_hash(),
            "bwd_kernel_source_sha256": kernel_source_hash(BWD_KERNEL_SOURCES), "scale": fac,
            "per_kernel": res}
    lines += ["", "```json", json.dumps(data, indent=1, sort_keys=True), "```", ""]
    with open(out, "w") as fh:
        fh.write("\n".join(lines))


def read_csv(d: str):
    """rows of run_counter_collection.csv: (dispatch, kernel, grid, counter, value)."""
    path = os.path.join(d, "run_counter_collection.csv")
    out = []
    with open(path) as f:
        for row in csv.DictReader(f):
            out.append((int(row["Dispatch_Id"]), row["Kernel_Name"], int(row["Grid_Size"]),
                        row["Counter_Name"], float(row["Counter_Value"])))
    return out


def per_xcc(d: str, counters=("TCC_HIT", "TCC_MISS")):
    """{dispatch_id: {counter: [sum over the instances of XCC x for x in 0..7]}} from the JSON.

    Records of a dispatch carry only the counter id; they are taken in the
    order of that counter's instance list, whose dimension indices give the
    XCC.  The one-workgroup launch checks this attribution."""
    path = os.path.join(d, "run_results.json")
    if not os.path.exists(path):
        return {}
    root = json.load(open(path))["rocprofiler-sdk-tool"][0]
    inst = {}
    names = {}
    for c in root["counters"]:
        cid = c["id"]["handle"]
        names[cid] = c["name"]
        xcc = []
        for i in c["instances"]:
            dims = {x["dimension_name"]: x["index"] for x in i["dimensions"]}
            xcc.append(dims.get("DIMENSION_XCC", 0))
        inst[cid] = xcc
    out = {}
    for rec in root["callback_records"]["counter_collection"]:
        did = rec["dispatch_data"]["dispatch_info"]["dispatch_id"]
        pos = defaultdict(int)
        sums = defaultdict(lambda: [0.0] * 8)
        for r in rec["records"]:
            cid = r["counter_id"]["handle"]
            k = pos[cid]
            pos[cid] += 1
            if names.get(cid) in counters and k < len(inst[cid]):
                sums[names[cid]][inst[cid][k]] += r["value"]
        out[did] = dict(sums)
    return out


def read_hit_bounds(hit: float, read: float, write: float):
    """Bounds on the L2 hit rate of read requests alone.

    The counters give hits and misses of all requests (TCC_HIT, TCC_MISS) and
    the number of read and write requests (TCC_READ, TCC_WRITE), but not how
    the hits split between reads and writes.  Every hit is a read hit when no
    write hits (upper bound), and at most TCC_WRITE hits are write hits (lower
    bound).  The all-request rate depends on how stores are split into
    requests; this one measures the reuse of what the kernel reads."""
    if read <= 0:
        return None
    return [round(max(0.0, hit - write) / read, 4), round(min(1.0, hit / read), 4)]


def summarise(dirs, workload: str):
    per_variant = defaultdict(lambda: defaultdict(list))
    copy = defaultdict(list)
    one_wg_dispatches = []
    xcc_tables = {}
    for d in dirs:
        rows = read_csv(d)
        for did, kname, grid, cname, val in rows:
            v = variant_of(kname)
            if v is not None and grid <= 512:   # the one-workgroup launch
                one_wg_dispatches.append((d, did))
                continue
            if v is not None:
                per_variant[v][cname].append((d, did, val))
            elif "copy" in kname.lower():
                copy[cname].append(val)
        xcc_tables[d] = per_xcc(d)

    def mean(vals):
        return sum(vals) / len(vals) if vals else None

    copy_bytes = 256 * 2 ** 20
    fetch_fac = write_fac = None
    if copy.get("FETCH_SIZE"):
        fetch_fac = copy_bytes / (mean(copy["FETCH_SIZE"]) * 1024)
    if copy.get("WRITE_SIZE"):
        write_fac = copy_bytes / (mean(copy["WRITE_SIZE"]) * 1024)

    # XCC attribution check on the one-workgroup launch
    xcc0_share = None
    for d, did in one_wg_dispatches:
        t = xcc_tables.get(d, {}).get(did)
        if t and "TCC_HIT" in t:
            tot = [t["TCC_HIT"][x] + t.get("TCC_MISS", [0] * 8)[x] for x in range(8)]
            if sum(tot) > 0:
                xcc0_share = tot[0] / sum(tot)

    result = {}
    for v, cs in sorted(per_variant.items()):
        ent = {}
        vals = {c: mean([x[2] for x in lst]) for c, lst in cs.items()}
        if "TCC_HIT" in vals and "TCC_MISS" in vals:
            ent["l2_hit_rate"] = round(vals["TCC_HIT"] / (vals["TCC_HIT"] + vals["TCC_MISS"]), 4)
            xs = []
            for (d, did, _) in cs["TCC_HIT"]:
                t = xcc_tables.get(d, {}).get(did)
                if t and "TCC_HIT" in t and "TCC_MISS" in t:
                    xs.append([t["TCC_HIT"][x] / max(1.0, t["TCC_HIT"][x] + t["TCC_MISS"][x])
                               for x in range(8)])
            if xs:
                ent["l2_hit_rate_per_xcd"] = [round(sum(col) / len(col), 4) for col in zip(*xs)]
            if vals.get("TCC_READ") and "TCC_WRITE" in vals:
                ent["l2_read_hit_rate_bounds"] = read_hit_bounds(
                    vals["TCC_HIT"], vals["TCC_READ"], vals["TCC_WRITE"])
                ent["l2_requests_read_write_over_hit_miss"] = round(
                    (vals["TCC_READ"] + vals["TCC_WRITE"]) /
                    max(1.0, vals["TCC_HIT"] + vals["TCC_MISS"]), 4)
        for c in ("TCC_HIT", "TCC_MISS", "TCC_READ", "TCC_WRITE", "TCC_EA0_RDREQ", "TCC_EA0_RDREQ_32B",
                  "TCC_EA0_RDREQ_DRAM", "SQ_INSTS_VALU", "SQ_INSTS_MFMA", "SQ_INSTS_LDS",
                  "SQ_LDS_BANK_CONFLICT", "SQ_WAIT_INST_LDS", "SQ_ACTIVE_INST_VALU",
                  "SQ_VALU_MFMA_BUSY_CYCLES", "GRBM_GUI_ACTIVE"):
            if c in vals:
                ent[c.lower()] = vals[c]
        if "MfmaUtil" in vals:
            ent["mfma_util_pct"] = round(vals["MfmaUtil"], 2)
        if "FETCH_SIZE" in vals:
            ent["fetch_kib"] = vals["FETCH_SIZE"]
        if "WRITE_SIZE" in vals:
            ent["write_kib"] = vals["WRITE_SIZE"]
        if fetch_fac and write_fac and "FETCH_SIZE" in vals and "WRITE_SIZE" in vals:
            ent["hbm_bytes_per_launch"] = int(vals["FETCH_SIZE"] * 1024 * fetch_fac +
                                              vals["WRITE_SIZE"] * 1024 * write_fac)
        result[v] = ent
    return result, fetch_fac, write_fac, xcc0_share


def compulsory_bytes(workload: str) -> int:
    sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
    import attn_inputs as ai
    w = ai.WORKLOADS[workload]
    qo = 2 * w["B"] * w["Hq"] * w["Sq"] * w["d"] * 2
    kv = 2 * w["B"] * w["Hkv"] * w["Skv"] * w["d"] * 2
    return qo + kv


def write_md(out: str, workload: str, cmd: str, result, fetch_fac, write_fac, xcc0_share):
    from paper_2511_02132_amd.build import kernel_source_hash

    comp = compulsory_bytes(workload)
    lines = ["# attn_fwd counters: %s" % workload, "",
             "rocprofv3 counter passes over `bench.py --profile` (2 launches per variant; "
             "values are per launch, averaged).", "",
             "Commands (run from the repository root; `cd /tmp` first, "
             "paths absolute in the run):", "", "```", cmd.strip(), "```", "",
             "Compulsory HBM bytes (Q, K, V read once, O written once): %d (%.1f MiB)."
             % (comp, comp / 2 ** 20), ""]
    if fetch_fac:
        lines.append("Copy-kernel scale factors (256 MiB device copy): FETCH_SIZE x%.4f, "
                     "WRITE_SIZE x%.4f." % (fetch_fac, write_fac or float('nan')))
    if xcc0_share is not None:
        lines.append("XCD attribution check: %.4f of the one-workgroup launch's L2 requests "
                     "land on XCD 0 instances." % xcc0_share)
    lines += ["L2 read hit: bounds on the hit rate of read requests alone, from TCC_HIT, "
              "TCC_READ and TCC_WRITE (between no write hitting and every write hitting).", ""]
    lines += ["", "| variant | L2 hit | L2 read hit | L2 hit per XCD (min..max) | HBM bytes / launch | "
                  "/ compulsory | MFMA util % | LDS instr / MFMA | LDS bank-conflict cycles |",
              "|---|---|---|---|---|---|---|---|---|"]
    for v, e in result.items():
        px = e.get("l2_hit_rate_per_xcd")
        hb = e.get("hbm_bytes_per_launch")
        rb = e.get("l2_read_hit_rate_bounds")
        lines.append("| %s | %s | %s | %s | %s | %s | %s | %s | %s |" % (
            v, "%.1f%%" % (100 * e["l2_hit_rate"]) if "l2_hit_rate" in e else "-",
            "%.1f..%.1f%%" % (100 * rb[0], 100 * rb[1]) if rb else "-",
            "%.1f..%.1f%%" % (100 * min(px), 100 * max(px)) if px else "-",
            "%.3e" % hb if hb else "-", "%.2f" % (hb / comp) if hb else "-",
            e.get("mfma_util_pct", "-"),
            "%.2f" % (e["sq_insts_lds"] / e["sq_insts_mfma"])
            if e.get("sq_insts_mfma") and "sq_insts_lds" in e else "-",
            "%.3e" % e["sq_lds_bank_conflict"]
            if "sq_lds_bank_conflict" in e else "-"))
    data = {"workload": workload, "kernel_source_sha256": kernel_source_hash(),
            "compulsory_bytes": comp, "fetch_scale": fetch_fac, "write_scale": write_fac,
            "xcc0_share_one_wg": xcc0_share, "per_mapping": result}
    lines += ["", "```json", json.dumps(data, indent=1, sort_keys=True), "```", ""]
    with open(out, "w") as f:
        f.write("\n".join(lines))


def write_stats_md(out: str, stats_csv: str, bench_json: str, cmd: str):
    """Kernel-trace statistics of a bench.py run next to the bench line it printed."""
    from paper_2511_02132_amd.build import kernel_source_hash

    rows = list(csv.DictReader(open(stats_csv)))
    line = open(bench_json).read().strip().splitlines()[-1]
    bench = json.loads(line)
    head = bench["config"]["mapping"]
    lines = ["# attn_fwd kernel trace: %s" % bench["config"]["workload"], "",
             "Command (run from the repository root; `cd /tmp` first, paths absolute):", "",
             "```", cmd.strip(), "```", "",
             "Kernel source sha256[:16]: `%s`" % kernel_source_hash(), "",
             "| kernel | calls | average us | min us | max us | share |",
             "|---|---|---|---|---|---|"]
    for r in rows:
        v = variant_of(r["Name"]) or r["Name"][:60]
        if variant_of(r["Name"]) and "attn_fwd_kernel<" in r["Name"]:
            v += " (d=64/56 kernel: the small workload)"
        lines.append("| %s | %s | %.1f | %.1f | %.1f | %s%% |" % (
            v, r["Calls"], float(r["AverageNs"]) / 1e3, float(r["MinNs"]) / 1e3,
            float(r["MaxNs"]) / 1e3, r["Percentage"]))
    avg = [float(r["AverageNs"]) / 1e3 for r in rows
           if variant_of(r["Name"]) == head and "attn_fwd_kernel<" not in r["Name"]]
    lines += ["", "Headline variant `%s`: bench.py timed %.1f us per step with HIP events on the "
              "launch stream (its K back-to-back steps); the profiler's average over all "
              "calls of that kernel (warm-up, timed steps and the cold/warm per-mapping reps) "
              "is %s us." % (head, bench["ms_per_step"] * 1e3,
                             "%.1f" % avg[0] if avg else "n/a"),
              "", "bench.py line printed under the profiler:", "", "```json", line, "```", ""]
    with open(out, "w") as f:
        f.write("\n".join(lines))


def write_bwd_stats_md(out: str, title: str, stats_csv: str, cmd: str, shape, note: str = ""):
    """Kernel-trace statistics of the backward's kernels (D, dK/dV and dQ per
    variant) and the headline variant's total.  shape: (B, Hq, S) of the run,
    causal, head dimension 128."""
    import paper_2511_02132_amd as pa
    from paper_2511_02132_amd.build import BWD_KERNEL_SOURCES, kernel_source_hash

    rows = []
    for r in csv.DictReader(open(stats_csv)):
        k = kernel_of(r["Name"])
        if k is None or not (k == "D" or k.startswith("dK/dV ") or k.startswith("dQ ")):
            continue
        rows.append((k, int(r["Calls"]), float(r["AverageNs"]) / 1e3, float(r["MinNs"]) / 1e3,
                     float(r["MaxNs"]) / 1e3))
    order = {"D": 0, "dK/dV": 1, "dQ": 2}
    rows.sort(key=lambda x: (order[x[0].split(" ")[0]], x[2]))
    lines = ["# %s" % title, "", "Command (run from the repository root; `cd /tmp` first, "
             "paths absolute in the run):", "", "```", cmd.strip(), "```", ""]
    if note:
        lines += [note, ""]
    lines += ["Backward kernel source sha256[:16]: `%s`" % kernel_source_hash(BWD_KERNEL_SOURCES),
              "", "| kernel | calls | average us | min us | max us |", "|---|---|---|---|---|"]
    for k, n, avg, mn, mx in rows:
        lines.append("| %s | %d | %.1f | %.1f | %.1f |" % (k, n, avg, mn, mx))
    head = pa.method_variant(True)
    dq_name = "dQ " + pa.variant_name(head)
    # the dK/dV kernel takes only the block-major bit of the order
    dkdv_name = "dK/dV " + pa.variant_name(head & ~pa.HEAVY_FIRST)
    avg = {k: a for k, _, a, _, _ in rows}
    if all(x in avg for x in ("D", dkdv_name, dq_name)):
        B, Hq, S = shape
        total = avg["D"] + avg[dkdv_name] + avg[dq_name]
        fl = 2.5 * pa.attention_flops(B, Hq, S, S, 128, True)
        lines += ["", "Headline variant `%s` (the dK/dV kernel takes only the block-major bit "
                  "of the order: its natural order already starts with the heaviest causal key "
                  "block): D %.1f + dK/dV %.1f + dQ %.1f = %.1f us, %.0f TFLOP/s in the "
                  "FlashAttention convention (2.5x the forward flops); the dK/dV kernel, counting "
                  "its four products (twice the forward flops), runs at %.0f TFLOP/s." % (
                      pa.variant_name(head), avg["D"], avg[dkdv_name], avg[dq_name], total,
                      fl / total / 1e6,
                      2.0 * pa.attention_flops(B, Hq, S, S, 128, True) / avg[dkdv_name] / 1e6)]
    lines.append("")
    with open(out, "w") as fh:
        fh.write("\n".join(lines))


def main(argv=None):
    p = argparse.ArgumentParser()
    p.add_argument("--workload")
    p.add_argument("--out", required=True)
    p.add_argument("--cmd", default="", help="the commands that produced the passes")
    p.add_argument("--stats-csv", help="kernel_stats.csv of a --kernel-trace --stats run")
    p.add_argument("--bench-json", help="the bench.py output of that run")
    p.add_argument("--per-kernel", metavar="TITLE",
                   help="write a per-kernel counter table (any attention kernels, the "
                        "backward's included) with this title")
    p.add_argument("--note", default="")
    p.add_argument("--bwd-trace", metavar="TITLE",
                   help="with --stats-csv: a backward kernel-trace table with this title")
    p.add_argument("--shape", type=int, nargs=3, metavar=("B", "HQ", "S"),
                   help="the backward run's shape (causal, d = 128)")
    p.add_argument("dirs", nargs="*")
    a = p.parse_args(argv)
    if a.bwd_trace:
        write_bwd_stats_md(a.out, a.bwd_trace, a.stats_csv, a.cmd, a.shape, a.note)
    elif a.per_kernel:
        write_kernels_md(a.out, a.per_kernel, a.cmd, a.dirs, a.note)
    elif a.stats_csv:
        write_stats_md(a.out, a.stats_csv, a.bench_json, a.cmd)
    else:
        res = summarise(a.dirs, a.workload)
        write_md(a.out, a.workload, a.cmd, *res)
    print(open(a.out).read())


if __name__ == "__main__":
    main()
