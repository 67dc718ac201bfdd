"""CPU tests of the measurement tooling: the kernel-name decoding and counter
arithmetic behind profiles/ (rocprof_counters), the mapping-sweep summary
(sweep), and bench.py's host-side checks.  No GPU is used."""

import json
import math
import os
import subprocess
import sys
from types import SimpleNamespace

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402  (imports torch only inside main())
import paper_2511_02132_amd as pa  # noqa: E402
from paper_2511_02132_amd import rocprof_counters as rc  # noqa: E402
from paper_2511_02132_amd import sweep  # noqa: E402


def _order_bits(mapping):
    return (1 if mapping & pa.HEAVY_FIRST else 0) | (2 if mapping & pa.XCD_BLOCK_MAJOR else 0) | \
        (4 if mapping & pa.PAIRED else 0)


def test_variant_of_kernel_names():
    ns = "void attn::(anonymous namespace)::"
    cases = {
        ns + "attn_fwd_pp_kernel<true, 2, 3>(attn::KernelArgs)":
            "swizzled_head_first+heavy_first+xcd_block_major",
        ns + "attn_fwd_pp_kernel<false, 0, 0>(attn::KernelArgs)": "naive_block_first",
        ns + "attn_fwd_kernel<64, 56, true, 3, 1>(attn::KernelArgs)":
            "swizzled_block_first+heavy_first",
        ns + "attn_fwd_kernel<64, 64, false, 1, 0>(attn::KernelArgs)": "naive_head_first",
        # not forward launches of the dispatched kernels
        ns + "attn_fwd_pp_persistent_kernel<true, 2, 3>(attn::KernelArgs)": None,
        ns + "attn_bwd_dq_kernel<true, 2, 3>(attn::BwdArgs)": None,
        "__amd_rocclr_copyBuffer": None,
    }
    for name, want in cases.items():
        assert rc.variant_of(name) == want, name
    # every variant the measurements compare decodes from its kernel name
    for causal in (False, True):
        for vname, m in pa.variants(causal):
            kname = ns + "attn_fwd_pp_kernel<%s, %d, %d>(attn::KernelArgs)" % (
                "true" if causal else "false", m & 0xF, _order_bits(m))
            assert rc.variant_of(kname) == vname


def _write_counters(d, rows):
    os.makedirs(d, exist_ok=True)
    with open(os.path.join(d, "run_counter_collection.csv"), "w") as f:
        f.write("Dispatch_Id,Kernel_Name,Grid_Size,Counter_Name,Counter_Value\n")
        for did, kname, grid, cname, val in rows:
            f.write('%d,"%s",%d,%s,%r\n' % (did, kname, grid, cname, val))


def test_counter_summary_arithmetic(tmp_path):
    """Hit rate, copy-kernel scale factors and HBM bytes from known counter values."""
    k_swz = "void attn::(anonymous namespace)::attn_fwd_pp_kernel<true, 2, 1>(attn::KernelArgs)"
    k_nbf = "void attn::(anonymous namespace)::attn_fwd_pp_kernel<true, 0, 1>(attn::KernelArgs)"
    copy = "__amd_rocclr_copyBuffer"
    mib256_kib = 256 * 1024
    a = str(tmp_path / "A")
    b = str(tmp_path / "B")
    _write_counters(a, [
        (1, copy, 1 << 20, "TCC_HIT", 5.0),
        (2, k_swz, 512 * 1024, "TCC_HIT", 900.0), (2, k_swz, 512 * 1024, "TCC_MISS", 100.0),
        (3, k_swz, 512 * 1024, "TCC_HIT", 700.0), (3, k_swz, 512 * 1024, "TCC_MISS", 300.0),
        (4, k_nbf, 512 * 1024, "TCC_HIT", 250.0), (4, k_nbf, 512 * 1024, "TCC_MISS", 750.0),
        # a one-workgroup launch (grid <= 512) is the XCD check, not a measurement
        (5, k_swz, 512, "TCC_HIT", 1.0), (5, k_swz, 512, "TCC_MISS", 1e6),
    ])
    _write_counters(b, [
        # the copy kernel's FETCH_SIZE reads half of the 256 MiB it moved
        (1, copy, 1 << 20, "FETCH_SIZE", mib256_kib / 2), (1, copy, 1 << 20, "WRITE_SIZE", mib256_kib),
        (2, k_swz, 512 * 1024, "FETCH_SIZE", 1000.0), (2, k_swz, 512 * 1024, "WRITE_SIZE", 500.0),
        (3, k_swz, 512 * 1024, "FETCH_SIZE", 3000.0), (3, k_swz, 512 * 1024, "WRITE_SIZE", 500.0),
    ])
    result, fetch_fac, write_fac, xcc0 = rc.summarise([a, b], "mha_b1_h32_s8192_d128_causal")
    assert fetch_fac == pytest.approx(2.0) and write_fac == pytest.approx(1.0)
    assert xcc0 is None   # no per-XCC records in these directories
    swz = result["swizzled_head_first+heavy_first"]
    assert swz["l2_hit_rate"] == pytest.approx(0.8)   # (900+700) / 2000
    assert swz["hbm_bytes_per_launch"] == int(2000 * 1024 * 2.0 + 500 * 1024 * 1.0)
    assert result["naive_block_first+heavy_first"]["l2_hit_rate"] == pytest.approx(0.25)
    assert "hbm_bytes_per_launch" not in result["naive_block_first+heavy_first"]


def test_compulsory_bytes():
    # MHA B1 H32 S8192 d128: Q, K, V, O once each, bf16
    assert rc.compulsory_bytes("mha_b1_h32_s8192_d128_causal") == 4 * 32 * 8192 * 128 * 2
    # GQA: K and V have 8 heads
    assert rc.compulsory_bytes("gqa_b1_hq64_hkv8_s8192_d128_causal") == \
        (2 * 64 + 2 * 8) * 8192 * 128 * 2


def test_sweep_summary(tmp_path):
    names = [n for n, _ in pa.variants(True)]
    recs = []
    for i, (S, B) in enumerate([(8192, 1), (32768, 2)]):
        tf = {n: 500.0 + 10 * j + 100 * i for j, n in enumerate(names)}
        recs.append({"family": "mha", "pass": "fwd", "causal": True, "S": S, "B": B, "Hq": 32,
                     "Hkv": 32, "d": 128, "ms": {n: 1.0 for n in names}, "tflops": tf})
    timing = tmp_path / "t.jsonl"
    timing.write_text("".join(json.dumps(r) + "\n" for r in recs))
    out = tmp_path / "s.md"
    args = SimpleNamespace(timing=[str(timing)], counters=[], manifest=None, manifests=[], out=str(out),
                           cmd="CMD", note="NOTE")
    sweep.summarise(args)
    text = out.read_text()
    assert text.startswith("# Mapping sweep: MHA forward, d=128, causal")
    assert "NOTE" in text and "CMD" in text
    rows = [l for l in text.splitlines() if l.startswith("| 8K") or l.startswith("| 32K")]
    assert len(rows) == 2 and all(l.count("|") == 3 + len(names) + 1 for l in rows)
    base = pa.variant_name(pa.method_variant(True))
    for n in names:
        g = math.exp(sum(math.log(r["tflops"][n] / r["tflops"][base]) for r in recs) / 2)
        assert "- %s: %.3f" % (n, g) in text


def test_bench_refuses_several_gpus():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_bench_uses_counters_of_this_kernel_source_only(tmp_path, monkeypatch):
    wl = "mha_b1_h32_s8192_d128_causal"
    os.makedirs(tmp_path / "profiles")
    path = tmp_path / "profiles" / ("attn_fwd_%s_counters.md" % wl)
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.counter_summary(wl) is None   # no summary at all
    for sha, found in ((bench.kernel_source_hash(), True), ("0" * 16, False)):
        data = {"kernel_source_sha256": sha, "per_mapping": {"x": {"hbm_bytes_per_launch": 7}}}
        path.write_text("# counters\n\n```json\n%s\n```\n" % json.dumps(data))
        got = bench.counter_summary(wl)
        assert (got is not None) == found
        if found:
            assert got["per_mapping"]["x"]["hbm_bytes_per_launch"] == 7


def test_bench_cpu_model_is_named():
    import bench
    name = bench.cpu_model()
    assert isinstance(name, str) and name


def test_read_hit_bounds():
    # 1000 requests: 900 reads, 100 writes, 800 hits.  If no write hits, all 800
    # hits are reads (800/900); if all 100 writes hit, 700 are (700/900).
    lo, hi = rc.read_hit_bounds(800.0, 900.0, 100.0)
    assert lo == pytest.approx(700 / 900, abs=1e-4) and hi == pytest.approx(800 / 900, abs=1e-4)
    # more writes than hits: the lower bound stops at zero; no reads: no bound
    assert rc.read_hit_bounds(50.0, 900.0, 100.0)[0] == 0.0
    assert rc.read_hit_bounds(50.0, 0.0, 100.0) is None


def test_counter_summary_read_hit_bounds(tmp_path):
    k_swz = "void attn::(anonymous namespace)::attn_fwd_pp_kernel<true, 2, 1>(attn::KernelArgs)"
    a = str(tmp_path / "A")
    e = str(tmp_path / "E")
    _write_counters(a, [(2, k_swz, 512 * 1024, "TCC_HIT", 800.0),
                        (2, k_swz, 512 * 1024, "TCC_MISS", 200.0)])
    _write_counters(e, [(2, k_swz, 512 * 1024, "TCC_READ", 900.0),
                        (2, k_swz, 512 * 1024, "TCC_WRITE", 100.0)])
    result, _, _, _ = rc.summarise([a, e], "mha_b1_h32_s8192_d128_causal")
    swz = result["swizzled_head_first+heavy_first"]
    assert swz["l2_hit_rate"] == pytest.approx(0.8)
    assert swz["l2_read_hit_rate_bounds"] == [pytest.approx(0.7778, abs=1e-4),
                                              pytest.approx(0.8889, abs=1e-4)]
    assert swz["l2_requests_read_write_over_hit_miss"] == pytest.approx(1.0)


def test_kernel_hash_ignores_comments_and_layout():
    from paper_2511_02132_amd.build import code_tokens
    a = 'int a = 1;  // one\n/* two\n */ const char *s = "x // y /* z */";\n'
    b = 'int a = 1;\nconst char *s = "x // y /* z */";  // other words\n'
    assert code_tokens(a) == code_tokens(b) == 'int a = 1; const char *s = "x // y /* z */";'
    # code changes do change the tokens
    assert code_tokens('int a = 2;') != code_tokens('int a = 1;')
    assert code_tokens('char c = \'/\'; int d;') == "char c = '/'; int d;"


def test_sweep_l2_counters_forward_and_backward(tmp_path):
    """Per-launch L2 hit rate and read-hit bounds from a sweep's counter run;
    a backward call's dK/dV and dQ dispatches count as one launch."""
    fwd = "void attn::(anonymous namespace)::attn_fwd_pp_kernel<true, 2, 3>(attn::KernelArgs)"
    d = tmp_path / "fwd"
    _write_counters(str(d), [
        (1, fwd, 512 * 1024, "TCC_HIT", 900.0), (1, fwd, 512 * 1024, "TCC_MISS", 100.0),
        (1, fwd, 512 * 1024, "TCC_READ", 950.0), (1, fwd, 512 * 1024, "TCC_WRITE", 50.0),
    ])
    cfg = {"B": 1, "Hq": 32, "Hkv": 32, "S": 8192}
    man = tmp_path / "fwd.json"
    man.write_text(json.dumps([{"config": cfg, "variant": pa.variant_name(0x32)}]))
    key = (1, 32, 32, 8192, pa.variant_name(0x32))
    assert sweep.l2_by_launch(str(d), str(man))[key] == pytest.approx(0.9)
    lo, hi = sweep.l2_read_bounds_by_launch(str(d), str(man))[key]
    assert lo == pytest.approx(850 / 950, abs=1e-4) and hi == pytest.approx(900 / 950, abs=1e-4)

    # backward: the forward that made O and lse is dropped; dK/dV + dQ are summed
    dkdv = "void attn::(anonymous namespace)::attn_bwd_dkdv_kernel<true, 2, 2>(attn::BwdArgs)"
    dq = "void attn::(anonymous namespace)::attn_bwd_dq_kernel<true, 2, 3>(attn::BwdArgs)"
    d = tmp_path / "bwd"
    _write_counters(str(d), [
        (1, fwd, 512 * 1024, "TCC_HIT", 1.0), (1, fwd, 512 * 1024, "TCC_MISS", 1.0),
        (2, dkdv, 256 * 256, "TCC_HIT", 300.0), (2, dkdv, 256 * 256, "TCC_MISS", 100.0),
        (3, dq, 256 * 256, "TCC_HIT", 500.0), (3, dq, 256 * 256, "TCC_MISS", 100.0),
    ])
    man = tmp_path / "bwd.json"
    man.write_text(json.dumps([{"config": cfg, "variant": pa.variant_name(0x32)}]))
    assert sweep.l2_by_launch(str(d), str(man))[key] == pytest.approx(0.8)   # 800 / 1000
    assert sweep.l2_read_bounds_by_launch(str(d), str(man)) == {}            # no read counts


def test_sweep_kv_heads_option():
    from paper_2511_02132_amd import sweep
    a = sweep.parse(["--family", "gqa", "--kv-heads", "1", "--heads", "8", "--contexts", "8192",
                     "--batches", "1", "4"])
    cs = list(sweep.configs(a.family, a.contexts, a.batches, a.heads, a.kv_heads))
    assert cs == [{"B": 1, "Hq": 8, "Hkv": 1, "S": 8192}, {"B": 4, "Hq": 8, "Hkv": 1, "S": 8192}]
    assert sweep.parse(["--family", "gqa"]).kv_heads == sweep.GQA_KV_HEADS
    assert sweep.parse([]).warmup_ms == 1000.0
    # the mha family ignores it: every q-head has its own KV head
    assert [c["Hkv"] for c in sweep.configs("mha", [4096], [1], [16], 1)] == [16]


def test_sweep_spread_comparisons():
    """A win counts only when the gap of the medians exceeds the larger
    interquartile range of the two variants' launch times."""
    assert sweep.iqr([1.0, 2.0, 3.0, 4.0, 5.0]) == 2.0
    assert sweep.iqr([7.0]) == 0.0
    r = {"ms": {"a": 1.00, "b": 1.05, "c": 1.01}, "ms_iqr": {"a": 0.02, "b": 0.01, "c": 0.03}}
    assert sweep.compare(r, "a", "b") == 1 and sweep.compare(r, "b", "a") == -1
    assert sweep.compare(r, "a", "c") == 0 and sweep.compare(r, "c", "a") == 0
    assert sweep.compare({"ms": {"a": 1.0, "b": 1.001}}, "a", "b") == 1   # no spreads: medians

    names = [n for n, _ in pa.variants(True)]
    recs = []
    for i, slow in enumerate((1.10, 1.001, 0.95)):
        ms = {n: 1.0 for n in names}
        ms["naive_block_first+heavy_first"] = slow          # vs the headline: win, tie, loss
        ms["swizzled_block_first+heavy_first"] = 1.2
        ms["naive_block_first+heavy_first+paired"] = 1.2
        ms["swizzled_block_first+heavy_first+paired"] = 1.2
        ms["naive_block_first"] = ms["swizzled_block_first"] = 1.3
        recs.append({"S": 8192 * (i + 1), "B": 1, "Hq": 32, "Hkv": 32, "ms": ms,
                     "ms_iqr": {n: 0.01 for n in names}})
    lines = sweep.comparisons(recs, names, lambda n: n, True)
    row = [l for l in lines if l.startswith("| swizzled_head_first+heavy_first vs the fastest")][0]
    cells = [c.strip() for c in row.strip("|").split("|")]
    assert cells[1:4] == ["1", "1", "1"], cells
    assert "24K B1 H32/32" in cells[4]


def test_per_kernel_counter_table(tmp_path):
    """Backward kernels are named by kind and variant; the per-kernel table
    averages each counter over a kernel's dispatches, scales FETCH_SIZE and
    WRITE_SIZE by the copy kernel, and reports LDS instructions per MFMA."""
    assert rc.kernel_of("void attn::(anonymous namespace)::attn_bwd_dkdv_kernel<true, 2, 2>"
                        "(attn::BwdArgs)") == "dK/dV swizzled_head_first+xcd_block_major"
    assert rc.kernel_of("void attn::(anonymous namespace)::attn_bwd_dq_kernel<false, 0, 1>"
                        "(attn::BwdArgs)") == "dQ naive_block_first+heavy_first"
    assert rc.kernel_of("attn::(anonymous namespace)::attn_bwd_delta_kernel(attn::BwdArgs)") == "D"
    assert rc.kernel_of("void at::native::elementwise_kernel<...>") is None
    d = tmp_path / "pass"
    d.mkdir()
    dq = "void attn::(anonymous namespace)::attn_bwd_dq_kernel<true, 2, 1>(attn::BwdArgs)"
    rows = [(1, dq, 256, "SQ_INSTS_MFMA", 100.0), (1, dq, 256, "SQ_INSTS_LDS", 150.0),
            (2, dq, 256, "SQ_INSTS_MFMA", 300.0), (2, dq, 256, "SQ_INSTS_LDS", 450.0),
            (1, dq, 256, "FETCH_SIZE", 10.0), (3, "__amd_rocclr_copyBuffer", 256, "FETCH_SIZE",
                                                131072.0)]
    with open(d / "run_counter_collection.csv", "w") as f:
        f.write("Dispatch_Id,Kernel_Name,Grid_Size,Counter_Name,Counter_Value\n")
        for r in rows:
            f.write('%d,"%s",%d,%s,%f\n' % r)
    res, fac = rc.summarise_kernels([str(d)])
    e = res["dQ swizzled_head_first+heavy_first"]
    assert e["SQ_INSTS_MFMA"] == 200.0 and e["SQ_INSTS_LDS"] == 300.0
    assert abs(fac["FETCH_SIZE"] - 2.0) < 1e-12
    out = tmp_path / "k.md"
    rc.write_kernels_md(str(out), "T", "CMD", [str(d)])
    line = [l for l in out.read_text().splitlines() if l.startswith("| dQ ")][0]
    assert "| 1.50 |" in line and "2.048e+04" in line


def test_backward_trace_summary(tmp_path):
    """The backward kernel-trace table lists D, dK/dV and dQ per variant and adds
    up the headline variant's three kernels (the dK/dV kernel carries only the
    block-major bit of the order) into FlashAttention-convention TFLOP/s."""
    ns = "void attn::(anonymous namespace)::"
    stats = tmp_path / "stats.csv"
    rows = [("attn::(anonymous namespace)::attn_bwd_delta_kernel(attn::BwdArgs)", 9, 40000.0),
            (ns + "attn_bwd_dkdv_kernel<true, 2, 0>(attn::BwdArgs)", 2, 1000000.0),
            (ns + "attn_bwd_dkdv_kernel<true, 0, 0>(attn::BwdArgs)", 2, 1200000.0),
            (ns + "attn_bwd_dq_kernel<true, 2, 1>(attn::BwdArgs)", 1, 500000.0),
            (ns + "attn_fwd_pp_kernel<true, 2, 1>(attn::KernelArgs)", 9, 300000.0)]
    with open(stats, "w") as f:
        f.write('"Name","Calls","TotalDurationNs","AverageNs","Percentage","MinNs","MaxNs"\n')
        for name, calls, avg in rows:
            f.write('"%s",%d,%d,%f,1.0,%d,%d\n' % (name, calls, calls * avg, avg, avg, avg))
    out = tmp_path / "t.md"
    rc.write_bwd_stats_md(str(out), "T", str(stats), "CMD", (1, 32, 8192))
    text = out.read_text()
    body = [l for l in text.splitlines() if l.startswith("| ") and "---" not in l][1:]
    assert [l.split("|")[1].strip() for l in body] == [
        "D", "dK/dV swizzled_head_first", "dK/dV naive_block_first",
        "dQ swizzled_head_first+heavy_first"]
    fl = 2.5 * pa.attention_flops(1, 32, 8192, 8192, 128, True)
    assert "D 40.0 + dK/dV 1000.0 + dQ 500.0 = 1540.0 us" in text
    assert "%.0f TFLOP/s in the" % (fl / 1540.0 / 1e6) in text
