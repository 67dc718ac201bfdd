"""GPU parity tests of the HIP attention-forward path against the fp64 oracle.

All calls go through the C ABI (libattn_numa.so via the ctypes binding).
Bar (floating point): max |O_gpu - O_oracle| <= 2e-2 and mean <= 2e-3 with bf16
inputs ~ N(0, 1) and scale = 1/sqrt(d).  Integer work (the placement of
workgroups) is compared bit-exactly with the oracle enumeration.  The output
must be bitwise identical across the three mappings and across repeated runs;
causal row 0 must equal V[0] exactly; a NaN-filled output buffer must be fully
overwritten.
"""

import numpy as np
import pytest
import torch

import attn_inputs as ai
import oracle
import paper_2511_02132_amd as pa
from oracle import mapping as mp

pytestmark = pytest.mark.gpu

# the four mappings, each with the paper's block order and with heavy-first order,
# and swizzled head-first with block-major order inside each XCD's piece
ALL_MAPPINGS = [m | f for m in (0, 1, 2, 3) for f in (0, 0x10)] + [0x22, 0x32]


def mappings_for(d):
    """ALL_MAPPINGS and, for d = 128, each of them also with paired row blocks."""
    return ALL_MAPPINGS + ([m | pa.PAIRED for m in ALL_MAPPINGS] if d == 128 else [])

MAX_ABS = 2e-2
MEAN_ABS = 2e-3
DEV = "cuda:0"


def _say(*a):
    print(*a, flush=True)


def _to_dev(*ts):
    return [t.to(DEV) for t in ts]


def _run(q, k, v, causal, scale, mapping):
    o = torch.full(q.shape, float("nan"), dtype=torch.bfloat16, device=DEV)
    pa.attn_fwd(q, k, v, o, causal=causal, scale=scale, mapping=mapping)
    torch.cuda.synchronize()
    return o


def _err(o_gpu, o_ref):
    diff = np.abs(o_gpu.float().cpu().numpy().astype(np.float64) - o_ref)
    return float(diff.max()), float(diff.mean())


# ------------------------------------------------------------------ placement


PROBE_SHAPES = [
    # B, Hq, Hkv, S, d
    (1, 4, 4, 256, 64), (1, 32, 32, 8192, 128), (1, 64, 8, 8192, 128), (8, 64, 64, 4096, 128),
    (1, 16, 16, 131072, 128), (2, 12, 4, 300, 128), (3, 5, 5, 1000, 64),
    (2, 128, 128, 2048, 56),   # short heads: block-major groups of 16 heads
]


@pytest.mark.parametrize("B,Hq,Hkv,S,d", PROBE_SHAPES)
def test_probe_matches_enumeration_and_dispatch(B, Hq, Hkv, S, d):
    _say("probe", B, Hq, Hkv, S, d)
    g = torch.Generator(device=DEV).manual_seed(3)
    q = torch.randn(B, Hq, S, d, device=DEV, generator=g).to(torch.bfloat16)
    k = torch.randn(B, Hkv, S, d, device=DEV, generator=g).to(torch.bfloat16)
    v = torch.randn(B, Hkv, S, d, device=DEV, generator=g).to(torch.bfloat16)
    nx = pa.num_xcd()
    BM = pa.block_m(d)
    outs = []
    for value in mappings_for(d):
        mapping, heavy, xbm, paired = mp.split_flags(value)
        o, probe = pa.attn_fwd_probe(q, k, v, causal=True, mapping=value)
        torch.cuda.synchronize()
        rec = probe.cpu().numpy()
        want = mp.enumerate_mapping(mapping, B, Hq, S, BM, nx, heavy_first=heavy,
                                    short_head_groups=(BM == 128),
                                    xcd_block_major=xbm, paired=paired)
        n = want.shape[0]   # workgroups launched (pair slots when paired)
        assert np.array_equal(rec[:n, :3], want), "placement differs from the enumeration"
        assert (rec[n:] == -1).all(), "a record past the paired grid was written"
        wid = np.arange(n)
        assert np.array_equal(rec[:n, 3], wid % nx), "XCC_ID != wid mod NX"
        outs.append(o)
    for o in outs[1:]:
        assert torch.equal(o, outs[0]), "output depends on the mapping"


def test_num_xcd_is_eight_on_mi355x():
    assert pa.num_xcd() == 8


# ------------------------------------------------------------------ full parity, small shapes

SMALL = [
    # B, Hq, Hkv, Sq, Skv, d, causal
    (1, 4, 4, 256, 256, 64, False),     # the small MHA workload
    (1, 4, 4, 256, 256, 64, True),
    (2, 8, 2, 384, 384, 128, True),     # GQA 4:1, several tiles
    (1, 8, 1, 200, 200, 128, False),    # GQA 8:1, ragged q and kv
    (1, 2, 2, 333, 517, 128, False),    # Sq != Skv, ragged
    (1, 2, 2, 517, 333, 128, True),     # causal with Sq > Skv
    (1, 2, 2, 333, 517, 64, True),      # causal with Sq < Skv
    (2, 6, 3, 129, 65, 64, False),      # one row / one key past a tile
    (1, 1, 1, 1, 1, 128, False),        # single element
    (1, 1, 1, 1, 1, 64, True),
    (1, 3, 1, 64, 1000, 128, False),    # short q, long kv
    (3, 2, 2, 1000, 64, 64, True),
    (1, 16, 16, 1024, 1024, 128, True),
    (1, 2, 2, 100, 128, 128, False),    # exactly two K/V tiles
    (1, 2, 2, 190, 190, 128, True),     # three tiles, the last ragged (odd trip count)
]


@pytest.mark.parametrize("B,Hq,Hkv,Sq,Skv,d,causal", SMALL)
def test_parity_small(B, Hq, Hkv, Sq, Skv, d, causal):
    _say("parity", B, Hq, Hkv, Sq, Skv, d, causal)
    q, k, v = ai.make_qkv(B, Hq, Hkv, Sq, Skv, d, seed_base=7000 + Sq + 3 * Skv + d)
    scale = ai.default_scale(d)
    ref = oracle.attn_fwd_f64(ai.bf16_bits(q), ai.bf16_bits(k), ai.bf16_bits(v), causal, scale)
    qd, kd, vd = _to_dev(q, k, v)
    outs = [_run(qd, kd, vd, causal, scale, m) for m in mappings_for(d)]
    for o in outs:
        assert not torch.isnan(o).any(), "unwritten output elements"
        mx, mean = _err(o, ref)
        assert mx <= MAX_ABS and mean <= MEAN_ABS, (mx, mean)
    for o in outs[1:]:
        assert torch.equal(o, outs[0])
    again = _run(qd, kd, vd, causal, scale, pa.SWIZZLED_HEAD_FIRST)
    assert torch.equal(again, outs[0]), "not deterministic"
    if causal:
        rep = Hq // Hkv
        assert torch.equal(outs[0][:, :, 0, :].cpu(),
                           v[:, :, 0, :].repeat_interleave(rep, dim=1)), "causal row 0 != V[0]"


def test_parity_small_workload_seeded():
    """The small MHA workload with its own seeds (B1 H4 S256 d64, non-causal)."""
    name = "mha_b1_h4_s256_d64"
    w = ai.WORKLOADS[name]
    q, k, v = ai.workload_inputs(name)
    scale = ai.default_scale(w["d"])
    ref = oracle.attn_fwd_f64(ai.bf16_bits(q), ai.bf16_bits(k), ai.bf16_bits(v), False, scale)
    qd, kd, vd = _to_dev(q, k, v)
    for m in mp.MAPPINGS:
        mx, mean = _err(_run(qd, kd, vd, False, scale, m), ref)
        assert mx <= MAX_ABS and mean <= MEAN_ABS, (m, mx, mean)


def test_extreme_scores_stay_finite():
    """Large scores (|s| ~ 1e3): the running max keeps every exponent <= 0."""
    B, H, S, d = 1, 2, 300, 128
    q, k, v = ai.make_qkv(B, H, H, S, S, d, seed_base=8100)
    q = q * 16
    k = k * 16
    scale = ai.default_scale(d)
    for causal in (False, True):
        ref = oracle.attn_fwd_f64(ai.bf16_bits(q), ai.bf16_bits(k), ai.bf16_bits(v), causal, scale)
        o = _run(*_to_dev(q, k, v), causal, scale, pa.SWIZZLED_HEAD_FIRST)
        mx, mean = _err(o, ref)
        assert torch.isfinite(o.float()).all()
        assert mx <= MAX_ABS and mean <= MEAN_ABS, (mx, mean)


def test_stream_argument():
    """Work enqueued on a side stream (default priority) lands on that stream."""
    q, k, v = _to_dev(*ai.make_qkv(1, 4, 4, 512, 512, 128, seed_base=8200))
    s = torch.cuda.Stream()
    ref = _run(q, k, v, True, 0.0884, pa.SWIZZLED_HEAD_FIRST)
    with torch.cuda.stream(s):
        o = torch.empty_like(q)
        pa.attn_fwd(q, k, v, o, causal=True, scale=0.0884, stream=s)
    s.synchronize()
    assert torch.equal(o, ref)


def test_errors_surface_as_exceptions():
    q = torch.zeros(1, 3, 128, 128, dtype=torch.bfloat16, device=DEV)
    k = torch.zeros(1, 2, 128, 128, dtype=torch.bfloat16, device=DEV)
    with pytest.raises(pa.AttnError) as e:
        pa.attn_fwd(q, k, k)
    assert e.value.code == -2
    with pytest.raises(pa.AttnError) as e:
        pa.attn_fwd(q, q, q, q)
    assert e.value.code == -8
    # paired row blocks: the d = 128 dispatched forward only
    q64 = torch.zeros(1, 2, 128, 64, dtype=torch.bfloat16, device=DEV)
    with pytest.raises(pa.AttnError) as e:
        pa.attn_fwd(q64, q64, q64, mapping=pa.SWIZZLED_HEAD_FIRST | pa.PAIRED)
    assert e.value.code == -3


# ------------------------------------------------------------------ full sizes, sampled rows

FULL = ["mha_b1_h32_s8192_d128_causal", "gqa_b1_hq64_hkv8_s8192_d128_causal",
        "mha_b8_h64_s4096_d128", "mha_b1_h16_s131072_d128_causal"]


@pytest.mark.parametrize("name", FULL)
def test_parity_full_size_sampled_rows(name):
    w = ai.WORKLOADS[name]
    _say("full-size", name)
    q, k, v = ai.workload_inputs(name)
    scale = ai.default_scale(w["d"])
    causal = w["causal"]
    qd, kd, vd = _to_dev(q, k, v)
    outs = [_run(qd, kd, vd, causal, scale, m) for m in mappings_for(w["d"])]
    for o in outs:
        assert not torch.isnan(o).any(), "unwritten output elements"
    for o in outs[1:]:
        assert torch.equal(o, outs[0]), "output depends on the mapping"
    n_random = 4 if w["B"] * w["Hq"] > 64 else 16
    rows = ai.sample_rows(w["B"], w["Hq"], w["Sq"], pa.block_m(w["d"]), n_random,
                          seed=w["index"])
    ref = oracle.attn_fwd_rows_f64(ai.bf16_bits(q), ai.bf16_bits(k), ai.bf16_bits(v), rows,
                                   causal, scale)
    got = outs[0].cpu()[rows[:, 0], rows[:, 1], rows[:, 2]].float().numpy().astype(np.float64)
    diff = np.abs(got - ref)
    _say("  rows", rows.shape[0], "max", diff.max(), "mean", diff.mean())
    assert diff.max() <= MAX_ABS and diff.mean() <= MEAN_ABS
    if causal:
        rep = w["Hq"] // w["Hkv"]
        assert torch.equal(outs[0][:, :, 0, :].cpu(), v[:, :, 0, :].repeat_interleave(rep, dim=1))


# ------------------------------------------------------------------ d = 56


D56_SHAPES = [
    # B, Hq, Hkv, Sq, Skv, causal: DeepSeek-V3-shaped heads (Section 4.5), not a
    # multiple of the matrix-core k-step; zero-padded to 64 inside the kernel
    (1, 2, 2, 100, 100, True),
    (2, 8, 2, 257, 300, False),
    (1, 4, 4, 1000, 1000, True),
    (1, 3, 3, 1, 1, False),
    (1, 4, 2, 1, 777, False),       # one query row against a long ragged key range, GQA
    (2, 6, 3, 130, 700, True),      # Sq < Skv under the top-left causal mask
]


@pytest.mark.parametrize("B,Hq,Hkv,Sq,Skv,causal", D56_SHAPES)
def test_parity_d56(B, Hq, Hkv, Sq, Skv, causal):
    _say("d56 parity", B, Hq, Hkv, Sq, Skv, causal)
    d = 56
    q = ai.randn_bf16((B, Hq, Sq, d), 8100 + Sq)
    k = ai.randn_bf16((B, Hkv, Skv, d), 8101 + Sq)
    v = ai.randn_bf16((B, Hkv, Skv, d), 8102 + Sq)
    scale = ai.default_scale(d)
    qd, kd, vd = _to_dev(q, k, v)
    outs = [_run(qd, kd, vd, causal, scale, m) for m in ALL_MAPPINGS]
    ref = oracle.attn_fwd_f64(ai.bf16_bits(q), ai.bf16_bits(k), ai.bf16_bits(v), causal, scale)
    mx, mean = _err(outs[0], ref)
    assert mx <= MAX_ABS and mean <= MEAN_ABS, (mx, mean)
    for o in outs[1:]:
        assert torch.equal(o, outs[0])
    # the padding columns are not written: the tensor stays 56 wide and fully finite
    assert torch.isfinite(outs[0].float()).all()
    o2, lse = pa.attn_fwd_lse(qd, kd, vd, causal=causal, scale=scale)
    torch.cuda.synchronize()
    assert torch.equal(o2, outs[0])
    rl, _ = oracle.attn_row_stats_f64(ai.bf16_bits(q), ai.bf16_bits(k), ai.bf16_bits(v), None,
                                      oracle.all_rows(B, Hq, Sq), causal, scale)
    assert np.abs(lse.cpu().numpy().astype(np.float64).ravel() - rl).max() <= lse_tolerance(56)


def test_parity_d56_deepseek_prefill_sampled():
    """DeepSeek-V3 prefill shape (MHA, 128 heads, d 56, 8K, causal): sampled rows."""
    B, H, S, d = 1, 128, 8192, 56
    _say("d56 full size", B, H, S)
    q = ai.randn_bf16((B, H, S, d), 8200)
    k = ai.randn_bf16((B, H, S, d), 8201)
    v = ai.randn_bf16((B, H, S, d), 8202)
    scale = ai.default_scale(d)
    qd, kd, vd = _to_dev(q, k, v)
    o = _run(qd, kd, vd, True, scale, pa.method_variant(True))
    rng = np.random.default_rng(3)
    rows = np.stack([np.zeros(48, np.int64), rng.integers(0, H, 48), rng.integers(0, S, 48)], 1)
    rows[:3, 2] = [0, 8191, 4096]
    ref = oracle.attn_fwd_rows_f64(ai.bf16_bits(q), ai.bf16_bits(k), ai.bf16_bits(v), rows, True,
                                   scale)
    got = o.float().cpu().numpy()[rows[:, 0], rows[:, 1], rows[:, 2]]
    err = np.abs(got - ref)
    assert err.max() <= MAX_ABS and err.mean() <= MEAN_ABS, (err.max(), err.mean())
    assert torch.isfinite(o.float()).all()


LSE_SHAPES = [
    # B, Hq, Hkv, Sq, Skv, d, causal
    (1, 4, 2, 200, 200, 56, True),
    (2, 3, 3, 129, 300, 56, False),
    (1, 4, 4, 256, 256, 64, True),
    (1, 6, 2, 70, 517, 64, False),
    (1, 2, 2, 333, 333, 128, True),
    (2, 8, 2, 96, 160, 128, False),
]


def lse_tolerance(d: int) -> float:
    """Bound on |lse_gpu - lse_oracle| (natural log).

    d = 128: the row sum is the fp32 sum of the fp32 exponentials; 1e-4 covers
    the fp32 rounding of scores, exponentials, sum and logarithm.
    d = 56, 64: the row sum is taken over the exponentials rounded to bf16 (the
    weights the output product uses).  Rounding to nearest with 8 significant
    bits changes each positive term by at most 2^-8 of itself, so the sum by
    at most 2^-8 of itself and its logarithm by at most ln(1 + 2^-8) < 3.9e-3;
    with the fp32 part, 4e-3."""
    return 1e-4 if d == 128 else 4e-3


@pytest.mark.parametrize("B,Hq,Hkv,Sq,Skv,d,causal", LSE_SHAPES)
def test_forward_lse_all_head_dims(B, Hq, Hkv, Sq, Skv, d, causal):
    """attn_fwd_lse: the row log-sum-exp (natural log of the scaled, masked scores)
    matches the oracle within lse_tolerance(d) for every head dimension, and O is
    bitwise the plain forward's."""
    _say("lse", B, Hq, Hkv, Sq, Skv, d, causal)
    q = ai.randn_bf16((B, Hq, Sq, d), 9100 + d)
    k = ai.randn_bf16((B, Hkv, Skv, d), 9101 + d)
    v = ai.randn_bf16((B, Hkv, Skv, d), 9102 + d)
    scale = ai.default_scale(d)
    qd, kd, vd = _to_dev(q, k, v)
    lse = torch.full((B, Hq, Sq), float("nan"), dtype=torch.float32, device=DEV)
    paired = (pa.method_variant(causal) | pa.PAIRED,) if d == 128 else ()
    for m in (pa.SWIZZLED_HEAD_FIRST, pa.method_variant(causal), pa.NAIVE_BLOCK_FIRST) + paired:
        o, lse = pa.attn_fwd_lse(qd, kd, vd, lse=lse, causal=causal, scale=scale, mapping=m)
        torch.cuda.synchronize()
        ref, _ = oracle.attn_row_stats_f64(ai.bf16_bits(q), ai.bf16_bits(k), ai.bf16_bits(v), None,
                                           oracle.all_rows(B, Hq, Sq), causal, scale)
        got = lse.cpu().numpy().astype(np.float64).ravel()
        assert np.isfinite(got).all()
        assert np.abs(got - ref).max() <= lse_tolerance(d), (m, np.abs(got - ref).max())
        assert torch.equal(o, _run(qd, kd, vd, causal, scale, m))
