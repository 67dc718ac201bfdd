"""GPU parity tests of the HIP attention backward (and the forward's lse) against the fp64 oracle.

All calls go through the C ABI (libattn_numa.so via the ctypes binding).

Bar (floating point), for each of dQ, dK, dV (bf16 outputs):
    max |g_gpu - g_ref| <= 1e-2 * max |g_ref| + 1e-5
    mean |g_gpu - g_ref| <= 4e-3 * mean |g_ref| + 1e-6
Derivation: the output is an fp32 sum rounded to bf16 (at most half an ulp,
2^-9 relative); the probabilities P and the products dS enter the matrix
cores as bf16 (again 2^-9 relative per term), so the error of an entry is
bounded by about 2^-9 |g| + 2^-9 sum |terms|, i.e. about one bf16 ulp (2^-8 =
3.9e-3) of the largest entries; 1e-2 of the max-norm leaves 2.5x headroom.
Averaged over entries, round-to-nearest contributes about 2^-10 relative per
rounding; 4e-3 of the mean magnitude bounds the three roundings.  The small
absolute terms cover gradients that vanish exactly (one key: dS = 0), where
D = <dO, O> and dP = <dO, V> are the same fp32 sum taken in two orders.
The row log-sum-exp is fp32 from an fp32 softmax: |lse_gpu - lse_ref| <= 1e-4.
Gradients must be bitwise identical across all mappings and repeated runs
(every output element is written by one workgroup in a fixed order).
"""

import numpy as np
import pytest
import torch

import attn_inputs as ai
import oracle
import paper_2511_02132_amd as pa

pytestmark = pytest.mark.gpu

ALL_MAPPINGS = [m | f for m in (0, 1, 2, 3) for f in (0, 0x10)] + [0x22, 0x32]
REL_MAX = 1e-2
REL_MEAN = 4e-3
LSE_ABS = 1e-4
DEV = "cuda:0"
D = 128


def _say(*a):
    print(*a, flush=True)


def _inputs(B, Hq, Hkv, Sq, Skv, seed):
    q = ai.randn_bf16((B, Hq, Sq, D), seed)
    k = ai.randn_bf16((B, Hkv, Skv, D), seed + 1)
    v = ai.randn_bf16((B, Hkv, Skv, D), seed + 2)
    do = ai.randn_bf16((B, Hq, Sq, D), seed + 3)
    return q, k, v, do


def _check(name, got, ref):
    got = got.float().cpu().numpy().astype(np.float64).reshape(ref.shape)
    err = np.abs(got - ref)
    assert np.isfinite(got).all(), name
    assert err.max() <= REL_MAX * np.abs(ref).max() + 1e-5, (name, err.max(), np.abs(ref).max())
    assert err.mean() <= REL_MEAN * np.abs(ref).mean() + 1e-6, (name, err.mean(),
                                                                np.abs(ref).mean())


def _grads(qd, kd, vd, dod, causal, scale, mapping=pa.SWIZZLED_HEAD_FIRST, fill=True):
    o, lse = pa.attn_fwd_lse(qd, kd, vd, causal=causal, scale=scale, mapping=mapping)
    outs = [torch.full_like(t, float("nan")) if fill else torch.empty_like(t)
            for t in (qd, kd, vd)]
    dq, dk, dv = pa.attn_bwd(qd, kd, vd, o, dod, lse, *outs, causal=causal, scale=scale,
                             mapping=mapping)
    torch.cuda.synchronize()
    return o, lse, dq, dk, dv


SHAPES = [
    # B, Hq, Hkv, Sq, Skv, causal
    (1, 2, 2, 64, 64, True),          # one tile
    (1, 2, 2, 200, 200, False),       # ragged tails
    (1, 2, 2, 200, 200, True),
    (2, 8, 2, 256, 256, True),        # GQA groups of 4, two batches
    (1, 4, 4, 96, 160, True),         # Sq < Skv, top-left causal
    (1, 4, 4, 160, 96, True),         # Sq > Skv: key blocks no query sees
    (1, 2, 1, 1024, 1024, True),      # several key blocks and query tiles
    (1, 3, 3, 1000, 1000, False),
    (1, 1, 1, 1, 1, True),            # smallest problem
    (1, 6, 3, 33, 129, False),
]


@pytest.mark.parametrize("B,Hq,Hkv,Sq,Skv,causal", SHAPES)
def test_backward_parity(B, Hq, Hkv, Sq, Skv, causal):
    _say("bwd parity", B, Hq, Hkv, Sq, Skv, causal)
    q, k, v, do = _inputs(B, Hq, Hkv, Sq, Skv, 7000 + Sq + Skv)
    scale = ai.default_scale(D)
    qd, kd, vd, dod = (t.to(DEV) for t in (q, k, v, do))
    o, lse, dq, dk, dv = _grads(qd, kd, vd, dod, causal, scale)
    qb, kb, vb, dob = (ai.bf16_bits(t) for t in (q, k, v, do))
    rl, _ = oracle.attn_row_stats_f64(qb, kb, vb, None, oracle.all_rows(B, Hq, Sq), causal, scale)
    got_lse = lse.cpu().numpy().astype(np.float64).ravel()
    assert np.abs(got_lse - rl).max() <= LSE_ABS
    rq, rk, rv = oracle.attn_bwd_f64(qb, kb, vb, dob, causal, scale)
    _check("dq", dq, rq)
    _check("dk", dk, rk)
    _check("dv", dv, rv)
    # the training forward writes the same O as the plain forward
    o2 = pa.attn_fwd(qd, kd, vd, causal=causal, scale=scale)
    torch.cuda.synchronize()
    assert torch.equal(o, o2)


@pytest.mark.parametrize("causal", [False, True])
def test_backward_bitwise_across_mappings_and_runs(causal):
    _say("bwd mappings", causal)
    q, k, v, do = _inputs(2, 8, 2, 700, 700, 7100)
    qd, kd, vd, dod = (t.to(DEV) for t in (q, k, v, do))
    scale = ai.default_scale(D)
    ref = None
    for m in ALL_MAPPINGS + [pa.SWIZZLED_HEAD_FIRST]:
        _, _, dq, dk, dv = _grads(qd, kd, vd, dod, causal, scale, mapping=m)
        if ref is None:
            ref = (dq, dk, dv)
        else:
            for a, b in zip(ref, (dq, dk, dv)):
                assert torch.equal(a, b), m


def test_backward_full_size_sampled_rows():
    """Llama-class prefill shape (MHA, 32 heads, 8K, causal): sampled rows vs the oracle."""
    B, Hq, Hkv, S, causal = 1, 32, 32, 8192, True
    _say("bwd full size", B, Hq, S)
    q, k, v, do = _inputs(B, Hq, Hkv, S, S, 7200)
    qd, kd, vd, dod = (t.to(DEV) for t in (q, k, v, do))
    scale = ai.default_scale(D)
    _, _, dq, dk, dv = _grads(qd, kd, vd, dod, causal, scale, mapping=pa.SWIZZLED_HEAD_FIRST | 0x10)
    qb, kb, vb, dob = (ai.bf16_bits(t) for t in (q, k, v, do))
    rng = np.random.default_rng(5)
    heads = [0, 17]
    rows = np.array([[0, h, i] for h in heads
                     for i in [0, 1, 255, 256, 4095, 8191] + list(rng.integers(0, S, 10))], np.int64)
    rq = oracle.attn_bwd_dq_rows_f64(qb, kb, vb, dob, rows, causal, scale)
    got = dq.float().cpu().numpy()[rows[:, 0], rows[:, 1], rows[:, 2]]
    _check("dq rows", torch.from_numpy(got), rq)
    # dK/dV rows need the statistics of every query row of the head
    for h in heads:
        hrows = oracle.all_rows(1, 1, S)
        hrows[:, 1] = h
        lse_h, D_h = oracle.attn_row_stats_f64(qb, kb, vb, dob, hrows, causal, scale)
        lse_all = np.zeros((B, Hq, S))
        D_all = np.zeros((B, Hq, S))
        lse_all[0, h] = lse_h
        D_all[0, h] = D_h
        keys = np.array([[0, h, j] for j in [0, 127, 128, 4096, 8191] + list(rng.integers(0, S, 6))],
                        np.int64)
        rk, rv = oracle.attn_bwd_dkdv_rows_f64(qb, kb, vb, dob, keys, causal, scale,
                                               stats=(lse_all, D_all))
        gk = dk.float().cpu().numpy()[keys[:, 0], keys[:, 1], keys[:, 2]]
        gv = dv.float().cpu().numpy()[keys[:, 0], keys[:, 1], keys[:, 2]]
        _check("dk rows", torch.from_numpy(gk), rk)
        _check("dv rows", torch.from_numpy(gv), rv)
    for t in (dq, dk, dv):
        assert torch.isfinite(t.float()).all()


def test_backward_gqa_noncausal_ragged_sampled():
    """GQA (groups of four), no mask, 4000 rows and keys (ragged 128-key and 64-key
    blocks): sampled dQ rows and dK/dV keys vs the oracle."""
    B, Hq, Hkv, S, causal = 1, 16, 4, 4000, False
    _say("bwd gqa non-causal ragged", B, Hq, Hkv, S)
    q, k, v, do = _inputs(B, Hq, Hkv, S, S, 7400)
    qd, kd, vd, dod = (t.to(DEV) for t in (q, k, v, do))
    scale = ai.default_scale(D)
    _, _, dq, dk, dv = _grads(qd, kd, vd, dod, causal, scale, mapping=pa.SWIZZLED_HEAD_FIRST | 0x10)
    qb, kb, vb, dob = (ai.bf16_bits(t) for t in (q, k, v, do))
    rng = np.random.default_rng(6)
    rows = np.array([[0, h, i] for h in (0, 13)
                     for i in [0, 31, 32, 3967, 3968, 3999] + list(rng.integers(0, S, 8))], np.int64)
    rq = oracle.attn_bwd_dq_rows_f64(qb, kb, vb, dob, rows, causal, scale)
    got = dq.float().cpu().numpy()[rows[:, 0], rows[:, 1], rows[:, 2]]
    _check("dq rows", torch.from_numpy(got), rq)
    # dK/dV of K/V head 1 sum over query heads 4-7: their statistics for every row
    g = 1
    heads = range(4 * g, 4 * g + 4)
    lse_all = np.zeros((B, Hq, S))
    D_all = np.zeros((B, Hq, S))
    for h in heads:
        hrows = oracle.all_rows(1, 1, S)
        hrows[:, 1] = h
        lse_all[0, h], D_all[0, h] = oracle.attn_row_stats_f64(qb, kb, vb, dob, hrows, causal, scale)
    keys = np.array([[0, g, j] for j in [0, 127, 128, 3967, 3968, 3999] + list(rng.integers(0, S, 6))],
                    np.int64)
    rk, rv = oracle.attn_bwd_dkdv_rows_f64(qb, kb, vb, dob, keys, causal, scale,
                                           stats=(lse_all, D_all))
    gk = dk.float().cpu().numpy()[keys[:, 0], keys[:, 1], keys[:, 2]]
    gv = dv.float().cpu().numpy()[keys[:, 0], keys[:, 1], keys[:, 2]]
    _check("dk rows", torch.from_numpy(gk), rk)
    _check("dv rows", torch.from_numpy(gv), rv)
    for t in (dq, dk, dv):
        assert torch.isfinite(t.float()).all()


def test_backward_errors():
    q, k, v, do = (t.to(DEV) for t in _inputs(1, 2, 2, 64, 64, 7300))
    o, lse = pa.attn_fwd_lse(q, k, v, causal=True)
    torch.cuda.synchronize()
    with pytest.raises(pa.AttnError) as e:   # d = 64 is forward-only
        q64 = torch.zeros(1, 2, 64, 64, dtype=torch.bfloat16, device=DEV)
        o64, lse64 = pa.attn_fwd_lse(q64, q64, q64)
        pa.attn_bwd(q64, q64, q64, o64, q64, lse64)
    assert e.value.code == -3
    with pytest.raises(pa.AttnError) as e:   # dq written over q
        pa.attn_bwd(q, k, v, o, do, lse, q)
    assert e.value.code == -8
    with pytest.raises(pa.AttnError) as e:
        pa.attn_bwd(q, k, v, o, do, lse, mapping=7)
    assert e.value.code == -4
    with pytest.raises(pa.AttnError) as e:   # paired row blocks: a forward-only order
        pa.attn_bwd(q, k, v, o, do, lse, mapping=pa.SWIZZLED_HEAD_FIRST | pa.PAIRED)
    assert e.value.code == -4
    torch.cuda.synchronize()
