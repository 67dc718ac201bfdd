"""GPU tests of the persistent form of the forward (attn_fwd_persistent, d = 128).

All calls go through the C ABI.  The persistent form must match the fp64
oracle (O within max-abs 2e-2 and mean-abs 2e-3, the row log-sum-exp within
1e-4) on host-drawn seeded inputs for every mapping variant, produce bitwise
the output of attn_fwd (same per-tile arithmetic), compute every tile exactly once
(the probe, indexed by workgroup id, equals the CPU enumeration of the
mapping), run each tile on the XCD its queue belongs to except for tiles taken
from another queue at the end, and leave the queue buffer zeroed so that the
next launch on the stream can reuse it.
"""

import numpy as np
import pytest
import torch

import attn_inputs as ai
import oracle
import paper_2511_02132_amd as pa
from oracle import mapping as mp

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
VARIANTS = [m | f for m in (0, 1, 2, 3) for f in (0, 0x10)] + [0x22, 0x32]
SHAPES = [
    # B, Hq, Hkv, Sq, Skv, causal
    (1, 32, 32, 8192, 8192, True),
    (1, 64, 8, 2048, 2048, True),
    (2, 12, 4, 700, 900, False),
    (1, 3, 1, 257, 257, True),      # fewer tiles than compute units, ragged
    (1, 1, 1, 1, 1, False),         # one tile
]


MAX_ABS = 2e-2
MEAN_ABS = 2e-3
LSE_ABS = 1e-4   # d = 128: fp32 sum of fp32 exponentials (as attn_fwd_lse)


def _inputs(B, Hq, Hkv, Sq, Skv, seed):
    return [t.to(DEV) for t in ai.make_qkv(B, Hq, Hkv, Sq, Skv, 128, seed_base=seed)]


def _persistent(q, k, v, causal, scale, value, queue, probe=None):
    B, Hq, Sq, _ = q.shape
    o = torch.full_like(q, float("nan"))
    lse = torch.full((B, Hq, Sq), float("nan"), dtype=torch.float32, device=DEV)
    pa.attn_fwd_persistent(q, k, v, o, lse=lse, queue=queue, probe=probe, causal=causal,
                           scale=scale, mapping=value)
    torch.cuda.synchronize()
    return o, lse


def _check_rows(o, lse, qc, kc, vc, rows, causal, scale, what):
    """O and lse rows of the persistent form against the oracle."""
    qb, kb, vb = ai.bf16_bits(qc), ai.bf16_bits(kc), ai.bf16_bits(vc)
    ref_o = oracle.attn_fwd_rows_f64(qb, kb, vb, rows, causal, scale)
    ref_l, _ = oracle.attn_row_stats_f64(qb, kb, vb, None, rows, causal, scale)
    oc = o.cpu()
    got_o = oc[rows[:, 0], rows[:, 1], rows[:, 2]].float().numpy().astype(np.float64)
    got_l = lse.cpu().numpy().astype(np.float64)[rows[:, 0], rows[:, 1], rows[:, 2]]
    err = np.abs(got_o - ref_o)
    assert not torch.isnan(oc).any(), (what, "unwritten output")
    assert err.max() <= MAX_ABS and err.mean() <= MEAN_ABS, (what, err.max(), err.mean())
    assert np.abs(got_l - ref_l).max() <= LSE_ABS, (what, np.abs(got_l - ref_l).max())


# Ragged GQA shapes with fewer tiles than compute units (at most 36 tiles of
# 256 rows), plus the two persistent-test shapes that no other test checks
# against the oracle.
ORACLE_SHAPES = [
    # B, Hq, Hkv, Sq, Skv, causal
    (1, 6, 2, 300, 450, True),
    (2, 4, 1, 700, 513, False),
    (1, 8, 4, 129, 1000, True),
    (2, 12, 4, 700, 900, False),
    (1, 64, 8, 2048, 2048, True),
]


@pytest.mark.parametrize("B,Hq,Hkv,Sq,Skv,causal", ORACLE_SHAPES)
def test_persistent_matches_oracle(B, Hq, Hkv, Sq, Skv, causal):
    """Every variant of the persistent form against the fp64 oracle: every row
    on the small shapes, sampled rows (fixed boundary rows plus seeded random
    ones per head) on the 2K GQA shape."""
    print("persistent vs oracle", B, Hq, Hkv, Sq, Skv, causal, flush=True)
    seed = 9300 + Sq + 7 * Skv
    qc, kc, vc = ai.make_qkv(B, Hq, Hkv, Sq, Skv, 128, seed_base=seed)
    q, k, v = qc.to(DEV), kc.to(DEV), vc.to(DEV)
    scale = ai.default_scale(128)
    if B * Hq * Sq <= 32768:
        rows = oracle.all_rows(B, Hq, Sq)
    else:
        rows = ai.sample_rows(B, Hq, Sq, pa.block_m(128), 4, seed=seed)
    queue = pa.new_queue(DEV)
    ref = pa.attn_fwd(q, k, v, causal=causal, scale=scale)
    torch.cuda.synchronize()
    for value in VARIANTS:
        o, lse = _persistent(q, k, v, causal, scale, value, queue)
        _check_rows(o, lse, qc, kc, vc, rows, causal, scale, hex(value))
        assert torch.equal(o, ref), hex(value)
        assert int(queue.abs().sum()) == 0, "queue not reset by the last workgroup"


def test_persistent_matches_oracle_8k_workload():
    """The MHA B1 H32 8K causal workload with its own seeds: every variant of the
    persistent form against the oracle on sampled rows (fixed boundary rows and
    seeded random rows of every head)."""
    name = "mha_b1_h32_s8192_d128_causal"
    w = ai.WORKLOADS[name]
    print("persistent vs oracle", name, flush=True)
    qc, kc, vc = ai.workload_inputs(name)
    q, k, v = qc.to(DEV), kc.to(DEV), vc.to(DEV)
    scale = ai.default_scale(128)
    rows = ai.sample_rows(w["B"], w["Hq"], w["Sq"], pa.block_m(128), 6, seed=w["index"])
    queue = pa.new_queue(DEV)
    for value in VARIANTS:
        o, lse = _persistent(q, k, v, True, scale, value, queue)
        _check_rows(o, lse, qc, kc, vc, rows, True, scale, hex(value))
        assert int(queue.abs().sum()) == 0


@pytest.mark.parametrize("B,Hq,Hkv,Sq,Skv,causal", SHAPES)
def test_persistent_equals_dispatched(B, Hq, Hkv, Sq, Skv, causal):
    print("persistent", B, Hq, Hkv, Sq, Skv, causal, flush=True)
    q, k, v = _inputs(B, Hq, Hkv, Sq, Skv, 11)
    scale = ai.default_scale(128)
    queue = pa.new_queue(DEV)
    nx = pa.num_xcd()
    n = pa.grid_size(B, Hq, Sq, 128)
    ref = pa.attn_fwd(q, k, v, causal=causal, scale=scale)
    ref_o, ref_lse = pa.attn_fwd_lse(q, k, v, causal=causal, scale=scale)
    torch.cuda.synchronize()
    for value in VARIANTS:
        mapping, heavy, xbm, _ = mp.split_flags(value)
        o = torch.full_like(q, float("nan"))
        lse = torch.full((B, Hq, Sq), float("nan"), dtype=torch.float32, device=DEV)
        probe = torch.full((n, 4), -1, dtype=torch.int32, device=DEV)
        pa.attn_fwd_persistent(q, k, v, o, lse=lse, queue=queue, probe=probe, causal=causal,
                               scale=scale, mapping=value)
        torch.cuda.synchronize()
        assert torch.equal(o, ref), hex(value)
        assert torch.equal(lse, ref_lse), hex(value)
        assert int(queue.abs().sum()) == 0, "queue not reset by the last workgroup"
        rec = probe.cpu().numpy()
        want = mp.enumerate_mapping(mapping, B, Hq, Sq, pa.block_m(128), nx, heavy_first=heavy,
                                    xcd_block_major=xbm)
        assert np.array_equal(rec[:, :3], want), hex(value)
        # Tiles leave their XCD only when taken from another queue at the end.
        # Checked where every XCD's queue holds several tiles: on a grid of a
        # few tiles, whichever workgroup asks first may take one, which changes
        # neither the result nor the speed.
        if n >= 8 * nx:
            on_own_xcd = np.mean(rec[:, 3] == np.arange(n) % nx)
            assert on_own_xcd >= (0.5 if n < 1024 else 0.9), (hex(value), on_own_xcd)


def test_persistent_reuses_queue_back_to_back():
    q, k, v = _inputs(1, 16, 16, 4096, 4096, 12)
    queue = pa.new_queue(DEV)
    ref = pa.attn_fwd(q, k, v, causal=True)
    outs = [pa.attn_fwd_persistent(q, k, v, causal=True, queue=queue,
                                   mapping=pa.method_variant(True)) for _ in range(5)]
    torch.cuda.synchronize()
    for o in outs:
        assert torch.equal(o, ref)
    assert int(queue.abs().sum()) == 0


def test_persistent_errors():
    q, k, v = _inputs(1, 2, 2, 64, 64, 13)
    with pytest.raises(pa.AttnError) as e:   # d = 64 has no persistent form
        q64 = torch.zeros(1, 2, 64, 64, dtype=torch.bfloat16, device=DEV)
        pa.attn_fwd_persistent(q64, q64, q64)
    assert e.value.code == -3
    with pytest.raises(pa.AttnError) as e:   # queue inside the output
        o = torch.empty_like(q)
        pa.attn_fwd_persistent(q, k, v, o, queue=o.view(torch.int32).view(-1)[:64])
    assert e.value.code == -8
    with pytest.raises(pa.AttnError) as e:   # paired row blocks: dispatched grid only
        pa.attn_fwd_persistent(q, k, v, mapping=pa.SWIZZLED_HEAD_FIRST | pa.PAIRED)
    assert e.value.code == -3
    torch.cuda.synchronize()
