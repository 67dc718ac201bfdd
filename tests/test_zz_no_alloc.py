"""GPU test of attn_fwd_persistent_noalloc, the entry point that allocates
nothing (its tile queues live in a device array the library owns).

Through the C ABI: two calls in a row, the second on a smaller problem, each
compared bitwise with attn_fwd_persistent (the existing entry point with a
caller-owned queue) on the same inputs, and with the fp64 oracle (max-abs
2e-2, mean-abs 2e-3; lse 1e-4).  Also checks that the array is left zero for
the next call, that the outputs are fully written, and the error paths.
"""

import numpy as np
import pytest
import torch

import attn_inputs as ai
import oracle
import paper_2511_02132_amd as pa

pytestmark = pytest.mark.gpu

DEV = "cuda:0"


def _case(B, Hq, Hkv, Sq, Skv, causal, mapping, seed):
    print("noalloc", B, Hq, Hkv, Sq, Skv, causal, hex(mapping), flush=True)
    qc, kc, vc = ai.make_qkv(B, Hq, Hkv, Sq, Skv, 128, seed_base=seed)
    q, k, v = qc.to(DEV), kc.to(DEV), vc.to(DEV)
    scale = ai.default_scale(128)
    o = torch.full_like(q, float("nan"))
    lse = torch.full((B, Hq, Sq), float("nan"), dtype=torch.float32, device=DEV)
    pa.attn_fwd_persistent_noalloc(q, k, v, o, lse=lse, causal=causal, scale=scale,
                                   mapping=mapping)
    torch.cuda.synchronize()
    ref_o = torch.full_like(q, float("nan"))
    ref_l = torch.full_like(lse, float("nan"))
    queue = pa.new_queue(DEV)
    pa.attn_fwd_persistent(q, k, v, ref_o, lse=ref_l, queue=queue, causal=causal, scale=scale,
                           mapping=mapping)
    torch.cuda.synchronize()
    assert not torch.isnan(o).any() and not torch.isnan(lse).any(), "unwritten output"
    assert torch.equal(o, ref_o), "differs from attn_fwd_persistent"
    assert torch.equal(lse, ref_l), "lse differs from attn_fwd_persistent"
    rows = oracle.all_rows(B, Hq, Sq)
    qb, kb, vb = ai.bf16_bits(qc), ai.bf16_bits(kc), ai.bf16_bits(vc)
    want = oracle.attn_fwd_rows_f64(qb, kb, vb, rows, causal, scale)
    want_l, _ = oracle.attn_row_stats_f64(qb, kb, vb, None, rows, causal, scale)
    got = o.cpu().float().numpy().astype(np.float64).reshape(-1, 128)
    err = np.abs(got - want)
    assert err.max() <= 2e-2 and err.mean() <= 2e-3, (err.max(), err.mean())
    assert np.abs(lse.cpu().numpy().astype(np.float64).ravel() - want_l).max() <= 1e-4


def test_noalloc_two_calls_second_smaller():
    # first call: 2 x 16 x 3 = 96 tiles over GQA groups of 4, ragged rows
    _case(2, 16, 4, 700, 700, True, pa.SWIZZLED_HEAD_FIRST | pa.HEAVY_FIRST, 9500)
    # second call, smaller: 3 tiles, non-causal, ragged keys
    _case(1, 3, 1, 600, 333, False, pa.NAIVE_BLOCK_FIRST, 9600)


def test_noalloc_errors():
    q = torch.zeros(1, 2, 64, 64, dtype=torch.bfloat16, device=DEV)
    with pytest.raises(pa.AttnError) as e:   # d = 64 has no persistent form
        pa.attn_fwd_persistent_noalloc(q, q, q, torch.empty_like(q))
    assert e.value.code == -3
    q = torch.zeros(1, 2, 64, 128, dtype=torch.bfloat16, device=DEV)
    with pytest.raises(pa.AttnError) as e:   # output overlaps an input
        pa.attn_fwd_persistent_noalloc(q, q, q, q)
    assert e.value.code == -8
    with pytest.raises(pa.AttnError) as e:   # paired row blocks: dispatched grid only
        pa.attn_fwd_persistent_noalloc(q, q, q, torch.empty_like(q),
                                       mapping=pa.SWIZZLED_HEAD_FIRST | pa.PAIRED)
    assert e.value.code == -3
    with pytest.raises(ValueError):
        pa.attn_fwd_persistent_noalloc(q, q, q, None)
