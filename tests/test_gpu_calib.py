"""GPU check of the matrix-core calibration (attn_calib_mfma) that bench.py
reads the roofline against: every workgroup records both counters, the clock
they give lies in the chip's range, and the measured rate respects the
per-clock limit of the compute units it ran on (1024 dense bf16 flop per
cycle per SIMD, four SIMDs per CU)."""

import numpy as np
import pytest
import torch

import paper_2511_02132_amd as pa

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def test_calib_records_and_rate():
    print("calib grid 64 iters 400", flush=True)
    grid, iters = 64, 400
    res = pa.calib_mfma(DEV, grid=grid, iters=iters, launches=3)
    assert len(res) == 3
    for r in res:
        assert 300.0 < r["clock_mhz"] < 2600.0, r
        assert r["ms"] > 0 and r["tflops"] > 0, r
        limit = grid * 4 * 1024 * r["clock_mhz"] * 1e6 / 1e12    # TFLOP/s at that clock
        assert r["tflops"] <= 1.05 * limit, (r, limit)


def test_calib_writes_every_record():
    print("calib records", flush=True)
    grid = 300
    rec = torch.full((grid, 4), -1, dtype=torch.int64, device=DEV)
    sink = torch.full((grid * pa.CALIB_THREADS,), float("nan"), dtype=torch.float32, device=DEV)
    pa.lib().attn_set_stream(None)
    assert pa.lib().attn_calib_mfma(grid, 8, rec.data_ptr(), sink.data_ptr()) == 0
    torch.cuda.synchronize()
    r = rec.cpu().numpy()
    assert (r[:, 1] > r[:, 0]).all() and (r[:, 3] > r[:, 2]).all()
    assert np.isfinite(sink.cpu().numpy()).all()
