// attn_calib.h -- launcher of the matrix-core calibration kernel (attn_calib.hip).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace attn {

constexpr int kCalibThreads = 512;       // 8 waves: two per SIMD
constexpr int kCalibMaxGrid = 65536;
constexpr int kCalibMaxIters = 1 << 24;

// grid workgroups of kCalibThreads; iters a positive multiple of 4.
// rec: 4*grid int64, sink: kCalibThreads*grid float (device memory).
hipError_t launch_calib_mfma(int grid, int iters, int64_t *rec, float *sink, hipStream_t stream);

}  // namespace attn
