// attn_calib.hip -- calibration of the compute ceiling of the roofline: the
// dense bf16 matrix-core rate the chip sustains, and the shader clock it runs
// at meanwhile.
//
// The published dense bf16 peak (2.5 PFLOP/s on MI355X) assumes the 2.4 GHz
// peak engine clock.  Under a sustained matrix-core load the power manager
// runs the chip at a lower clock, so no kernel reaches that figure.  This
// kernel issues only independent 32x32x16 bf16 MFMAs on register operands (no
// memory or LDS traffic) and records, per workgroup, the 100 MHz real-time
// counter and the shader-clock counter at its start and end; their ratio is
// the clock the workgroup ran at.  It is not part of the attention method.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "attn_calib.h"
#include "attn_device.h"

namespace attn {
namespace {

using dev::bf16x8;
using dev::f32x16;

// Each wave: 4 accumulators, 4 A and 4 B operands, iters/4 trips of 16 MFMAs
// (4*iters per wave).  The operand pairs rotate so that consecutive MFMAs see
// different data, as in a real contraction.
__global__ __launch_bounds__(kCalibThreads, 1) void calib_mfma_kernel(float *sink, int64_t *rec,
                                                                      int iters) {
    const long long r0 = __builtin_amdgcn_s_memrealtime();
    const long long c0 = __builtin_amdgcn_s_memtime();
    const int lane = threadIdx.x & 63;
    bf16x8 a[4], b[4];
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const unsigned hsh = ((unsigned)lane * 2654435761u) ^
                                 (unsigned)(u * 40503 + e * 977 + (int)threadIdx.x * 7);
            a[u][e] = (__bf16)((float)((int)(hsh & 255u) - 128) * (1.0f / 64.0f));
            b[u][e] = (__bf16)((float)((int)((hsh >> 8) & 255u) - 128) * (1.0f / 64.0f));
        }
    f32x16 acc[4];
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[u][r] = 0.0f;
    for (int it = 0; it < iters; it += 4) {
#pragma unroll
        for (int s = 0; s < 4; ++s)
#pragma unroll
            for (int u = 0; u < 4; ++u)
                acc[u] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[(u + s) & 3], b[(u + 2 * s) & 3],
                                                                acc[u], 0, 0, 0);
    }
    float total = 0.0f;
#pragma unroll
    for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int r = 0; r < 16; ++r) total += acc[u][r];
    sink[(int64_t)blockIdx.x * kCalibThreads + threadIdx.x] = total;
    if (threadIdx.x == 0) {
        int64_t *const w = rec + 4 * (int64_t)blockIdx.x;
        w[0] = r0;
        w[1] = __builtin_amdgcn_s_memrealtime();
        w[2] = c0;
        w[3] = __builtin_amdgcn_s_memtime();
    }
}

}  // namespace

hipError_t launch_calib_mfma(int grid, int iters, int64_t *rec, float *sink, hipStream_t stream) {
    hipLaunchKernelGGL(calib_mfma_kernel, dim3(grid), dim3(kCalibThreads), 0, stream, sink, rec,
                       iters);
    return hipGetLastError();
}

}  // namespace attn
