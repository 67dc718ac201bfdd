// attn_bwd_common.h -- shared pieces of the backward kernels (attn_bwd.hip,
// attn_bwd_dq.hip): head-dimension constants, the dual swizzle of tiles that
// are read both as rows and transposed, and the transposed-operand and
// row-store helpers.  Device code only; each kernel file includes it once.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "attn_device.h"

namespace attn {
namespace bwd {

using namespace dev;

constexpr int D = 128;
constexpr int ROW_BYTES = D * 2;
constexpr int KSTEPS = D / 16;   // MFMA k-steps over the head dimension
constexpr int DBLK = D / 32;     // 32-row blocks of a transposed gradient
constexpr float kLog2e = 1.44269504088896340736f;

// The calling lane's index, computed where it is called: the volatile asm is
// neither hoisted nor merged with an earlier copy, so no register has to hold
// the lane index across a loop.
__device__ __forceinline__ int lane_index_here() {
    int l;
    asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(l));
    return l;
}

// Instruction classes of __builtin_amdgcn_sched_group_barrier.
constexpr int kSchedValu = 0x002;   // vector ALU, transcendentals excluded
constexpr int kSchedMfma = 0x008;
constexpr int kSchedDsRead = 0x100;
constexpr int kSchedTrans = 0x400;

// Chunk c (16 bytes) of row r of a tile is stored at c ^ dual_swizzle(r).
//  * 16-byte row reads: 16 consecutive rows, one logical chunk -> the 16
//    values of dual_swizzle over 16 consecutive rows are all distinct.
//  * transposing reads: 4 consecutive rows x 64 bytes per 32 lanes -> the
//    64-byte block index moves by (r & 3) and so differs between the rows.
__device__ __forceinline__ int dual_swizzle(int r) { return ((r & 3) << 2) | ((r >> 2) & 3); }

__device__ __forceinline__ uint32_t sw_off(int row, int byte) {
    return (uint32_t)(row * ROW_BYTES + ((((byte >> 4) ^ dual_swizzle(row)) << 4) | (byte & 15)));
}

// Global source offset (within a tile) of LDS slot `slot` (16 bytes) of a
// dual-swizzled tile: the copies fill LDS linearly and fetch the chunk that
// belongs there.
__device__ __forceinline__ uint32_t slot_src(int slot) {
    const int row = slot / 16;
    const int phys = slot % 16;
    return (uint32_t)(row * ROW_BYTES + ((phys ^ dual_swizzle(row)) << 4));
}

// Per-lane offsets of the transposing read of a dual-swizzled tile: lane i of
// 16-lane group gsel addresses row 4h + i/4 of a 16-row chunk (+8 rows for the
// upper half of the operand) and columns 32db + 16gsel + 4(i%4).  The chunk's
// first row (16kc + 8hi) is a multiple of 4, so the swizzle of the addressed
// row depends only on (i/4, h, hi) and the chunk offset is an immediate.
__device__ __forceinline__ void tr_offsets(int lane, uint32_t (&off)[DBLK][2]) {
    const int li = lane & 15;
    const int gsel = (lane >> 4) & 1;
    const int h = lane >> 5;
#pragma unroll
    for (int db = 0; db < DBLK; ++db)
#pragma unroll
        for (int hi = 0; hi < 2; ++hi) {
            const int row = 8 * hi + 4 * h + (li >> 2);   // row within a 16-row chunk
            const int byte = 64 * db + 32 * gsel + 8 * (li & 3);
            off[db][hi] = sw_off(row, byte) - 8 * hi * ROW_BYTES;
        }
}

// A operand rows 16kc.. of a transposing read (see tr_offsets).
__device__ __forceinline__ bf16x8 tr_operand(lds_char *base, const uint32_t (&off)[DBLK][2], int db,
                                             int kc) {
    const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
        (lds_bf16x4 *)(base + off[db][0] + 16 * kc * ROW_BYTES));
    const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
        (lds_bf16x4 *)(base + off[db][1] + (16 * kc + 8) * ROW_BYTES));
    return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
}

// Rows of a transposed accumulator (lane holds column c; register r of block
// db holds row 32db + 8(r/4) + 4h + r%4) scaled and stored as bf16 rows:
// `row` of the output head, bounded by the descriptor.
__device__ __forceinline__ void store_rows(const f32x16 (&acc)[DBLK], float s,
                                           __amdgpu_buffer_rsrc_t r, int row, int h) {
#pragma unroll
    for (int db = 0; db < DBLK; ++db) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const f32x4 v4 = {acc[db][4 * j + 0] * s, acc[db][4 * j + 1] * s,
                              acc[db][4 * j + 2] * s, acc[db][4 * j + 3] * s};
            const bf16x4 b4 = __builtin_convertvector(v4, bf16x4);
            const uint32_t off = (uint32_t)(row * D + 32 * db + 8 * j + 4 * h) * 2u;
            __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2, b4), r, (int)off, 0, 0);
        }
    }
}

}  // namespace bwd
}  // namespace attn
