// attn_bwd_dq.hip -- the dQ kernel of the attention backward pass (gfx950,
// head dimension 128); the other two kernels and the pass's description are in
// attn_bwd.hip.
//
// dQ_i = scale sum_j dS_ij K_j (Section 2.3, Eq. "eq:ba"): one workgroup per
// (batch b, query head, block of 128 rows), streaming K and V tiles of 64 keys
// like the forward; S^T, dP^T (64 keys x 32 queries) = K Q^T, V dO^T with K, V
// rows from LDS and Q, dO in registers, dS^T = P^T o (dP^T - D), then
// dQ^T += K^T dS^T through the transposing read of the K tile.
//
// This file is compiled with the matrix-core results in ordinary vector
// registers (-mllvm --amdgpu-mfma-vgpr-form, set by the build).  Left to its
// heuristic the compiler puts every accumulator in AGPRs once a wave may use
// more than 256 registers, and the softmax then copies S and dP out and back on
// every tile; in vector registers the kernel needs 228, so two workgroups fit
// on a CU (__launch_bounds__(256, 2): two waves per SIMD) and one's vector work
// overlaps the other's matrix-core work.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "attn_bwd_common.h"
#include "attn_internal.h"
#include "attn_numa.h"

namespace attn {
namespace {

using namespace dev;
using namespace bwd;

// ---------------------------------------------------------------- dQ

constexpr int kRowsPerWg = 128;
constexpr int kKeyTile = 64;

template <bool CAUSAL, int MAPPING, int ORDER>
__global__ __launch_bounds__(256, 2) void attn_bwd_dq_kernel(const BwdArgs p) {
    constexpr int BN = kKeyTile;
    constexpr int TILE = BN * ROW_BYTES;   // 16 KiB: K or V rows of one tile
    constexpr int STAGE = 2 * TILE;
    constexpr int IPW = TILE / 1024 / 4;   // copy instructions per wave per tile
    __shared__ __attribute__((aligned(1024))) char smem[2 * STAGE];
    lds_char *const lds = (lds_char *)smem;
    const uint32_t lds_base = (uint32_t)(uintptr_t)lds;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int c = lane & 31;
    const int h = lane >> 5;

    const Tile t = map_wid(MAPPING, ORDER, blockIdx.x, p.B, p.Hq, p.NBQ, p.NX);
    const int g = t.hq / (p.Hq / p.Hkv);
    const int q_wave0 = t.m * kRowsPerWg + 32 * w;
    const int my_q = q_wave0 + c;

    const int64_t q_head = ((int64_t)t.b * p.Hq + t.hq) * p.Sq;   // row index of the head's row 0
    const int64_t kv_head = ((int64_t)t.b * p.Hkv + g) * p.Skv * D;
    const __amdgpu_buffer_rsrc_t rq = __builtin_amdgcn_make_buffer_rsrc(
        (void *)((const char *)p.q + q_head * ROW_BYTES), 0, p.Sq * ROW_BYTES, kBufferFlags);
    const __amdgpu_buffer_rsrc_t rdo = __builtin_amdgcn_make_buffer_rsrc(
        (void *)((const char *)p.dout + q_head * ROW_BYTES), 0, p.Sq * ROW_BYTES, kBufferFlags);
    const __amdgpu_buffer_rsrc_t rstat = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(p.lse + q_head), 0, p.Sq * 4, kBufferFlags);
    const __amdgpu_buffer_rsrc_t rdelta = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(p.delta + q_head), 0, p.Sq * 4, kBufferFlags);
    // Q and dO rows as B operands (lane: row my_q, columns 16kk + 8h .. +7);
    // rows past Sq read zeros, and so do their statistics.
    bf16x8 qreg[KSTEPS], doreg[KSTEPS];
#pragma unroll
    for (int kk = 0; kk < KSTEPS; ++kk) {
        const uint32_t off = (uint32_t)(my_q * D + 16 * kk + 8 * h) * 2u;
        qreg[kk] = __builtin_bit_cast(bf16x8, load16(rq, off));
        doreg[kk] = __builtin_bit_cast(bf16x8, load16(rdo, off));
    }
    const float lse2 = __builtin_bit_cast(
        float, __builtin_amdgcn_raw_buffer_load_b32(rstat, my_q * 4, 0, 0)) * kLog2e;
    const float dq_d = __builtin_bit_cast(
        float, __builtin_amdgcn_raw_buffer_load_b32(rdelta, my_q * 4, 0, 0));

    const int kv_end = CAUSAL ? min((t.m + 1) * kRowsPerWg, p.Skv) : p.Skv;
    const int n_tiles = (kv_end + BN - 1) / BN;
    const uint32_t kv_bytes = p.Skv * ROW_BYTES;
    const uint32_t kv_lim = min(kv_bytes, (uint32_t)n_tiles * TILE);
    uint32_t src[IPW];
#pragma unroll
    for (int i = 0; i < IPW; ++i) src[i] = slot_src((w * IPW + i) * 64 + lane);
    const char *const k_head = (const char *)p.k + kv_head * 2;
    const char *const v_head = (const char *)p.v + kv_head * 2;
    auto copy_tile = [&](const int n, const int buf) __attribute__((always_inline)) {
        const uint32_t off = (uint32_t)n * TILE;
        const uint32_t left = off < kv_lim ? kv_lim - off : 0u;
        const i32x4 dk_ = buffer_words(k_head + (off < kv_lim ? off : 0u), left);
        const i32x4 dv_ = buffer_words(v_head + (off < kv_lim ? off : 0u), left);
        const uint32_t dst = lds_base + buf * STAGE;
#pragma unroll
        for (int i = 0; i < IPW; ++i) {
            lds_copy16(dk_, src[i], dst + (w * IPW + i) * 1024);
            lds_copy16(dv_, src[i], dst + TILE + (w * IPW + i) * 1024);
        }
    };

    uint32_t row_off[KSTEPS];   // A operand rows: row c (+32 kb2), logical chunk 2kk + h
#pragma unroll
    for (int kk = 0; kk < KSTEPS; ++kk) row_off[kk] = sw_off(c, (2 * kk + h) * 16);
    uint32_t tro[DBLK][2];
    tr_offsets(lane, tro);

    f32x16 dqacc[DBLK];
#pragma unroll
    for (int db = 0; db < DBLK; ++db)
        for (int r = 0; r < 16; ++r) dqacc[db][r] = 0.0f;
    const float sl2 = p.scale_log2;

    auto compute = [&](const int n, auto buf_c) __attribute__((always_inline)) {
        constexpr int BUF = decltype(buf_c)::value;
        lds_char *const kb = lds + BUF * STAGE;
        lds_char *const vb = kb + TILE;
        f32x16 sacc[2] = {}, dpacc[2] = {};
#pragma unroll
        for (int kk = 0; kk < KSTEPS; ++kk) {
#pragma unroll
            for (int kb2 = 0; kb2 < 2; ++kb2) {
                const bf16x8 ak = *(const lds_bf16x8 *)(kb + row_off[kk] + kb2 * 32 * ROW_BYTES);
                sacc[kb2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ak, qreg[kk], sacc[kb2], 0, 0, 0);
                const bf16x8 av = *(const lds_bf16x8 *)(vb + row_off[kk] + kb2 * 32 * ROW_BYTES);
                dpacc[kb2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, doreg[kk], dpacc[kb2], 0, 0, 0);
            }
        }
        // Register r of block kb2 holds key 32kb2 + 8(r/4) + 4h + r%4 of the tile.
        // Key 32kb2 + 8(r/4) + 4h + r%4 of the tile is seen by the lane's row
        // iff 32kb2 + 8(r/4) + r%4 <= last_key (always, without a causal mask).
        const int key0 = n * BN;
        const int last_key = CAUSAL ? my_q - key0 - 4 * h : BN;
        f32x8 ds8[4];
#pragma unroll
        for (int kb2 = 0; kb2 < 2; ++kb2)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                float pr = exp2_hw(__builtin_fmaf(sacc[kb2][r], sl2, -lse2));
                if (CAUSAL && 32 * kb2 + 8 * (r >> 2) + (r & 3) > last_key) pr = 0.0f;
                ds8[2 * kb2 + (r >> 3)][r & 7] = pr * (dpacc[kb2][r] - dq_d);
            }
        bf16x8 dsb[4];
#pragma unroll
        for (int kc = 0; kc < 4; ++kc) dsb[kc] = __builtin_convertvector(ds8[kc], bf16x8);
#pragma unroll
        for (int kc = 0; kc < 4; ++kc)
#pragma unroll
            for (int db = 0; db < DBLK; ++db)
                dqacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(tr_operand(kb, tro, db, kc),
                                                                     dsb[kc], dqacc[db], 0, 0, 0);
    };

    copy_tile(0, 0);
    for (int n = 0; n < n_tiles; n += 2) {
        __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
        __syncthreads();
        if (n + 1 < n_tiles) copy_tile(n + 1, 1);
        compute(n, Int<0>{});
        if (n + 1 < n_tiles) {
            __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
            __syncthreads();
            if (n + 2 < n_tiles) copy_tile(n + 2, 0);
            compute(n + 1, Int<1>{});
        }
    }

    const __amdgpu_buffer_rsrc_t rdq = __builtin_amdgcn_make_buffer_rsrc(
        (void *)((char *)p.dq + q_head * ROW_BYTES), 0, p.Sq * ROW_BYTES, kBufferFlags);
    store_rows(dqacc, p.scale, rdq, my_q, h);
}

// ---------------------------------------------------------------- launchers

// The block-major order inside an XCD's piece exists for mapping 2 only.
template <bool CAUSAL, int MAPPING>
hipError_t launch_dq_order(const BwdArgs &a, hipStream_t stream) {
    const int g_q = a.B * a.Hq * a.NBQ;
    switch (MAPPING == ATTN_MAP_SWIZZLED_HEAD_FIRST ? a.order : (a.order & kOrderHeavyFirst)) {
        case 0:
            hipLaunchKernelGGL((attn_bwd_dq_kernel<CAUSAL, MAPPING, 0>), dim3(g_q), dim3(256), 0, stream, a);
            break;
        case 1:
            hipLaunchKernelGGL((attn_bwd_dq_kernel<CAUSAL, MAPPING, 1>), dim3(g_q), dim3(256), 0, stream, a);
            break;
        case 2:
            hipLaunchKernelGGL((attn_bwd_dq_kernel<CAUSAL, MAPPING, (MAPPING == 2 ? 2 : 0)>), dim3(g_q),
                               dim3(256), 0, stream, a);
            break;
        default:
            hipLaunchKernelGGL((attn_bwd_dq_kernel<CAUSAL, MAPPING, (MAPPING == 2 ? 3 : 1)>), dim3(g_q),
                               dim3(256), 0, stream, a);
            break;
    }
    return hipGetLastError();
}

template <bool CAUSAL>
hipError_t launch_dq_mapping(const BwdArgs &a, int mapping, hipStream_t stream) {
    switch (mapping) {
        case ATTN_MAP_NAIVE_BLOCK_FIRST: return launch_dq_order<CAUSAL, 0>(a, stream);
        case ATTN_MAP_NAIVE_HEAD_FIRST: return launch_dq_order<CAUSAL, 1>(a, stream);
        case ATTN_MAP_SWIZZLED_HEAD_FIRST: return launch_dq_order<CAUSAL, 2>(a, stream);
        default: return launch_dq_order<CAUSAL, 3>(a, stream);
    }
}

}  // namespace

hipError_t launch_attn_bwd_dq(const BwdArgs &a, bool causal, int mapping, hipStream_t stream) {
    return causal ? launch_dq_mapping<true>(a, mapping, stream)
                  : launch_dq_mapping<false>(a, mapping, stream);
}

}  // namespace attn
