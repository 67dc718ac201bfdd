// attn_bwd.hip -- attention backward pass for gfx950 (head dimension 128).
//
// Computes the gradients of Section 2.3, Eq. "eq:ba" for the forward of
// Eq. "eq:fa" (softmax scale, GQA, optional top-left causal mask), given dO,
// the forward output O and the forward's row log-sum-exp lse_i:
//   P_ij  = exp(scale s_ij - lse_i)              (recomputed, never stored)
//   dV_j  = sum_i P_ij dO_i
//   dP_ij = <dO_i, V_j>
//   dS_ij = P_ij (dP_ij - D_i),  D_i = <dO_i, O_i>  (= sum_j P_ij dP_ij)
//   dQ_i  = scale sum_j dS_ij K_j
//   dK_j  = scale sum_i dS_ij Q_i
// in three kernels on one stream:
//   1. D_i for every query row (vector ALU; HBM-bound);
//   2. dK, dV: one workgroup per (batch b, K/V head g, block of 128 keys) --
//      the FlashAttention-2 split of the backward over key blocks (Section
//      2.3.1); it streams every query head of the group and every query tile
//      of 32 rows through LDS, keeping the block's K and V rows in registers
//      and dK, dV in fp32 accumulators, so a GQA group's sum needs no atomics;
//   3. dQ: one workgroup per (b, query head, block of 128 rows), streaming
//      K and V tiles of 64 keys like the forward, dQ accumulated in registers
//      (attn_bwd_dq.hip, built with its own register-class option).
// Splitting dQ from dK/dV recomputes S and dP once more, but every output is
// written by exactly one workgroup in a fixed order: the gradients are
// deterministic and bitwise independent of the workgroup mapping.
//
// Placement: both gradient kernels decode their workgroup id with the forward's
// mappings (attn_internal.h), over (b, K/V head, key block) for dK/dV and over
// (b, query head, row block) for dQ, so workgroups sharing Q/dO (dK/dV) or
// K/V (dQ) stay on one XCD under swizzled head-first (Section 3.1: the
// backward's attention compute clusters).  ATTN_ORDER_HEAVY_FIRST reverses the
// row blocks of the dQ kernel as in the forward; the dK/dV kernel's natural
// order already starts with the most expensive causal key block.
//
// MFMA forms (v_mfma_f32_32x32x16_bf16):
//   dK/dV kernel, lanes <-> keys:
//     S  (32 q x 32 keys)  = Q_tile K^T      A = Q rows (LDS), B = K (registers)
//     dP (32 q x 32 keys)  = dO_tile V^T     A = dO rows (LDS), B = V (registers)
//     dV^T (128 x 32 keys) += dO^T P         A = dO^T (transposing LDS read), B = P
//     dK^T (128 x 32 keys) += Q^T dS         A = Q^T (transposing LDS read), B = dS
//   dQ kernel, lanes <-> queries:
//     S^T, dP^T (64 keys x 32 q) = K Q^T, V dO^T    A = K, V rows (LDS), B = Q, dO (registers)
//     dQ^T (128 x 32 q) += K^T dS^T                  A = K^T (transposing LDS read), B = dS^T
// The accumulator of S (or S^T) converted to bf16 is directly the B operand of
// the next product; the transposing reads pick the rows in the order of the
// accumulator's registers.  Tiles read both ways use dual_swizzle, under which
// both access patterns are free of LDS bank conflicts.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "attn_bwd_common.h"
#include "attn_internal.h"
#include "attn_numa.h"

namespace attn {
namespace {

using namespace dev;
using namespace bwd;

// ---------------------------------------------------------------- D = <dO, O>

__global__ __launch_bounds__(256) void attn_bwd_delta_kernel(const BwdArgs p) {
    const int64_t rows = (int64_t)p.B * p.Hq * p.Sq;
    const int64_t row = (int64_t)blockIdx.x * 16 + (threadIdx.x >> 4);
    const int part = threadIdx.x & 15;   // 16 bytes (8 elements) of the row
    float acc = 0.0f;
    if (row < rows) {
        const int64_t off = row * ROW_BYTES + part * 16;
        const bf16x8 x = __builtin_bit_cast(bf16x8, *(const u32x4 *)((const char *)p.o + off));
        const bf16x8 y = __builtin_bit_cast(bf16x8, *(const u32x4 *)((const char *)p.dout + off));
#pragma unroll
        for (int e = 0; e < 8; ++e) acc += (float)x[e] * (float)y[e];
    }
    acc += __shfl_xor(acc, 8, 16);
    acc += __shfl_xor(acc, 4, 16);
    acc += __shfl_xor(acc, 2, 16);
    acc += __shfl_xor(acc, 1, 16);
    if (row < rows && part == 0) p.delta[row] = acc;
}

// ---------------------------------------------------------------- dK, dV

constexpr int kKeysPerWg = 128;
constexpr int kQTile = 32;
// LDS operand reads issued ahead of the MFMA that consumes them, in MFMA steps.
constexpr int kReadAhead = 1;

// Declared for two waves per SIMD (two workgroups per CU), so a wave has 256
// registers: the block's K and V operands (64), the dK and dV accumulators
// (128), S and dP (32) and the operands in flight.  The LDS addresses are
// rebuilt per tile from three registers instead of sixteen (see compute), which
// keeps it within 256 without spills.
// Per query tile a wave computes S and dP, then P and dS of the tile's first 16
// rows, then the dV and dK MFMAs of those rows with the softmax of the other 16
// rows issued between them, then the MFMAs of the other rows.
template <bool CAUSAL, int MAPPING, int ORDER>
__global__ __launch_bounds__(256, 2) void attn_bwd_dkdv_kernel(const BwdArgs p) {
    constexpr int BQ = kQTile;
    constexpr int TILE = BQ * ROW_BYTES;          // 8 KiB: Q or dO rows of one tile
    constexpr int STAT = 1024;                     // 32 fp32 row statistics (one 64-lane copy)
    constexpr int STAGE = 2 * TILE + 2 * STAT;     // Q, dO, lse, D
    __shared__ __attribute__((aligned(1024))) char smem[2 * STAGE];
    lds_char *const lds = (lds_char *)smem;
    const uint32_t lds_base = (uint32_t)(uintptr_t)lds;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int c = lane & 31;
    const int h = lane >> 5;

    // (b, K/V head g, key block n); only the block-major order bit applies
    const Tile t = map_wid(MAPPING, ORDER, blockIdx.x, p.B, p.Hkv, p.NKV, p.NX);
    const int Gs = p.Hq / p.Hkv;
    const int k0 = t.m * kKeysPerWg;
    const int kw0 = k0 + 32 * w;
    const int my_key = kw0 + c;

    const int64_t kv_head = ((int64_t)t.b * p.Hkv + t.hq) * p.Skv * D;
    const __amdgpu_buffer_rsrc_t rk = __builtin_amdgcn_make_buffer_rsrc(
        (void *)((const char *)p.k + kv_head * 2), 0, p.Skv * ROW_BYTES, kBufferFlags);
    const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc(
        (void *)((const char *)p.v + kv_head * 2), 0, p.Skv * ROW_BYTES, kBufferFlags);
    // K, V rows of this wave as B operands: lane holds key my_key, columns 16kk + 8h .. +7.
    bf16x8 kreg[KSTEPS], vreg[KSTEPS];
#pragma unroll
    for (int kk = 0; kk < KSTEPS; ++kk) {
        const uint32_t off = (uint32_t)(my_key * D + 16 * kk + 8 * h) * 2u;
        kreg[kk] = __builtin_bit_cast(bf16x8, load16(rk, off));
        vreg[kk] = __builtin_bit_cast(bf16x8, load16(rv, off));
    }

    // Query tiles: every query head of the group, rows from the block's first
    // key on (causal) or all rows.
    const int qt_begin = CAUSAL ? k0 / BQ : 0;
    const int qt_end = (p.Sq + BQ - 1) / BQ;
    const int n_qt = qt_end > qt_begin ? qt_end - qt_begin : 0;
    const int total = Gs * n_qt;

    // Copies of tile tt into stage buffer `buf`: wave w fills 1 KiB slots 2w,
    // 2w+1 of the Q and dO tiles; wave 0 the lse rows, wave 1 the D rows (one
    // 64-lane copy each; lanes past the 32 rows read zeros).
    uint32_t src[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) src[i] = slot_src((2 * w + i) * 64 + lane);
    auto copy_tile = [&](const int tt, const int buf) __attribute__((always_inline)) {
        const int hq = t.hq * Gs + tt / n_qt;
        const int q0 = (qt_begin + tt % n_qt) * BQ;
        const int64_t row0 = ((int64_t)t.b * p.Hq + hq) * p.Sq + q0;
        const uint32_t left = (uint32_t)(p.Sq - q0) * ROW_BYTES;
        const uint32_t dst = lds_base + buf * STAGE;
        const i32x4 dq = buffer_words((const char *)p.q + row0 * ROW_BYTES, left);
        const i32x4 ddo = buffer_words((const char *)p.dout + row0 * ROW_BYTES, left);
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            lds_copy16(dq, src[i], dst + (2 * w + i) * 1024);
            lds_copy16(ddo, src[i], dst + TILE + (2 * w + i) * 1024);
        }
        const uint32_t nrows = (uint32_t)min(BQ, p.Sq - q0);
        if (w == 0) lds_copy16(buffer_words(p.lse + row0, nrows * 4), lane * 16, dst + 2 * TILE);
        if (w == 1)
            lds_copy16(buffer_words(p.delta + row0, nrows * 4), lane * 16, dst + 2 * TILE + STAT);
    };

    // A operand rows of the S and dP products: row c, logical chunk 2kk + h,
    // at sw_off(c, 32kk + 16h) = rb ^ 32kk, since the chunk index reaches the
    // offset (bits 4-7) only through an XOR with the row's swizzle.  For the
    // same reason the transposing reads' offsets are tro[db][hi] = tb[hi] ^ 64db.
    uint32_t rb = sw_off(c, 16 * h);
    uint32_t tb[2];
    {
        uint32_t tro0[DBLK][2];
        tr_offsets(lane, tro0);
        tb[0] = tro0[0][0];
        tb[1] = tro0[0][1];
    }

    f32x16 dvacc[DBLK], dkacc[DBLK];
#pragma unroll
    for (int db = 0; db < DBLK; ++db)
        for (int r = 0; r < 16; ++r) dvacc[db][r] = dkacc[db][r] = 0.0f;
    const float sl2 = p.scale_log2;

    auto compute = [&](const int tt, auto buf_c) __attribute__((always_inline)) {
        constexpr int BUF = decltype(buf_c)::value;
        const int q0 = (qt_begin + tt % n_qt) * BQ;
        // Rows before the wave's first key see none of its keys (causal).
        if (CAUSAL && q0 + BQ - 1 < kw0) return;
        lds_char *const qb = lds + BUF * STAGE;
        lds_char *const dob = qb + TILE;
        lds_char *const lseb = qb + 2 * TILE;
        lds_char *const db_ = lseb + STAT;

        // Offsets rebuilt for this tile (one XOR per read), each set right
        // before the step that uses it, rather than held in sixteen registers
        // across the loop: the empty asm hides that they are loop invariant.
        asm volatile("" : "+v"(rb));
        uint32_t row_off[KSTEPS];
#pragma unroll
        for (int kk = 0; kk < KSTEPS; ++kk) row_off[kk] = rb ^ (uint32_t)(32 * kk);

        // S and dP.  Each step's two A operands are read kReadAhead steps
        // before its two MFMAs (pinned by the group barriers); left to itself
        // the compiler waits for every read right before its MFMA.
        f32x16 sacc = {}, dpacc = {};
        __builtin_amdgcn_sched_barrier(0);
        {
            bf16x8 aq[KSTEPS], ado[KSTEPS];
#pragma unroll
            for (int kk = 0; kk < KSTEPS; ++kk) {
                aq[kk] = *(const lds_bf16x8 *)(qb + row_off[kk]);
                ado[kk] = *(const lds_bf16x8 *)(dob + row_off[kk]);
            }
#pragma unroll
            for (int kk = 0; kk < KSTEPS; ++kk) {
                sacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(aq[kk], kreg[kk], sacc, 0, 0, 0);
                dpacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ado[kk], vreg[kk], dpacc, 0, 0, 0);
            }
            __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 2 * kReadAhead, 0);
#pragma unroll
            for (int kk = 0; kk < KSTEPS; ++kk) {
                __builtin_amdgcn_sched_group_barrier(kSchedMfma, 2, 0);
                if (kk + kReadAhead < KSTEPS) __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 2, 0);
            }
        }
        __builtin_amdgcn_sched_barrier(0);
        // Register r holds query row 8(r/4) + 4h + r%4 of the tile, so
        // registers 8kc..8kc+7 are rows 16kc..16kc+15: the k-block kc of the
        // dV and dK products.  Row 8j + 4h + e of the tile sees the lane's key
        // iff 8j + e >= first_row (no row is masked when first_row <= 0, e.g.
        // without a causal mask).
        const int first_row = CAUSAL ? my_key - q0 - 4 * h : 0;
        f32x4 lse4[4], d4[4];   // statistics of rows 8j + 4h .. +3
        auto read_stats = [&](const int kc) __attribute__((always_inline)) {
#pragma unroll
            for (int j = 2 * kc; j < 2 * kc + 2; ++j) {
                lse4[j] = *(const lds_f32x4 *)(lseb + (8 * j + 4 * h) * 4);
                d4[j] = *(const lds_f32x4 *)(db_ + (8 * j + 4 * h) * 4);
            }
        };
        // P and dS of k-block kc, as bf16 B operands
        bf16x8 pb[2], dsb[2];
        auto softmax_block = [&](auto kc_c) __attribute__((always_inline)) {
            constexpr int KC = decltype(kc_c)::value;
            f32x8 p8, ds8;
#pragma unroll
            for (int j = 2 * KC; j < 2 * KC + 2; ++j)
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int r = 4 * j + e;
                    float pr = exp2_hw(__builtin_fmaf(sacc[r], sl2, -lse4[j][e] * kLog2e));
                    if (CAUSAL && 8 * j + e < first_row) pr = 0.0f;
                    p8[r & 7] = pr;
                    ds8[r & 7] = pr * (dpacc[r] - d4[j][e]);
                }
            pb[KC] = __builtin_convertvector(p8, bf16x8);
            dsb[KC] = __builtin_convertvector(ds8, bf16x8);
        };
        // k-block 0 now; k-block 1's statistics are read here and its softmax
        // runs between the k-block 0 MFMAs below.
        read_stats(0);
        softmax_block(Int<0>{});
        __builtin_amdgcn_sched_barrier(0);
        read_stats(1);
        // dV and dK, each MFMA's transposed operand (two reads) read
        // kReadAhead MFMAs ahead, and k-block 1's softmax spread over the
        // k-block 0 MFMAs, which need only k-block 0's P and dS.
        constexpr int NPROD = 2 * 2 * DBLK;
        asm volatile("" : "+v"(tb[0]), "+v"(tb[1]));
        uint32_t tro[DBLK][2];
#pragma unroll
        for (int db = 0; db < DBLK; ++db) {
            tro[db][0] = tb[0] ^ (uint32_t)(64 * db);
            tro[db][1] = tb[1] ^ (uint32_t)(64 * db);
        }
        __builtin_amdgcn_sched_barrier(0);
        {
            bf16x8 av[2][DBLK], ak[2][DBLK];
#pragma unroll
            for (int kc = 0; kc < 2; ++kc)
#pragma unroll
                for (int db = 0; db < DBLK; ++db) {
                    av[kc][db] = tr_operand(dob, tro, db, kc);
                    ak[kc][db] = tr_operand(qb, tro, db, kc);
                }
            softmax_block(Int<1>{});
#pragma unroll
            for (int kc = 0; kc < 2; ++kc)
#pragma unroll
                for (int db = 0; db < DBLK; ++db) {
                    dvacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av[kc][db], pb[kc], dvacc[db],
                                                                         0, 0, 0);
                    dkacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ak[kc][db], dsb[kc], dkacc[db],
                                                                         0, 0, 0);
                }
            __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 2 * kReadAhead, 0);
#pragma unroll
            for (int i = 0; i < NPROD; ++i) {
                __builtin_amdgcn_sched_group_barrier(kSchedMfma, 1, 0);
                if (i + kReadAhead < NPROD) __builtin_amdgcn_sched_group_barrier(kSchedDsRead, 2, 0);
                if (i < NPROD / 2) {
                    __builtin_amdgcn_sched_group_barrier(kSchedValu, 8, 0);
                    __builtin_amdgcn_sched_group_barrier(kSchedTrans, 1, 0);
                }
            }
        }
        __builtin_amdgcn_sched_barrier(0);
    };

    if (total > 0) copy_tile(0, 0);
    for (int tt = 0; tt < total; tt += 2) {
        __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
        __syncthreads();
        if (tt + 1 < total) copy_tile(tt + 1, 1);
        compute(tt, Int<0>{});
        if (tt + 1 < total) {
            __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
            __syncthreads();
            if (tt + 2 < total) copy_tile(tt + 2, 0);
            compute(tt + 1, Int<1>{});
        }
    }
    // no copy is left in flight here: the last tile's copies were waited for

    const __amdgpu_buffer_rsrc_t rdk = __builtin_amdgcn_make_buffer_rsrc(
        (void *)((char *)p.dk + kv_head * 2), 0, p.Skv * ROW_BYTES, kBufferFlags);
    const __amdgpu_buffer_rsrc_t rdv = __builtin_amdgcn_make_buffer_rsrc(
        (void *)((char *)p.dv + kv_head * 2), 0, p.Skv * ROW_BYTES, kBufferFlags);
    // Without the causal mask the loop does not use the lane's key: rebuilt
    // here instead of held in a register across the loop.
    const int key_e = CAUSAL ? my_key : kw0 + (lane_index_here() & 31);
    store_rows(dkacc, p.scale, rdk, key_e, h);
    store_rows(dvacc, 1.0f, rdv, key_e, h);
}

// ---------------------------------------------------------------- launchers

template <bool CAUSAL, int MAPPING, int ORDER>
hipError_t launch_grads(const BwdArgs &a, hipStream_t stream) {
    const int g_kv = a.B * a.Hkv * a.NKV;
    // The dK/dV kernel's natural order already starts with the heaviest causal
    // key block; it takes only the block-major bit.
    hipLaunchKernelGGL((attn_bwd_dkdv_kernel<CAUSAL, MAPPING, (ORDER & kOrderXcdBlockMajor)>),
                       dim3(g_kv), dim3(256), 0, stream, a);
    return hipGetLastError();
}

// The block-major order inside an XCD's piece exists for mapping 2 only.
template <bool CAUSAL, int MAPPING>
hipError_t launch_grads_order(const BwdArgs &a, hipStream_t stream) {
    switch (MAPPING == ATTN_MAP_SWIZZLED_HEAD_FIRST ? a.order : (a.order & kOrderHeavyFirst)) {
        case 0: return launch_grads<CAUSAL, MAPPING, 0>(a, stream);
        case 1: return launch_grads<CAUSAL, MAPPING, 1>(a, stream);
        case 2: return launch_grads<CAUSAL, MAPPING, (MAPPING == 2 ? 2 : 0)>(a, stream);
        default: return launch_grads<CAUSAL, MAPPING, (MAPPING == 2 ? 3 : 1)>(a, stream);
    }
}

template <bool CAUSAL>
hipError_t launch_grads_mapping(const BwdArgs &a, int mapping, hipStream_t stream) {
    switch (mapping) {
        case ATTN_MAP_NAIVE_BLOCK_FIRST: return launch_grads_order<CAUSAL, 0>(a, stream);
        case ATTN_MAP_NAIVE_HEAD_FIRST: return launch_grads_order<CAUSAL, 1>(a, stream);
        case ATTN_MAP_SWIZZLED_HEAD_FIRST: return launch_grads_order<CAUSAL, 2>(a, stream);
        default: return launch_grads_order<CAUSAL, 3>(a, stream);
    }
}

}  // namespace

hipError_t launch_attn_bwd(const BwdArgs &a, bool causal, int mapping, hipStream_t stream) {
    const int64_t rows = (int64_t)a.B * a.Hq * a.Sq;
    hipLaunchKernelGGL(attn_bwd_delta_kernel, dim3((unsigned)((rows + 15) / 16)), dim3(256), 0,
                       stream, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    e = causal ? launch_grads_mapping<true>(a, mapping, stream)
               : launch_grads_mapping<false>(a, mapping, stream);
    if (e != hipSuccess) return e;
    return launch_attn_bwd_dq(a, causal, mapping, stream);
}

}  // namespace attn
