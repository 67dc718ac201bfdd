// attn_fwd_pp.hip -- fused attention forward for gfx950, head dimension 128:
// two wave groups that alternate matrix-core and vector work ("ping-pong").
//
// Same result as the 4-wave kernel of attn_fwd.hip (Section 2.3, Eq. "eq:fa",
// with the FlashAttention-2 partition of Section 2.3.1 and the mappings of
// Sections 3.2 and 3.3), organised so that the two contractions run on the
// matrix cores while the softmax of another tile runs on the vector ALUs.
//
// Workgroup: 512 threads = 8 waves over BLOCK_M = 256 query rows.  Waves w and
// w+4 share a SIMD (the hardware places them so; checked on MI355X), wave w
// owns rows 32w..32w+31.  Group A = waves 0-3 (rows 0..127), group B = waves
// 4-7 (rows 128..255); both stream the same K/V tiles of 64 keys.
//
// Per tile j a group does two steps:
//   E(j): softmax of S(j): mask, P = exp2(...) against a lazily raised
//         reference maximum, the row sums of P, P -> bf16 (vector ALU);
//   G(j): S(j+1) = K(j+1) Q^T and O^T += V(j)^T P(j)^T (32 MFMAs).
// The groups run these one phase apart, phases separated by workgroup
// barriers:
//   phase 2k:   A: E(k)   B: G(k-1)
//   phase 2k+1: A: G(k)   B: E(k)
// so on every SIMD one wave feeds the matrix core while the other computes
// exponentials.  Both groups execute the same instruction stream (E, G, E,
// G, ...); only their first barrier differs.
//
// LDS: kStages stages of 32 KiB, stage j = {K(j+1), V(j)}, read in phases
// 2j+1 (A) and 2j+2 (B) and copied global -> LDS (buffer_load ... lds) kAhead
// stages ahead, inside the loop by group B alone, during its softmax step, so
// that group A's product step starts on MFMAs; optionally (kQInLds) the
// block's Q rows as well.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>

#include "attn_device.h"
#include "attn_internal.h"
#include "attn_numa.h"

namespace attn {
namespace {

using namespace dev;

constexpr int kPPThreads = 512;
// LDS operand reads issued this many MFMAs ahead in the product step.
constexpr int kPrefetch = 6;
// Q operands in LDS (true) or in registers (false).
constexpr bool kQInLds = false;
// K/V stages resident in LDS, and how many stages ahead each copy is issued.
constexpr int kStages = 2;
constexpr int kAhead = 1;
static_assert(kAhead >= 1 && kAhead < kStages, "a copy must not overwrite a stage in use");


// Waits and the workgroup barrier.  The copies into LDS are invisible to the
// compiler, so the waits are explicit; the barrier is a compiler memory fence
// but does not wait for outstanding copies.
// The scheduling barriers keep each step's instructions on its side of the
// workgroup barrier, so that the phases stay separated.
__device__ __forceinline__ void barrier_lds() {
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
}
__device__ __forceinline__ void barrier_lds_copies() {
    asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
}
// Pin a value's computation before this point: without it the compiler sinks
// the softmax arithmetic (and the MFMAs) next to their uses in the next step,
// across the barrier, which would merge the two phases again.
template <typename T>
__device__ __forceinline__ void anchor(T &x) {
    asm volatile("" : "+v"(x));
}

// Instruction-class masks of __builtin_amdgcn_sched_group_barrier.
constexpr int kSchedMfma = 0x008;
constexpr int kSchedDsRead = 0x100;

// LDS reads feeding MFMA i of the product step: a K chunk (one 16-byte read)
// for even i, a V column chunk (two transposing reads) for odd i.
__host__ __device__ constexpr int a_reads(int i) { return (i & 1) ? 2 : 1; }

// Scheduling groups of the product step (see gemm_step): the prologue reads,
// then per MFMA i the reads for MFMA i+PF (and, before each even k-step, the
// next Q operand) followed by MFMA i.
__host__ __device__ constexpr int prologue_reads(int pf) {
    int n = kQInLds ? 1 : 0;   // Q operand of k-step 0
    for (int i = 0; i < pf; ++i) n += a_reads(i);
    return n;
}
__host__ __device__ constexpr int step_reads(int pf, int i) {
    return (i + pf < 32 ? a_reads(i + pf) : 0) +
           ((kQInLds && (i & 1) == 0 && ((i >> 1) & 1) == 0 && (i >> 2) + 1 < 8) ? 1 : 0);
}
template <int PF, int I>
__device__ __forceinline__ void gemm_schedule_step() {
    if constexpr (I < 32) {
        constexpr int n = step_reads(PF, I);
        if constexpr (n > 0) __builtin_amdgcn_sched_group_barrier(kSchedDsRead, n, 0);
        __builtin_amdgcn_sched_group_barrier(kSchedMfma, 1, 0);
        gemm_schedule_step<PF, I + 1>();
    }
}
template <int PF>
__device__ __forceinline__ void gemm_schedule_impl() {
    __builtin_amdgcn_sched_group_barrier(kSchedDsRead, prologue_reads(PF), 0);
    gemm_schedule_step<PF, 0>();
}

// Wait until every copy this wave issued has landed in LDS.
__device__ __forceinline__ void wait_copies() {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

// LDS of one workgroup: kStages stages of a K and a V tile (64 x 128 bf16),
// plus the block's Q rows when kQInLds.
constexpr int kPPLdsBytes = kStages * 2 * kBlockN * 256 + (kQInLds ? kBlockM128 * 256 : 0);

// One tile (b, hq, m) of the output, with the LDS at `smem`.  It starts and
// ends with every wave at the same barrier count, so a workgroup can run it
// repeatedly (a paired slot, the persistent loop).
// B_COPIES: inside the loop group B issues every copy of a stage (the
// dispatched kernel); otherwise each group copies its own share (the
// persistent kernel, whose scalar registers are all in use: the extra LDS
// addresses of the first scheme would spill).
template <bool CAUSAL, bool B_COPIES>
__device__ __forceinline__ void pp_tile(const KernelArgs &p, const Tile t, char *smem) {
    constexpr int D = 128;
    constexpr int BM = kBlockM128;
    constexpr int BN = kBlockN;
    constexpr int KSTEPS = D / 16;
    constexpr int DBLK = D / 32;
    constexpr int CHUNKS_PER_ROW = D / 8;
    constexpr int ROW_BYTES = D * 2;
    constexpr int TILE_BYTES = BN * ROW_BYTES;
    constexpr int STAGE_BYTES = 2 * TILE_BYTES;
    constexpr int WAVES = kPPThreads / 64;
    constexpr int IPW = TILE_BYTES / 1024 / WAVES;   // copy instructions per wave per tile
    static_assert(IPW * 1024 * WAVES == TILE_BYTES, "tile not divisible");

    static_assert(kPPLdsBytes == kStages * STAGE_BYTES + (kQInLds ? BM * ROW_BYTES : 0),
                  "LDS layout");
    lds_char *const lds = (lds_char *)smem;
    lds_char *const q_lds = lds + kStages * STAGE_BYTES;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int grp = w >> 2;
    const int c = lane & 31;
    const int h = lane >> 5;

    const int g = t.hq / (p.Hq / p.Hkv);
    const int64_t q_head = ((int64_t)t.b * p.Hq + t.hq) * p.Sq * D;
    const int64_t kv_head = ((int64_t)t.b * p.Hkv + g) * p.Skv * D;
    const __amdgpu_buffer_rsrc_t ro = __builtin_amdgcn_make_buffer_rsrc(
        (void *)((char *)p.o + q_head * 2), 0, p.Sq * ROW_BYTES, kBufferFlags);

    // Q^T is the B operand of S^T = K Q^T: lane holds Q[row][16kk + 8h .. +7]
    // for each k-step, in registers (the default) or, with kQInLds, read from
    // the block's Q rows in LDS (same swizzle as K; each wave copies its own
    // 32 rows).
    const int q_wave0 = t.m * BM + 32 * w;
    const int my_q = q_wave0 + c;
    // Tile copies straight into LDS: each instruction of a wave fills 1024
    // contiguous LDS bytes (lane j at 16*j); wave w fills slots
    // (w*IPW + i)*64 + lane of a tile, fetching the global chunk that the
    // swizzled layout puts there.
    // Source offsets for this wave's slots (i < IPW) and, for a group-B wave,
    // for those of wave w - 4 (i >= IPW), which group B copies inside the loop.
    uint32_t k_src[2 * IPW], v_src[2 * IPW];
    const int w_other = w >= 4 ? w - 4 : w;
#pragma unroll
    for (int i = 0; i < 2 * IPW; ++i) {
        const int slot = ((i < IPW ? w : w_other) * IPW + (i % IPW)) * 64 + lane;
        const int row = slot / CHUNKS_PER_ROW;
        const int phys = slot % CHUNKS_PER_ROW;
        k_src[i] = row * ROW_BYTES + ((phys ^ k_swizzle<D>(row)) * 16);
        const int seg = (phys >> 1) ^ v_swizzle<D>(row);
        v_src[i] = row * ROW_BYTES + (seg * 2 + (phys & 1)) * 16;
    }
    const char *const k_head = (const char *)p.k + kv_head * 2;
    const char *const v_head = (const char *)p.v + kv_head * 2;
    const uint32_t kv_bytes = p.Skv * ROW_BYTES;
    const uint32_t lds_base = (uint32_t)(uintptr_t)lds;
    const int kv_end = CAUSAL ? min((t.m + 1) * BM, p.Skv) : p.Skv;
    const int n_tiles = (kv_end + BN - 1) / BN;
    // Tile n of K or V into LDS at byte offset dst.  The descriptor ends at the
    // block's last tile (or at Skv), so copies of tiles beyond write zeros and
    // fetch nothing (the last product step's K(n_tiles) among them).
    const uint32_t kv_lim = min(kv_bytes, (uint32_t)n_tiles * TILE_BYTES);
    auto copy_tile = [&](const char *head, const uint32_t *src, const int n, const uint32_t dst) __attribute__((always_inline)) {
        const uint32_t off = (uint32_t)n * TILE_BYTES;
        const uint32_t left = off < kv_lim ? kv_lim - off : 0u;
        const i32x4 d = buffer_words(head + (off < kv_lim ? off : 0u), left);
#pragma unroll
        for (int i = 0; i < IPW; ++i)
            lds_copy16(d, src[i], lds_base + dst + (w * IPW + i) * 1024);
    };
    // Tile n into both slot sets of a group-B wave (its own and wave w - 4's).
    auto copy_tile_both = [&](const char *head, const uint32_t *src, const int n, const uint32_t dst) __attribute__((always_inline)) {
        const uint32_t off = (uint32_t)n * TILE_BYTES;
        const uint32_t left = off < kv_lim ? kv_lim - off : 0u;
        const i32x4 d = buffer_words(head + (off < kv_lim ? off : 0u), left);
#pragma unroll
        for (int i = 0; i < 2 * IPW; ++i)
            lds_copy16(d, src[i], lds_base + dst + ((i < IPW ? w : w_other) * IPW + (i % IPW)) * 1024);
    };
    auto copy_stage_both = [&](const int j) __attribute__((always_inline)) {
        const uint32_t base = (uint32_t)(j % kStages) * STAGE_BYTES;
        copy_tile_both(k_head, k_src, j + 1, base);
        copy_tile_both(v_head, v_src, j, base + TILE_BYTES);
    };
    // Stage j = {K(j+1), V(j)} into buffer j % kStages.
    auto copy_stage = [&](const int j) __attribute__((always_inline)) {
        const uint32_t base = (uint32_t)(j % kStages) * STAGE_BYTES;
        copy_tile(k_head, k_src, j + 1, base);
        copy_tile(v_head, v_src, j, base + TILE_BYTES);
    };

    // Per-lane LDS read offsets.
    uint32_t k_off[KSTEPS];
#pragma unroll
    for (int kk = 0; kk < KSTEPS; ++kk)
        k_off[kk] = c * ROW_BYTES + (((2 * kk + h) ^ k_swizzle<D>(c)) * 16);
    const int li = lane & 15;
    const int gsel = (lane >> 4) & 1;
    uint32_t v_off[DBLK];
#pragma unroll
    for (int db = 0; db < DBLK; ++db)
        v_off[db] = (4 * h + (li >> 2)) * ROW_BYTES + 8 * (li & 3) +
                    (((2 * db + gsel) ^ v_swizzle<D>(4 * h + (li >> 2))) * 32);

    // This wave's Q rows in LDS; row c (the lane's query) uses the same swizzle
    // as K row c, so the Q operand offsets equal the K operand offsets.
    lds_char *const q_wave = q_lds + w * 32 * ROW_BYTES;
    bf16x8 qreg[kQInLds ? 1 : KSTEPS];
    if constexpr (!kQInLds) {
        const __amdgpu_buffer_rsrc_t rq = __builtin_amdgcn_make_buffer_rsrc(
            (void *)((const char *)p.q + q_head * 2), 0, p.Sq * ROW_BYTES, kBufferFlags);
#pragma unroll
        for (int kk = 0; kk < KSTEPS; ++kk)
            qreg[kk] = __builtin_bit_cast(
                bf16x8, load16(rq, (uint32_t)(my_q * D + 16 * kk + 8 * h) * 2u));
    }
    auto q_operand = [&](const int kk) __attribute__((always_inline)) -> bf16x8 {
        if constexpr (kQInLds) return *(const lds_bf16x8 *)(q_wave + k_off[kk]);
        else return qreg[kk];
    };

    f32x16 oacc[DBLK];
#pragma unroll
    for (int db = 0; db < DBLK; ++db)
        for (int r = 0; r < 16; ++r) oacc[db][r] = 0.0f;
    // Online-softmax state: a reference maximum m_ref that the exponentials
    // are taken against.  It is set from the first tile's row maximum and
    // raised (O and l rescaled) only when a tile's exponentials sum to more
    // than 2^24 for some lane, so the common step needs no maximum at all;
    // any reference gives the same result in exact arithmetic, because O and l
    // are divided by the same factor, and p <= 2^24 keeps fp32 sums far from
    // overflow.
    float m_ref = -__builtin_inff();
    float mb = -__builtin_inff();
    // Row sum of P over this lane's keys (the lane l^32 holds the row's other
    // keys; the two halves are added once, at the end).
    float lsum = 0.0f;
    const float sl2 = p.scale_log2;

    f32x16 s_cur[2];    // scores of the tile the next E step works on
    bf16x8 pbuf[4];     // P of the tile the next G step multiplies, 4 chunks of 16 keys

    // E(j): softmax of s_cur (tile j) into pbuf.
    auto softmax_step = [&](const int j) __attribute__((always_inline)) {
        const int key0 = j * BN;
        const bool need_mask = (key0 + BN > p.Skv) || (CAUSAL && key0 + BN - 1 > q_wave0);
        if (need_mask) {
#pragma unroll
            for (int kb2 = 0; kb2 < 2; ++kb2)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int key = key0 + 32 * kb2 + 8 * (r >> 2) + 4 * h + (r & 3);
                    const bool dead = key >= p.Skv || (CAUSAL && key > my_q);
                    s_cur[kb2][r] = dead ? -__builtin_inff() : s_cur[kb2][r];
                }
        }
        // Exponentials against the current reference and their sum over this
        // lane's keys.  The sum shows, without a maximum over the tile, whether
        // the reference is unset (first tile: inf/NaN) or a score exceeds it by
        // more than 2^24 in the exp2 domain; only then is the row maximum taken,
        // O and l rescaled and the exponentials recomputed.
        auto exps = [&](f32x8 (&p8)[4]) __attribute__((always_inline)) {
            float ts = 0.0f;
#pragma unroll
            for (int kc = 0; kc < 4; ++kc)
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    p8[kc][e] = exp2_hw(__builtin_fmaf(s_cur[kc >> 1][8 * (kc & 1) + e], sl2, -mb));
#pragma unroll
            for (int kc = 0; kc < 4; ++kc)
#pragma unroll
                for (int e = 0; e < 8; ++e) ts += p8[kc][e];
            return ts;
        };
        f32x8 p8[4];
        float tsum = exps(p8);
        if (__any(!(tsum <= 16777216.0f))) {
            float mx = s_cur[0][0];
#pragma unroll
            for (int kb2 = 0; kb2 < 2; ++kb2)
#pragma unroll
                for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s_cur[kb2][r]);
            const float m_new = fmaxf(m_ref, fmaxf(mx, xor32(mx)));
            const float alpha = exp2_hw((m_ref - m_new) * sl2);
            lsum *= alpha;
#pragma unroll
            for (int db = 0; db < DBLK; ++db)
#pragma unroll
                for (int r = 0; r < 16; ++r) oacc[db][r] *= alpha;
            m_ref = m_new;
            mb = m_ref * sl2;
            tsum = exps(p8);
        }
        lsum += tsum;
#pragma unroll
        for (int kc = 0; kc < 4; ++kc) pbuf[kc] = __builtin_convertvector(p8[kc], bf16x8);
#pragma unroll
        for (int kc = 0; kc < 4; ++kc) anchor(pbuf[kc]);
    };

    // G(j): S(j+1) = K(j+1) Q^T into s_cur (free once P(j) is formed) and
    // O^T += V(j)^T P(j)^T, stage j in LDS buffer (j % 2).  The 32 MFMAs
    // alternate between the two products (even i: scores, odd i: output) and
    // their A operands are read from LDS kPrefetch MFMAs ahead, so the matrix
    // core does not wait for LDS latency.
    auto gemm_step = [&](const int j, auto buf_c) __attribute__((always_inline)) {
        constexpr int BUF = decltype(buf_c)::value;   // j % kStages
        (void)j;
        lds_char *const kb = lds + BUF * STAGE_BYTES;
        lds_char *const vb = kb + TILE_BYTES;
        f32x16 (&s_next)[2] = s_cur;
        // A operand of MFMA i: a K row chunk (scores) or a V column chunk.
        auto a_operand = [&](const int i) __attribute__((always_inline)) -> bf16x8 {
            if ((i & 1) == 0) {
                const int si = i >> 1, kk = si >> 1, kb2 = si & 1;
                return *(const lds_bf16x8 *)(kb + k_off[kk] + kb2 * 32 * ROW_BYTES);
            }
            const int vi = i >> 1, kc = vi >> 2, db = vi & 3;
            const int chunk = 16 * kc * ROW_BYTES;
            const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
                (lds_bf16x4 *)(vb + v_off[db] + chunk));
            const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
                (lds_bf16x4 *)(vb + v_off[db] + chunk + 8 * ROW_BYTES));
            return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
        };
        // The wave feeding the matrix core gets issue priority over the
        // softmax wave sharing its SIMD (by default the older wave, group A,
        // would win every conflict and slow group B's MFMAs).
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_setprio(1);
        __builtin_amdgcn_sched_barrier(0);
        bf16x8 ring[kPrefetch];
        bf16x8 qop[2];
#pragma unroll
        for (int i = 0; i < kPrefetch; ++i) ring[i] = a_operand(i);
        qop[0] = q_operand(0);
#pragma unroll
        for (int i = 0; i < 32; ++i) {
            const bf16x8 a = ring[i % kPrefetch];
            if (i + kPrefetch < 32) ring[i % kPrefetch] = a_operand(i + kPrefetch);
            if ((i & 1) == 0) {
                const int si = i >> 1, kk = si >> 1, kb2 = si & 1;
                // the Q operand of the next k-step, read one score-MFMA pair ahead
                if (kb2 == 0 && kk + 1 < KSTEPS) qop[(kk + 1) & 1] = q_operand(kk + 1);
                const f32x16 zero = {};
                s_next[kb2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                    a, qop[kk & 1], kk == 0 ? zero : s_next[kb2], 0, 0, 0);
            } else {
                const int vi = i >> 1, kc = vi >> 2, db = vi & 3;
                oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pbuf[kc], oacc[db], 0, 0, 0);
            }
        }
        // Pin the order above: the prologue reads, then per MFMA i the reads
        // for MFMA i+kPrefetch (and the next Q operand) followed by MFMA i.
        gemm_schedule_impl<kPrefetch>();
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_setprio(0);
        __builtin_amdgcn_sched_barrier(0);
        anchor(s_next[0]);
        anchor(s_next[1]);
#pragma unroll
        for (int db = 0; db < DBLK; ++db) anchor(oacc[db]);

    };

    // Prologue: this wave's Q rows, K(0) into the K slot of buffer 1, stage 0
    // into buffer 0; S(0).
    if constexpr (kQInLds) {
        const char *const q_base = (const char *)p.q + q_head * 2;
        const uint32_t q_bytes = p.Sq * ROW_BYTES;
        const uint32_t off = (uint32_t)q_wave0 * ROW_BYTES;   // 32 rows = 8 KiB
        const i32x4 d = buffer_words(q_base + (off < q_bytes ? off : 0u),
                                     off < q_bytes ? q_bytes - off : 0u);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int slot = i * 64 + lane;                 // 16-byte slot within the 32 rows
            const int row = slot / CHUNKS_PER_ROW;
            const int phys = slot % CHUNKS_PER_ROW;
            lds_copy16(d, row * ROW_BYTES + ((phys ^ k_swizzle<D>(row)) * 16),
                       lds_base + 2 * STAGE_BYTES + w * 32 * ROW_BYTES + i * 1024);
        }
    }
    // K(0) goes into the K slot of the last buffer, which stage kStages-1
    // (issued after the scores of tile 0 are computed) later overwrites.
    copy_tile(k_head, k_src, 0, (kStages - 1) * STAGE_BYTES);
    for (int j = 0; j < kAhead && j < n_tiles; ++j) copy_stage(j);
    barrier_lds_copies();
    {
        lds_char *const kb = lds + (kStages - 1) * STAGE_BYTES;
#pragma unroll
        for (int kb2 = 0; kb2 < 2; ++kb2)
            for (int r = 0; r < 16; ++r) s_cur[kb2][r] = 0.0f;
#pragma unroll
        for (int kk = 0; kk < KSTEPS; ++kk) {
            const bf16x8 qop = q_operand(kk);
#pragma unroll
            for (int kb2 = 0; kb2 < 2; ++kb2) {
                const bf16x8 a = *(const lds_bf16x8 *)(kb + k_off[kk] + kb2 * 32 * ROW_BYTES);
                s_cur[kb2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qop, s_cur[kb2], 0, 0, 0);
            }
        }
    }

    // Every wave runs E(0) G(0) E(1) G(1) ... with a barrier after each step;
    // group B starts one barrier late (and group A ends with one extra), so
    // the groups stay one phase apart.  Stage k+1 is copied at global phase
    // 2k+1 into the buffer of stage k-1, which both groups finished reading by
    // phase 2k, and read from phase 2k+3 on.  With B_COPIES group B copies all
    // of it before its E(k) (each B wave fills its own slots and those of the
    // A wave on its SIMD), so A's product step starts on MFMAs; otherwise A
    // copies its share before G(k) and B its share before E(k).  Each wave
    // waits for its own copies before the barrier that ends phase 2k+2.
    static_assert(kAhead == 1, "every wave waits for all of its copies one phase after issuing them");
    if (grp == 1) barrier_lds();
    auto tile = [&](const int k, auto buf_c) __attribute__((always_inline)) {
        if (grp == 1 && k + 1 < n_tiles) {
            if constexpr (B_COPIES) copy_stage_both(k + 1);
            else copy_stage(k + 1);
        }
        softmax_step(k);
        // A's share of stage k, copied during G(k-1)
        if constexpr (!B_COPIES) if (grp == 0) wait_copies();
        barrier_lds();
        if constexpr (!B_COPIES) if (grp == 0 && k + 1 < n_tiles) copy_stage(k + 1);
        gemm_step(k, buf_c);
        if (grp == 1) wait_copies();
        barrier_lds();
    };
    // kStages tiles per trip, so that every LDS buffer offset is an immediate.
    static_assert(kStages == 2, "the trip below is written for two stages");
    for (int k = 0; k < n_tiles; k += 2) {
        tile(k, Int<0>{});
        if (k + 1 < n_tiles) tile(k + 1, Int<1>{});
    }
    if (grp == 0) barrier_lds();

    // O = acc / l, rounded to bf16; lane holds d = 32db + 8j + 4h + 0..3 of its row.
    // The wave's 32 rows are consecutive in O, so they leave through LDS as
    // whole rows: each store instruction then writes 1 KiB of consecutive
    // bytes instead of 32 separate 16-byte pieces.  After the last barrier no
    // wave reads the stage buffers and every copy into them has landed, so
    // wave w can use bytes [8 KiB w, 8 KiB (w+1)) of them; no other wave
    // touches that range before the next tile's prologue (a persistent
    // workgroup passes a barrier first).  Chunks are swizzled as in a K tile, so
    // the 16 chunks of a row that one read instruction takes hit distinct banks.
    const float l_tot = lsum + xor32(lsum);
    const float inv = 1.0f / l_tot;
    store_lse(p.lse == nullptr ? nullptr : p.lse + ((int64_t)t.b * p.Hq + t.hq) * p.Sq, p.Sq, my_q,
              lane, mb, l_tot);
    static_assert(WAVES * 32 * ROW_BYTES <= kStages * STAGE_BYTES, "O staging exceeds the stage buffers");
    lds_char *const ow = lds + w * 32 * ROW_BYTES;
#pragma unroll
    for (int db = 0; db < DBLK; ++db) {
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
            const f32x4 o4 = {oacc[db][4 * jj + 0] * inv, oacc[db][4 * jj + 1] * inv,
                              oacc[db][4 * jj + 2] * inv, oacc[db][4 * jj + 3] * inv};
            const bf16x4 ob = __builtin_convertvector(o4, bf16x4);
            const int q = 4 * db + jj;
            *(lds_u32x2 *)(ow + c * ROW_BYTES + ((q ^ k_swizzle<D>(c)) * 16) + 8 * h) =
                __builtin_bit_cast(u32x2, ob);
        }
    }
    // One wave's LDS accesses complete in order; this only keeps the compiler
    // from hoisting the reads above the writes of other lanes.
    asm volatile("" ::: "memory");
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int r = 4 * i + (lane >> 4);
        const int q = lane & 15;
        const u32x4 val = *(const lds_u32x4 *)(ow + r * ROW_BYTES + ((q ^ k_swizzle<D>(r)) * 16));
        __builtin_amdgcn_raw_buffer_store_b128(val, ro, (q_wave0 + r) * ROW_BYTES + q * 16, 0, 0);
    }
}

// With a probe buffer, thread 0 records (b, hq, m, XCC_ID) of workgroup `wid`
// (for a paired slot, its first tile).
__device__ __forceinline__ void record_probe(const KernelArgs &p, const int wid, const Tile t) {
    if (p.probe != nullptr && threadIdx.x == 0) {
        unsigned xcc;
        asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(xcc));
        int32_t *rec = p.probe + 4 * (int64_t)wid;
        rec[0] = t.b;
        rec[1] = t.hq;
        rec[2] = t.m;
        rec[3] = (int)(xcc & 0xf);
    }
}

// One workgroup per tile or, with kOrderPaired in ORDER, per pair slot: the
// slot's later (under a causal mask heavier) row block first, then its mirror.
template <bool CAUSAL, int MAPPING, int ORDER>
__global__ __launch_bounds__(kPPThreads, 1) void attn_fwd_pp_kernel(const KernelArgs p) {
    __shared__ __attribute__((aligned(1024))) char smem[kPPLdsBytes];
    const int wid = blockIdx.x;
    if constexpr ((ORDER & kOrderPaired) != 0) {
        Tile t = map_wid(MAPPING, ORDER, wid, p.B, p.Hq, pair_slots(p.NB), p.NX);
        const int slot = t.m;
        t.m = p.NB - 1 - slot;
        record_probe(p, wid, t);
        pp_tile<CAUSAL, true>(p, t, smem);
        if (slot != t.m) {
            // every wave is done with the first tile's LDS before the next copies land
            __syncthreads();
            t.m = slot;
            pp_tile<CAUSAL, true>(p, t, smem);
        }
    } else {
        const Tile t = map_wid(MAPPING, ORDER, wid, p.B, p.Hq, p.NB, p.NX);
        record_probe(p, wid, t);
        pp_tile<CAUSAL, true>(p, t, smem);
    }
}

// Persistent form: one workgroup per CU takes tiles from per-XCD queues
// instead of one workgroup per tile from the hardware dispatcher.  Queue x
// hands out, in order, the workgroup ids wid = x + NX*t (t = 0, 1, ...) that
// the dispatcher would send to XCD x, so every mapping keeps its placement,
// whatever order the hardware starts workgroups in.  A workgroup serves the
// queue of the XCD it runs on (XCC_ID) and, once that queue is empty, takes
// what is left in the others (so every tile is computed even if some XCD got
// no workgroup).  The ticket for the next tile is requested when a tile
// starts, so its latency hides behind the tile; the launch gap between
// workgroups (about 5 us on MI355X) disappears.  (The paired order is for
// the dispatched grid only: the queues balance the work by themselves.)
//
// p.queue: kQueueInts int32, zero before the launch; the last workgroup to
// finish sets it back to zero, so launches ordered on one stream can share it.
template <bool CAUSAL, int MAPPING, int ORDER>
__global__ __launch_bounds__(kPPThreads, 1) void attn_fwd_pp_persistent_kernel(const KernelArgs p) {
    __shared__ __attribute__((aligned(1024))) char smem[kPPLdsBytes];
    __shared__ int next_wid;
    const int N = p.B * p.Hq * p.NB;
    const int NX = p.NX;
    unsigned xcc;
    asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(xcc));
    const int x = (int)(xcc & 0xf) % NX;
    int *const queue = p.queue;
    // wid of ticket t of queue qx, or -1 past its end
    auto ticket_wid = [&](const int qx, const int tk) -> int {
        const int n_q = (N - qx + NX - 1) / NX;
        return tk < n_q ? qx + NX * tk : -1;
    };
    // Own queue first, then the others in turn.
    auto take = [&](int first_ticket) -> int {
        int w = ticket_wid(x, first_ticket);
        for (int i = 1; w < 0 && i < NX; ++i) {
            const int qx = (x + i) % NX;
            w = ticket_wid(qx, atomicAdd(&queue[qx], 1));
        }
        return w;
    };
    if (threadIdx.x == 0) next_wid = take(atomicAdd(&queue[x], 1));
    __syncthreads();
    int cur = next_wid;
    while (cur >= 0) {
        int pending = 0;
        if (threadIdx.x == 0) pending = atomicAdd(&queue[x], 1);   // result needed at the end
        const Tile t = map_wid(MAPPING, ORDER, cur, p.B, p.Hq, p.NB, p.NX);
        record_probe(p, cur, t);
        pp_tile<CAUSAL, false>(p, t, smem);
        if (threadIdx.x == 0) next_wid = take(pending);
        __syncthreads();
        cur = next_wid;
        __syncthreads();
    }
    // The last workgroup out clears the queue for the next launch.
    if (threadIdx.x == 0) {
        __threadfence();
        if (atomicAdd(&queue[kQueueDone], 1) == (int)gridDim.x - 1) {
            __threadfence();
            for (int i = 0; i < NX; ++i) atomicExch(&queue[i], 0);
            atomicExch(&queue[kQueueDone], 0);
        }
    }
}

template <bool CAUSAL, int MAPPING, int ORDER>
hipError_t launch_pp(const KernelArgs &a, int grid, hipStream_t stream) {
    if (a.queue != nullptr) {
        if constexpr ((ORDER & kOrderPaired) != 0) {
            return hipErrorInvalidValue;   // no paired persistent form
        } else {
            hipLaunchKernelGGL((attn_fwd_pp_persistent_kernel<CAUSAL, MAPPING, ORDER>),
                               dim3(grid), dim3(kPPThreads), 0, stream, a);
            return hipGetLastError();
        }
    }
    hipLaunchKernelGGL((attn_fwd_pp_kernel<CAUSAL, MAPPING, ORDER>), dim3(grid), dim3(kPPThreads),
                       0, stream, a);
    return hipGetLastError();
}

// The block-major order inside an XCD's piece exists for mapping 2 only.
template <bool CAUSAL, int MAPPING, int PAIRED>
hipError_t launch_pp_order(const KernelArgs &a, int grid, hipStream_t stream) {
    constexpr int HF = kOrderHeavyFirst;
    constexpr int BM = MAPPING == ATTN_MAP_SWIZZLED_HEAD_FIRST ? kOrderXcdBlockMajor : 0;
    const bool hf = (a.order & HF) != 0;
    if ((a.order & BM) != 0)
        return hf ? launch_pp<CAUSAL, MAPPING, PAIRED | BM | HF>(a, grid, stream)
                  : launch_pp<CAUSAL, MAPPING, PAIRED | BM>(a, grid, stream);
    return hf ? launch_pp<CAUSAL, MAPPING, PAIRED | HF>(a, grid, stream)
              : launch_pp<CAUSAL, MAPPING, PAIRED>(a, grid, stream);
}

template <bool CAUSAL, int MAPPING>
hipError_t launch_pp_paired(const KernelArgs &a, int grid, hipStream_t stream) {
    if ((a.order & kOrderPaired) != 0)
        return launch_pp_order<CAUSAL, MAPPING, kOrderPaired>(a, grid, stream);
    return launch_pp_order<CAUSAL, MAPPING, 0>(a, grid, stream);
}

template <bool CAUSAL>
hipError_t launch_pp_mapping(const KernelArgs &a, int mapping, int grid, hipStream_t stream) {
    switch (mapping) {
        case ATTN_MAP_NAIVE_BLOCK_FIRST: return launch_pp_paired<CAUSAL, 0>(a, grid, stream);
        case ATTN_MAP_NAIVE_HEAD_FIRST: return launch_pp_paired<CAUSAL, 1>(a, grid, stream);
        case ATTN_MAP_SWIZZLED_HEAD_FIRST: return launch_pp_paired<CAUSAL, 2>(a, grid, stream);
        default: return launch_pp_paired<CAUSAL, 3>(a, grid, stream);
    }
}

// The tile queues of attn_fwd_persistent_noalloc: a device array the library
// owns, for callers that cannot allocate device memory.  Every GPU holds its
// own copy (zero when the code object loads) until the process ends.  In host
// code `scratch` names a host-side stand-in, not the device address: the
// address comes from hipGetSymbolAddress, once per device (static_queue).
static __device__ __align__(256) int scratch[kQueueInts];

// Zeroes a queue buffer on the stream before a launch that uses it (a kernel,
// not hipMemsetAsync, so that the launch sequence can be captured in a graph).
__global__ __launch_bounds__(64, 1) void clear_queue_kernel(int *queue) {
    if (threadIdx.x < kQueueInts) queue[threadIdx.x] = 0;
}

}  // namespace

hipError_t static_queue(int **queue) {
    constexpr int kMaxDevices = 64;
    static std::mutex mu;
    static int *ptrs[kMaxDevices] = {};
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (ptrs[dev] == nullptr) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (p == nullptr) return hipErrorInvalidSymbol;
        ptrs[dev] = (int *)p;
    }
    *queue = ptrs[dev];
    return hipSuccess;
}

hipError_t launch_clear_queue(int *queue, hipStream_t stream) {
    hipLaunchKernelGGL(clear_queue_kernel, dim3(1), dim3(64), 0, stream, queue);
    return hipGetLastError();
}

hipError_t launch_attn_fwd_d128(const KernelArgs &a, bool causal, int mapping, int grid,
                                hipStream_t stream) {
    return causal ? launch_pp_mapping<true>(a, mapping, grid, stream)
                  : launch_pp_mapping<false>(a, mapping, grid, stream);
}

}  // namespace attn
