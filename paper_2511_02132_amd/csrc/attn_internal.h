// attn_internal.h -- declarations shared by the host launcher and the kernels
// of libattn_numa.so (not part of the public C ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace attn {

// Query rows per workgroup and keys per K/V tile.  Section 4.3 uses 128 x 64;
// the head-dimension-128 kernel runs two wave groups over 256 rows per
// workgroup so that each K/V tile copied into LDS serves twice as many rows.
constexpr int kBlockM = 128;      // d = 64 (4 waves)
constexpr int kBlockM128 = 256;   // d = 128 (8 waves, two groups)
constexpr int kBlockN = 64;
constexpr int kMaxBlockM = 256;

__host__ __device__ constexpr int block_m_for(int d) { return d == 128 ? kBlockM128 : kBlockM; }

// Kernel arguments; tensors are bf16, BHSD contiguous.
struct KernelArgs {
    const void *q;
    const void *k;
    const void *v;
    void *o;
    int32_t *probe;   // NULL, or 4 int32 per workgroup: b, hq, m, xcc
    float *lse;       // NULL, or [B][Hq][Sq] fp32: log sum_j exp(scale * s_ij) per row
    int *queue;       // NULL (one workgroup per tile), or the persistent form's tile queues
    int B, Hq, Hkv, Sq, Skv;
    int NB;           // ceil(Sq / block_m_for(d))
    int NX;           // XCD count used by the mapping
    int order;        // kOrder* bits of the ATTN_ORDER_* flags
    float scale_log2; // scale * log2(e): softmax evaluated with exp2
};

struct Tile {
    int b, hq, m;
};

// Persistent launch: int32 words of the queue buffer -- one ticket counter per
// XCD (at most kQueueMaxXcd) and a count of finished workgroups.
constexpr int kQueueMaxXcd = 32;
constexpr int kQueueDone = kQueueMaxXcd;
constexpr int kQueueInts = 64;

// Order bits (from ATTN_ORDER_HEAVY_FIRST, ATTN_ORDER_XCD_BLOCK_MAJOR and
// ATTN_ORDER_PAIRED).
constexpr int kOrderHeavyFirst = 1;
constexpr int kOrderXcdBlockMajor = 2;
// Paired row blocks (head dimension 128, forward): the grid has
// pair_slots(NB) slots per head instead of NB row blocks; map_wid decodes a
// workgroup id over (B, Hq, pair_slots(NB)) with the other order bits, and
// slot p computes row block NB-1-p and then row block p (once, when the two
// coincide).  Under a causal mask with Sq == Skv every pair costs the same
// NB+1 block-widths of K/V (the middle block of an odd NB costs about half).
constexpr int kOrderPaired = 4;

__host__ __device__ constexpr int pair_slots(int NB) { return (NB + 1) / 2; }
// Heads per block-major group: one per shader engine of an XCD; for heads of
// at most kShortHeadBlocks row blocks, kBlockMajorHeadsShort.
constexpr int kBlockMajorHeads = 4;
constexpr int kBlockMajorHeadsShort = 16;
constexpr int kShortHeadBlocks = 16;
// Block-major groups apply only up to this many row blocks per head.
constexpr int kBlockMajorMaxBlocks = 64;

// Workgroup id -> tile (b, hq, m) for base mapping 0..3 (ATTN_MAP_*);
// integer only.  In the kernel the arguments are uniform, so this runs on the
// scalar unit.
//   0 naive block-first:   digits of wid over (B, NB, Hq), heads fastest
//   1 naive head-first:    digits of wid over (B, Hq, NB), blocks fastest
//   2 swizzled head-first: digits over (B, Hq, NB) of the rank of wid in the
//     XCD-major listing of the grid (XCD x = wid mod NX receives its k-th WG
//     as wid = x + k*NX; the first N mod NX XCDs hold one WG more).
//   3 swizzled block-first: as 0, but within each (b, m) row of Hq WGs the
//     position j takes head (j mod NX)*qh + min(j mod NX, rh) + j div NX,
//     (qh, rh) = divmod(Hq, NX): the WGs of a row that one XCD receives carry
//     contiguous heads, so a GQA group stays on one XCD when Hkv == NX.
// Order bits:
//  kOrderXcdBlockMajor (mapping 2 only): when XCD x's piece of the head-major
//    order consists of whole heads (hx of them), the piece is cut into groups
//    of G consecutive heads (the last group may be smaller) and each group is
//    dispatched block-major: within a group of g heads, its
//    j-th WG takes the group's head j mod g and block j div g.  Same tiles on
//    the same XCD, different order inside the XCD.  The hardware hands an XCD
//    its WGs in order, one per shader engine in turn (four per XCD); with this
//    order four consecutive WGs cover one row block of four heads and cost the
//    same under a causal mask, while the WGs in flight still share the K/V of
//    only four heads.  G = kBlockMajorHeads (4), or, with short_groups (set for
//    the 128-row blocks of head dimension 56 and 64, four WGs per CU),
//    kBlockMajorHeadsShort (16) for heads of at most kShortHeadBlocks row
//    blocks: such heads finish their blocks quickly, a heavy-first prefix over
//    more heads balances the CUs better, and their K/V streams are short.  (At
//    d = 128 a head of 16 row blocks streams 2 MiB of K/V and 16 of them
//    overflow the L2.)  Pieces that are not whole
//    heads, and heads of more than kBlockMajorMaxBlocks row blocks, keep the
//    head-major order: the engine imbalance that head-major order leaves is
//    about 6/NB of the work, and at long contexts four K/V streams in flight
//    cost more L2 hits than that.
//  kOrderHeavyFirst then replaces m by NB-1-m: the XCD of every (b, hq) is
//    unchanged, but each head's row blocks are dispatched from the last (under
//    a causal mask the most expensive) to the first.
__host__ __device__ inline Tile map_wid(int mapping, int order, int wid, int B, int Hq,
                                        int NB, int NX,
                                        bool short_groups = false) {
    const bool heavy_first = (order & kOrderHeavyFirst) != 0;
    Tile t;
    if (mapping == 0 || mapping == 3) {
        int j = wid % Hq;
        const int rest = wid / Hq;
        t.m = rest % NB;
        t.b = rest / NB;
        if (mapping == 3) {
            const int x = j % NX;
            const int qh = Hq / NX;
            const int rh = Hq % NX;
            j = x * qh + (x < rh ? x : rh) + j / NX;
        }
        t.hq = j;
        if (heavy_first) t.m = NB - 1 - t.m;
        return t;
    }
    int L = wid;
    if (mapping == 2) {
        const int N = B * Hq * NB;
        const int x = wid % NX;
        const int k = wid / NX;
        const int q = N / NX;
        const int r = N % NX;
        const int L0 = x * q + (x < r ? x : r);
        const int nx = q + (x < r ? 1 : 0);
        if ((order & kOrderXcdBlockMajor) != 0 && NB <= kBlockMajorMaxBlocks && L0 % NB == 0 &&
            nx % NB == 0) {
            const int hx = nx / NB;
            const int G = (short_groups && NB <= kShortHeadBlocks) ? kBlockMajorHeadsShort
                                                                  : kBlockMajorHeads;
            const int span = G * NB;
            const int g0 = (k / span) * G;   // first local head of k's group
            const int g = (hx - g0 < G) ? hx - g0 : G;
            const int j = k - g0 * NB;
            L = L0 + (g0 + j % g) * NB + j / g;
        } else {
            L = L0 + k;
        }
    }
    t.m = L % NB;
    const int rest = L / NB;
    t.hq = rest % Hq;
    t.b = rest / Hq;
    if (heavy_first) t.m = NB - 1 - t.m;
    return t;
}

// Backward-pass arguments (head dimension 128).  Tensors are BHSD contiguous:
// q, o, dout, dq [B][Hq][Sq][128] and k, v, dk, dv [B][Hkv][Skv][128] bf16;
// lse and delta [B][Hq][Sq] fp32 (delta is written by the first kernel).
struct BwdArgs {
    const void *q;
    const void *k;
    const void *v;
    const void *o;
    const void *dout;
    const float *lse;
    float *delta;
    void *dq;
    void *dk;
    void *dv;
    int B, Hq, Hkv, Sq, Skv;
    int NBQ;          // ceil(Sq / 128): row blocks of the dQ kernel
    int NKV;          // ceil(Skv / 128): key blocks of the dK/dV kernel
    int NX;
    int order;        // kOrder* bits
    float scale;
    float scale_log2;
};

// Enqueue the forward kernel for head dimension d (64 or 128) and base mapping
// 0..3 (one kernel instantiation per combination).
hipError_t launch_attn_fwd(const KernelArgs &args, int d, bool causal, int mapping, int grid,
                           hipStream_t stream);
// The head-dimension-128 kernel (attn_fwd_pp.hip).
hipError_t launch_attn_fwd_d128(const KernelArgs &args, bool causal, int mapping, int grid,
                                hipStream_t stream);
// Device address of the library-owned tile-queue array (kQueueInts int32) on
// the current device, looked up once per device (attn_fwd_pp.hip).
hipError_t static_queue(int **queue);
// Enqueue a one-workgroup kernel that zeroes kQueueInts int32 at `queue`.
hipError_t launch_clear_queue(int *queue, hipStream_t stream);
// The backward pass (attn_bwd.hip): D, then dK/dV, then dQ, on one stream.
hipError_t launch_attn_bwd(const BwdArgs &args, bool causal, int mapping, hipStream_t stream);
// The dQ kernel alone (attn_bwd_dq.hip); launch_attn_bwd calls it last.
hipError_t launch_attn_bwd_dq(const BwdArgs &args, bool causal, int mapping, hipStream_t stream);

}  // namespace attn
