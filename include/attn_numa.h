/*
 * attn_numa.h -- C ABI of the MI355X (gfx950) attention-forward library
 * libattn_numa.so.
 *
 * The library computes the attention forward pass of Section 2.3, Eq. (1)
 * ("eq:fa") with the FlashAttention-2 work split of Section 2.3.1: one
 * workgroup (WG) per (batch, query head, block of BLOCK_M query rows), each WG
 * streaming the whole K and V of its head.  The WG -> XCD placement is chosen
 * by `mapping` (Sections 3.2 and 3.3):
 *
 *   ATTN_MAP_NAIVE_BLOCK_FIRST   -- block-major order (Section 3.2)
 *   ATTN_MAP_NAIVE_HEAD_FIRST    -- head-major order (Section 3.2)
 *   ATTN_MAP_SWIZZLED_HEAD_FIRST -- head-major order cut into one contiguous
 *                                   piece per XCD (Section 3.3, the method)
 *   ATTN_MAP_SWIZZLED_BLOCK_FIRST -- block-major order with each row block's
 *                                   heads renumbered so that one XCD gets a
 *                                   contiguous range of them, keeping a GQA
 *                                   group on one XCD (Section 3.2; the paper
 *                                   gives no formula, see map_tiles below)
 *
 * The hardware dispatches WG `wid` to XCD `wid mod NX` (Section 2.2); each
 * mapping is a permutation wid -> (b, hq, m) computed in the kernel prologue.
 * The output does not depend on the mapping (bitwise).
 *
 * No C++ types, exceptions or torch types cross this boundary.  Every entry
 * point returns an int status (ATTN_OK or a negative ATTN_ERR_* code) unless
 * stated otherwise; arguments are validated on the host before any HIP call.
 */
#ifndef ATTN_NUMA_H
#define ATTN_NUMA_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
    ATTN_MAP_NAIVE_BLOCK_FIRST = 0,
    ATTN_MAP_NAIVE_HEAD_FIRST = 1,
    ATTN_MAP_SWIZZLED_HEAD_FIRST = 2,
    ATTN_MAP_SWIZZLED_BLOCK_FIRST = 3,
    /* Optional flag OR-ed into any mapping: dispatch each head's row blocks
     * from the last to the first (m -> NB-1-m).  The XCD that runs each
     * (batch, head) is unchanged; under a causal mask, where block m costs m+1
     * K/V tiles, the expensive blocks start first and the tail shrinks.  Not
     * part of the paper's mappings (Sections 3.2, 3.3), which dispatch blocks
     * in increasing order. */
    ATTN_ORDER_HEAVY_FIRST = 0x10,
    /* Optional flag for ATTN_MAP_SWIZZLED_HEAD_FIRST only (ATTN_ERR_MAPPING
     * otherwise): each XCD receives exactly the tiles it gets without the
     * flag, but when its contiguous piece of the head-major order is made of
     * whole heads, it cuts them into groups of four consecutive heads (the
     * last group may hold fewer) and dispatches each group block-major.
     * MI355X hands an XCD its workgroups in order, one per shader engine in
     * turn (four per XCD); under a causal mask this makes four consecutive
     * workgroups equally expensive (measured: head-major order left one
     * shader engine with 9% more work), while the workgroups in flight read
     * the K/V of only four heads.  For head dimension 56 and 64 (128-row
     * blocks, four workgroups per CU) and heads of at most 16 row blocks the
     * groups hold 16 heads: short heads finish their blocks quickly and the
     * longer heavy-first prefix balances the compute units better (measured
     * +2 to +16% on 2K-token heads of 128-head prefill shapes), while their
     * K/V streams are short.  Applies only when a head has at most 64
     * row blocks (the imbalance shrinks like 1/blocks, and at long contexts
     * head-major order shares K/V better); otherwise the order is unchanged.
     * Not part of the paper's mappings. */
    ATTN_ORDER_XCD_BLOCK_MAJOR = 0x20,
    /* Optional flag for the dispatched forward with head dimension 128
     * (attn_fwd, attn_fwd_lse, attn_fwd_probe; ATTN_ERR_UNSUPPORTED for
     * another d or a persistent form, ATTN_ERR_MAPPING for attn_bwd): the grid
     * has P = ceil(NB/2) slots per head instead of NB row blocks (NB =
     * ceil(Sq/attn_block_m(d))).  The mapping and the other flags place the
     * B*Hq*P slots exactly as they place tiles, with P in place of NB, and
     * the workgroup of slot p computes row block NB-1-p and then row block p
     * (once, if they coincide).  Under a causal mask with Sq == Skv block m
     * costs m+1 block-widths of K/V, so every pair costs NB+1 (the middle
     * block of an odd NB about half): the workgroups an XCD hands to its four
     * shader engines cost the same whatever their order, and each XCD still
     * serves the contiguous slots of one (batch, head) at a time under
     * ATTN_MAP_SWIZZLED_HEAD_FIRST.  The output is bitwise that of the order
     * without the flag.  Not part of the paper's mappings. */
    ATTN_ORDER_PAIRED = 0x40
};

enum {
    ATTN_OK = 0,
    ATTN_ERR_NULL = -1,        /* a required pointer is NULL */
    ATTN_ERR_SHAPE = -2,       /* a dimension <= 0, Hq % Hkv != 0, or a size limit exceeded */
    ATTN_ERR_UNSUPPORTED = -3, /* head dimension other than 56, 64 or 128 (or a form that lacks it) */
    ATTN_ERR_MAPPING = -4,     /* mapping not one of ATTN_MAP_* with the flags allowed for it */
    ATTN_ERR_SCALE = -5,       /* scale not finite or not > 0 */
    ATTN_ERR_ALIGN = -6,       /* a bf16 tensor not 16-byte aligned, or an fp32/int32 buffer not 4-byte aligned */
    ATTN_ERR_HIP = -7,         /* a HIP runtime call failed; see attn_last_hip_error() */
    ATTN_ERR_ALIAS = -8        /* o overlaps q, k or v */
};

/*
 * attn_fwd -- attention forward, Section 2.3 Eq. (1) with GQA (Section 2.3,
 * MHA/GQA paragraph) and an optional causal mask:
 *
 *   O[b,h,i,:] = sum_j softmax_j( scale * <Q[b,h,i,:], K[b,g,j,:]> ) * V[b,g,j,:]
 *   g = h / (Hq / Hkv)      (contiguous groups of query heads share a K/V head)
 *   causal: j ranges over 0..min(i, Skv-1) (top-left aligned); else 0..Skv-1
 *
 * q : device pointer, bf16, [B][Hq][Sq][d] contiguous, 16-byte aligned
 * k : device pointer, bf16, [B][Hkv][Skv][d] contiguous, 16-byte aligned
 * v : device pointer, bf16, [B][Hkv][Skv][d] contiguous, 16-byte aligned
 * o : device pointer, bf16, [B][Hq][Sq][d] contiguous, 16-byte aligned;
 *     must not overlap q, k or v.  Every element is written.
 * d : 56, 64 or 128.  d = 56 (the DeepSeek-V3 head of Section 4.5, not a
 *     multiple of the matrix-core step) runs the d = 64 kernel on rows padded
 *     with zeros inside the kernel; the tensors stay 56 wide.  Sq*d*2 and
 *     Skv*d*2 must each be below 2^31 bytes, and the grid
 *     B*Hq*ceil(Sq/BLOCK_M) below 2^31.
 * scale : finite and > 0 (the paper uses 1/sqrt(d)); softmax is taken in fp32
 *     with bf16 inputs, fp32 accumulation and bf16 rounding (RNE) of P and O.
 * mapping : one of ATTN_MAP_NAIVE_BLOCK_FIRST, ATTN_MAP_NAIVE_HEAD_FIRST,
 *     ATTN_MAP_SWIZZLED_HEAD_FIRST, ATTN_MAP_SWIZZLED_BLOCK_FIRST, optionally
 *     | ATTN_ORDER_HEAVY_FIRST, for ATTN_MAP_SWIZZLED_HEAD_FIRST optionally
 *     | ATTN_ORDER_XCD_BLOCK_MAJOR, and for d = 128 optionally
 *     | ATTN_ORDER_PAIRED.
 *
 * Ownership: all buffers belong to the caller; nothing is retained after the
 * call returns and nothing is allocated.  The kernel is enqueued on the stream
 * set by attn_set_stream() for the calling thread (default: the null stream)
 * and the call returns without waiting; the caller synchronises.
 */
int attn_fwd(const void *q, const void *k, const void *v, void *o,
             int B, int Hq, int Hkv, int Sq, int Skv, int d,
             int causal, float scale, int mapping);

/*
 * attn_fwd_probe -- attn_fwd plus a record of the placement (Sections 2.2,
 * 3.2, 3.3): the same kernel writes, for every workgroup id wid, four int32
 * values probe[4*wid + 0..3] = (b, hq, m, xcc) where (b, hq, m) is the tile
 * that WG computed and xcc the XCD it ran on (hardware register XCC_ID).
 * With ATTN_ORDER_PAIRED only the B*Hq*ceil(NB/2) workgroups of the paired
 * grid write, and m is the first row block of the slot (NB-1-p); the records
 * past them are left as they were.
 * probe : device pointer to attn_grid_size(B, Hq, Sq, d) * 4 int32, owned by
 * the caller.  Other arguments and behaviour as attn_fwd.
 */
int attn_fwd_probe(const void *q, const void *k, const void *v, void *o,
                   int B, int Hq, int Hkv, int Sq, int Skv, int d,
                   int causal, float scale, int mapping, int32_t *probe);

/*
 * attn_fwd_lse -- attn_fwd that also writes each row's log-sum-exp, the
 * statistic the backward pass recomputes P from (Section 2.3.1):
 *   lse[b][hq][i] = log sum_{j in J_i} exp(scale * <Q[b,hq,i], K[b,g,j]>)
 * (natural log, fp32; J_i as in attn_fwd).  For d = 128 the sum is an fp32
 * sum of the fp32 exponentials.  For d = 56 and 64 it is taken over the
 * exponentials rounded to bf16 (the weights the output product uses), so lse
 * is within ln(1 + 2^-8) < 3.9e-3 of the exact value plus fp32 rounding.
 * lse : device pointer to B*Hq*Sq fp32, 4-byte aligned, owned by the caller;
 *     must not overlap q, k, v or o.  Other arguments and behaviour as
 *     attn_fwd.
 */
int attn_fwd_lse(const void *q, const void *k, const void *v, void *o, float *lse,
                 int B, int Hq, int Hkv, int Sq, int Skv, int d,
                 int causal, float scale, int mapping);

/*
 * attn_bwd -- attention backward pass, Section 2.3 Eq. (2) ("eq:ba"), for the
 * forward of attn_fwd with the same (scale, causal, GQA grouping):
 *   P_ij  = exp(scale * s_ij - lse_i),  s_ij = <Q_i, K_j>
 *   dV_j  = sum_i P_ij dO_i                        (dV = P^T dO)
 *   dP_ij = <dO_i, V_j>                             (dP = dO V^T)
 *   dS_ij = P_ij (dP_ij - D_i), D_i = <dO_i, O_i>   (dS = dsoftmax(dP))
 *   dQ_i  = scale * sum_j dS_ij K_j                 (dQ = dS K)
 *   dK_j  = scale * sum_i dS_ij Q_i                 (dK = dS^T Q)
 * summed over the query heads of a group for dK and dV (GQA), with i, j over
 * the same (causal) pairs as the forward.
 *
 * q, k, v : the forward's inputs (layouts as attn_fwd).
 * o : the forward's output, bf16 [B][Hq][Sq][d].
 * dout : dL/dO, bf16 [B][Hq][Sq][d].
 * lse : the forward's row log-sum-exp (attn_fwd_lse), fp32 [B][Hq][Sq].
 * delta : workspace, fp32 [B][Hq][Sq], 4-byte aligned; overwritten with D.
 * dq : output, bf16 [B][Hq][Sq][d].   dk, dv : outputs, bf16 [B][Hkv][Skv][d].
 *     Every element of dq, dk and dv is written.
 * d : 128 only (ATTN_ERR_UNSUPPORTED otherwise).
 * mapping : as attn_fwd, without ATTN_ORDER_PAIRED (ATTN_ERR_MAPPING).  The
 *     dQ kernel decodes its workgroups over
 *     (b, hq, row block of 128) and the dK/dV kernel over (b, K/V head, key
 *     block of 128) with that mapping; ATTN_ORDER_HEAVY_FIRST reverses the row
 *     blocks of the dQ kernel (the dK/dV kernel's natural order already starts
 *     with the most expensive causal block).  The result is bitwise the same
 *     for every mapping.
 *
 * Tensor pointers must be 16-byte aligned and the outputs and the workspace
 * must not overlap any input or each other (ATTN_ERR_ALIGN / ATTN_ERR_ALIAS).
 * Ownership, streams and asynchrony as attn_fwd.
 */
int attn_bwd(const void *q, const void *k, const void *v, const void *o, const void *dout,
             const float *lse, float *delta, void *dq, void *dk, void *dv,
             int B, int Hq, int Hkv, int Sq, int Skv, int d,
             int causal, float scale, int mapping);

/*
 * attn_fwd_persistent -- attn_fwd (optionally also writing lse, as
 * attn_fwd_lse) in a persistent, dispatch-independent form (head dimension 128
 * only): one workgroup per compute unit (or per tile, if there are fewer tiles)
 * reads the XCD it runs on (XCC_ID) and
 * takes tiles from a queue per XCD.  Queue x hands out the workgroup ids
 * wid = x + NX*t, t = 0, 1, ..., i.e. exactly the tiles the round-robin
 * dispatcher of Section 2.2 would send to XCD x under `mapping`, in the same
 * order, so the placement no longer depends on the hardware's dispatch policy
 * (which the paper notes may change).  A workgroup whose queue is empty takes
 * tiles left in the other queues, so every tile is computed.  The next ticket
 * is requested while a tile runs, hiding the gap between workgroups.
 *
 * queue : device pointer to ATTN_QUEUE_INTS int32, 4-byte aligned, owned by the
 *     caller; all zero before the call (e.g. allocated zeroed once).  The last
 *     workgroup of each launch sets it back to zero, so launches ordered on
 *     one stream may reuse it; launches that may run concurrently need
 *     separate queues.  Must not overlap the tensors.
 * lse : NULL, or as attn_fwd_lse.
 * probe : NULL, or as attn_fwd_probe (indexed by wid; xcc is the XCD that ran
 *     the tile).
 * Other arguments and behaviour as attn_fwd; ATTN_ERR_UNSUPPORTED for d != 128,
 * more than 32 XCDs, or ATTN_ORDER_PAIRED (the queues already balance the
 * work).  The output is bitwise that of attn_fwd.
 */
#define ATTN_QUEUE_INTS 64
int attn_fwd_persistent(const void *q, const void *k, const void *v, void *o, float *lse,
                        int32_t *queue, int32_t *probe, int B, int Hq, int Hkv, int Sq, int Skv,
                        int d, int causal, float scale, int mapping);

/*
 * attn_fwd_persistent_noalloc -- attn_fwd_persistent for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc): the tile queues live in a device array
 * that the library owns instead of a caller buffer.  The call makes no
 * hipMalloc, hipFree or other allocating call; the caller still provides q, k,
 * v, o (and optionally lse and probe), with the meaning, layout and checks of
 * attn_fwd_persistent.
 *
 * The array holds ATTN_QUEUE_INTS int32 (256 bytes) per GPU, for any grid;
 * each GPU the library runs on keeps its copy until the process ends.  Its
 * device address is looked up once per device, on the first call with that
 * device current.  Each call first enqueues a one-workgroup kernel that zeroes
 * the array, then the persistent kernel, both on the calling thread's stream;
 * the array keeps the last call's contents (zero after a completed launch).
 * Every call on one GPU shares that GPU's array: calls whose kernels may
 * overlap on one GPU (different streams without ordering between them) race
 * on it and may compute tiles twice or not at all; order them on one stream.
 *
 * Errors: as attn_fwd_persistent; ATTN_ERR_UNSUPPORTED for d != 128,
 * ATTN_ORDER_PAIRED or more than 32 XCDs (the array's maximum); ATTN_ERR_HIP
 * if the array's address cannot be obtained.  The output is bitwise that of attn_fwd_persistent.
 */
int attn_fwd_persistent_noalloc(const void *q, const void *k, const void *v, void *o, float *lse,
                                int32_t *probe, int B, int Hq, int Hkv, int Sq, int Skv,
                                int d, int causal, float scale, int mapping);

/* Number of workgroups attn_fwd launches: B * Hq * ceil(Sq / attn_block_m(d)),
 * or a negative ATTN_ERR_* code for an invalid shape. */
int64_t attn_grid_size(int B, int Hq, int Sq, int d);

/*
 * attn_map_tiles -- the placement the kernel uses, evaluated on the host by the
 * same integer code the kernel prologue runs (Sections 3.2 and 3.3): for
 * wid = 0 .. N-1, N = B*Hq*ceil(Sq/attn_block_m(d)), writes
 * out[3*wid + 0..2] = (b, hq, m) of workgroup wid under `mapping` with NX XCDs.
 * With ATTN_ORDER_PAIRED (d = 128 only, else ATTN_ERR_UNSUPPORTED) the rows
 * wid < B*Hq*ceil(NB/2) hold the first row block m = NB-1-p of the
 * workgroup's slot p (the second is NB-1-m when it differs from m), and the
 * rows past them hold -1.
 * out : host pointer to N*3 int32, owned by the caller.  No HIP call is made.
 */
int attn_map_tiles(int mapping, int B, int Hq, int Sq, int d, int NX, int32_t *out);

/* Query rows per workgroup (BLOCK_M, Section 4.3) for head dimension d, or
 * ATTN_ERR_UNSUPPORTED. */
int attn_block_m(int d);

/* Keys per K/V tile of the inner loop (BLOCK_N, Section 4.3) for head
 * dimension d, or ATTN_ERR_UNSUPPORTED. */
int attn_block_n(int d);

/* XCD count NX that the mappings use: the ATTN_NUM_XCD environment variable
 * when set to a positive integer, else hipDeviceAttributeNumberOfXccs of the
 * current device (cached per device).  Negative ATTN_ERR_* on failure. */
int attn_num_xcd(void);

/*
 * attn_calib_mfma -- calibration of the compute ceiling that the roofline is
 * read against; not part of the paper's method.  The published dense bf16
 * peak assumes the peak engine clock, which a sustained matrix-core load does
 * not get.  Launches `grid` workgroups of 512 threads whose 8 waves each
 * issue 4*iters independent dense bf16 MFMAs (32x32x16, 32768 flop each) on
 * register operands, with no memory or LDS traffic: 32768*4*iters*8*grid flop
 * in total.  Asynchronous on the calling thread's stream.
 * rec  : device pointer to 4*grid int64, owned by the caller; workgroup g
 *        writes rec[4g+0], rec[4g+1] = the 100 MHz real-time counter at its
 *        start and end, and rec[4g+2], rec[4g+3] = the shader-clock counter at
 *        its start and end, so that (rec[4g+3]-rec[4g+2]) /
 *        (rec[4g+1]-rec[4g+0]) * 100 MHz is the clock it ran at.
 * sink : device pointer to 512*grid float, owned by the caller; receives
 *        values that only keep the products live.
 * grid in [1, 65536] and iters a positive multiple of 4 up to 2^24
 * (ATTN_ERR_SHAPE); rec 8-byte and sink 4-byte aligned (ATTN_ERR_ALIGN); the
 * two must not overlap (ATTN_ERR_ALIAS).
 */
int attn_calib_mfma(int grid, int iters, int64_t *rec, float *sink);

/* Stream for subsequent calls from the calling thread (a hipStream_t; NULL is
 * the null stream).  The library does not take ownership. */
int attn_set_stream(void *hip_stream);

/* Stream currently set for the calling thread. */
void *attn_get_stream(void);

/* Static description of a status code (never NULL). */
const char *attn_strerror(int code);

/* Text of the last HIP error seen by the calling thread ("" if none). */
const char *attn_last_hip_error(void);

#ifdef __cplusplus
}
#endif

#endif /* ATTN_NUMA_H */
