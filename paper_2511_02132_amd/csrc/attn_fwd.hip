// attn_fwd.hip -- fused attention forward for gfx950 (MI355X) with a selectable
// workgroup -> XCD mapping.
//
// Computes O = softmax(scale * Q K^T [causal mask]) V (Section 2.3, Eq. "eq:fa")
// with the FlashAttention-2 partition of Section 2.3.1: one workgroup (WG) per
// (batch b, query head hq, block m of BLOCK_M = 128 query rows), each WG
// streaming every BLOCK_N = 64-key tile of its K/V head through LDS and
// keeping an online-softmax state (reference maximum, running sum, fp32
// accumulator) per query row; the reference is raised, and the sum and
// accumulator rescaled (the cross-tile "fix-up" of Section 2.3.1), only when
// a tile's exponentials against it would grow too large.  With GQA, query head hq reads K/V
// head hq / (Hq / Hkv).
//
// Placement (Sections 2.2, 3.2, 3.3): the hardware dispatches WG id `wid` to XCD
// `wid mod NX`; the prologue turns `wid` into the tile (b, hq, m) by one of
// four permutations, so the mapping alone decides which XCD's private L2 a
// head's K/V stream goes through:
//   0 naive block-first:   (b, m, hq) = digits of wid, heads fastest
//   1 naive head-first:    (b, hq, m) = digits of wid, blocks fastest
//   2 swizzled head-first: (b, hq, m) = digits of L, where L is the rank of wid
//     in the XCD-major listing of the grid: with x = wid mod NX,
//     k = wid div NX and (q, r) = divmod(N, NX), L = x*q + min(x, r) + k.
//     XCD x then runs one contiguous piece of the head-major order, i.e. whole
//     heads (whole K/V groups under GQA), one after another.
//   3 swizzled block-first: block-major like 0, with the heads of each row
//     block renumbered (the same XCD-major rank, within the row of Hq WGs) so
//     that one XCD gets a contiguous range of heads -- a GQA group when the
//     group count equals NX.
// (map_wid in attn_internal.h.)  This kernel serves head dimensions 64 and 56
// (computed as 64 with zero columns); head dimension 128 runs the two-group
// kernel of attn_fwd_pp.hip.
//
// Work split inside a WG (256 threads = 4 waves of 64 lanes, one per SIMD):
// wave w owns query rows 32w..32w+31 of the block.  Both contractions use
// v_mfma_f32_32x32x16_bf16 in transposed form so that every lane owns one
// query row:
//   S^T (64 keys x 32 queries) = K_tile (64 x d) * Q^T (d x 32)
//     A operand = K rows from LDS (16-byte reads), B operand = Q (registers)
//     accumulator: lane l holds query 32w + l%32 and keys 8(r/4)+4(l/32)+r%4
//   O^T (d x 32 queries) += V^T (d x 64 keys) * P^T (64 keys x 32)
//     B operand = P from the S^T accumulator, converted to bf16 in place
//     A operand = V columns, read with ds_read_b64_tr_b16 (transposing read)
// so the softmax row sums are lane-local; lanes l and l^32 add their halves
// once, at the end (and exchange maxima only when the reference is raised).
//
// LDS (double-buffered K and V tiles, 2 x 2 x 64 x d bf16) is filled directly
// by buffer loads (no register staging): the copy of tile n+1 runs while tile
// n is computed.  Rows are stored swizzled (see k_swizzle / v_swizzle) so that
// the MFMA operand reads are free of bank conflicts.  Buffer loads out of
// range read zero (ragged Sq / Skv tails); stores out of range are dropped.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "attn_device.h"
#include "attn_internal.h"
#include "attn_numa.h"

namespace attn {
namespace {

using namespace dev;

// a + b + acc for two bf16 values, in fp32 (one v_dot2 against (1, 1)).
__device__ __forceinline__ float sum_bf16_pair(__bf16 a, __bf16 b, float acc) {
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    const bf16x2_t v = {a, b};
    const bf16x2_t ones = {(__bf16)1.0f, (__bf16)1.0f};
    return __builtin_amdgcn_fdot2_f32_bf16(v, ones, acc, false);
}

// D is the head dimension the kernel computes with (64); DG <= D is the head
// dimension of the tensors in memory (64, or 56 for DeepSeek-V3-shaped heads,
// Section 4.5).  Rows of DG elements are read into D-wide LDS and register
// rows whose last D-DG elements are zero -- the copies of those 16-byte chunks
// use an out-of-range offset, which the buffer hardware turns into zeros --
// and only the first DG output columns are stored.  Zero columns change no
// score and add zero output columns, so the result is that of the DG-wide
// problem.
template <int D, int DG, bool CAUSAL, int MAPPING, int ORDER>
__global__ __launch_bounds__(kThreads, 2) void attn_fwd_kernel(const KernelArgs p) {
    static_assert(DG <= D && DG % 8 == 0, "stored rows are whole 16-byte chunks of the LDS rows");
    constexpr int BM = kBlockM;
    constexpr int BN = kBlockN;
    constexpr int ROW_BYTES_G = DG * 2;            // a row in memory
    constexpr int TILE_BYTES_G = BN * ROW_BYTES_G;
    constexpr int CHUNKS_G = DG / 8;               // 16-byte chunks stored per row
    constexpr uint32_t kOutOfRange = 0x80000000u;  // past every descriptor: reads zero
    constexpr int KSTEPS = D / 16;             // MFMA k-steps of S^T = K Q^T
    constexpr int DBLK = D / 32;               // 32-row blocks of O^T
    constexpr int CHUNKS_PER_ROW = D / 8;      // 16-byte chunks per K/V row
    constexpr int ROW_BYTES = D * 2;
    constexpr int TILE_BYTES = BN * ROW_BYTES;
    constexpr int IPW = TILE_BYTES / 1024 / (kThreads / 64);   // LDS-copy instructions per wave
    static_assert(IPW * 1024 * (kThreads / 64) == TILE_BYTES, "tile not divisible");

    __shared__ __attribute__((aligned(1024))) char smem[4 * TILE_BYTES];
    lds_char *const lds = (lds_char *)smem;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave index, kept scalar
    const int c = lane & 31;   // query column of the MFMA tiles
    const int h = lane >> 5;   // which half of the 64 lanes

    const Tile t = map_wid(MAPPING, ORDER, blockIdx.x, p.B, p.Hq, p.NB, p.NX, true);
    if (p.probe != nullptr && tid == 0) {
        unsigned xcc;
        asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(xcc));
        int32_t *rec = p.probe + 4 * (int64_t)blockIdx.x;
        rec[0] = t.b;
        rec[1] = t.hq;
        rec[2] = t.m;
        rec[3] = (int)(xcc & 0xf);
    }
    const int g = t.hq / (p.Hq / p.Hkv);

    const int64_t q_head = ((int64_t)t.b * p.Hq + t.hq) * p.Sq * DG;
    const int64_t kv_head = ((int64_t)t.b * p.Hkv + g) * p.Skv * DG;
    const __amdgpu_buffer_rsrc_t rq = __builtin_amdgcn_make_buffer_rsrc(
        (void *)((const char *)p.q + q_head * 2), 0, p.Sq * ROW_BYTES_G, kBufferFlags);
    const __amdgpu_buffer_rsrc_t ro = __builtin_amdgcn_make_buffer_rsrc(
        (void *)((char *)p.o + q_head * 2), 0, p.Sq * ROW_BYTES_G, kBufferFlags);
    // Byte offset of 16-byte chunk `ch` of row `row` in memory (zeros past DG).
    auto mem_chunk = [&](const int row, const int ch) -> uint32_t {
        return ch < CHUNKS_G ? (uint32_t)(row * ROW_BYTES_G + ch * 16) : kOutOfRange;
    };

    // Q^T as the B operand: lane holds Q[row][16kk + 8h .. +7] for each k-step.
    const int q_wave0 = t.m * BM + 32 * w;   // first query row of this wave
    const int my_q = q_wave0 + c;
    bf16x8 qreg[KSTEPS];
#pragma unroll
    for (int kk = 0; kk < KSTEPS; ++kk)
        qreg[kk] = __builtin_bit_cast(bf16x8, load16(rq, mem_chunk(my_q, 2 * kk + h)));

    // K/V tiles go straight from global memory to LDS (buffer_load ... lds):
    // each instruction of a wave fills 1024 contiguous LDS bytes, lane j the
    // 16 bytes at j*16, so the swizzled layout is made by choosing which
    // global 16-byte chunk each lane fetches.  Wave w fills LDS slots
    // (w*IPW + i)*64 + lane, i < IPW, of each tile.
    //
    // LDS holds two K buffers and two V buffers.  The K stream runs one tile
    // ahead of the V stream: while tile n's probabilities are formed and
    // multiplied into V(n), the scores of tile n+1 are already being computed
    // from K(n+1).  At the top of iteration n, K(n+1) and V(n) have landed and
    // every wave is done with K(n) and V(n-1), whose buffers then receive
    // K(n+2) and V(n+1).
    uint32_t k_src[IPW], v_src[IPW];
#pragma unroll
    for (int i = 0; i < IPW; ++i) {
        const int slot = (w * IPW + i) * 64 + lane;
        const int row = slot / CHUNKS_PER_ROW;
        const int phys = slot % CHUNKS_PER_ROW;
        k_src[i] = mem_chunk(row, phys ^ k_swizzle<D>(row));
        const int seg = (phys >> 1) ^ v_swizzle<D>(row);
        v_src[i] = mem_chunk(row, seg * 2 + (phys & 1));
    }
    const char *const k_head = (const char *)p.k + kv_head * 2;
    const char *const v_head = (const char *)p.v + kv_head * 2;
    const uint32_t kv_bytes = p.Skv * ROW_BYTES_G;
    const uint32_t lds_base = (uint32_t)(uintptr_t)lds;
    // Copy of tile n of K (or V) into LDS buffer `buf`; the descriptor starts
    // at the tile, so the per-lane offsets stay fixed.
    auto copy_tile = [&](const char *head, const uint32_t *src, const int n, const int buf) __attribute__((always_inline)) {
        const uint32_t off = (uint32_t)n * TILE_BYTES_G;
        const i32x4 d = buffer_words(head + off, kv_bytes - off);
#pragma unroll
        for (int i = 0; i < IPW; ++i)
            lds_copy16(d, src[i], lds_base + buf * TILE_BYTES + (w * IPW + i) * 1024);
    };
    // buffers: K0, K1, V0, V1
    auto copy_k = [&](const int n, const int kbuf) __attribute__((always_inline)) { copy_tile(k_head, k_src, n, kbuf); };
    auto copy_v = [&](const int n, const int vbuf) __attribute__((always_inline)) { copy_tile(v_head, v_src, n, 2 + vbuf); };

    const int kv_end = CAUSAL ? min((t.m + 1) * BM, p.Skv) : p.Skv;
    const int n_tiles = (kv_end + BN - 1) / BN;

    // Per-lane LDS read offsets (the buffer offsets are immediates).
    //   K operand: row 32kb + c, logical chunk 2kk + h.
    uint32_t k_off[KSTEPS];
#pragma unroll
    for (int kk = 0; kk < KSTEPS; ++kk)
        k_off[kk] = c * ROW_BYTES + (((2 * kk + h) ^ k_swizzle<D>(c)) * 16);
    //   V operand (transposing read, 16-lane groups): lane i = l%16 of group
    //   gsel = (l%32)/16 addresses row 4h + i/4 of a 16-key chunk (the same
    //   swizzle for all chunks and for the +8 rows) and columns
    //   32db + 16gsel + 4(i%4), i.e. 32-byte segment 2db + gsel.
    const int li = lane & 15;
    const int gsel = (lane >> 4) & 1;
    uint32_t v_off[DBLK];
#pragma unroll
    for (int db = 0; db < DBLK; ++db)
        v_off[db] = (4 * h + (li >> 2)) * ROW_BYTES + 8 * (li & 3) +
                    (((2 * db + gsel) ^ v_swizzle<D>(4 * h + (li >> 2))) * 32);

    // S^T of one tile from K buffer `kbuf`.
    auto scores = [&](const int kbuf, f32x16 (&sacc)[2]) {
        lds_char *const kb = lds + kbuf * TILE_BYTES;
#pragma unroll
        for (int kb2 = 0; kb2 < 2; ++kb2)
            for (int r = 0; r < 16; ++r) sacc[kb2][r] = 0.0f;
#pragma unroll
        for (int kk = 0; kk < KSTEPS; ++kk) {
#pragma unroll
            for (int kb2 = 0; kb2 < 2; ++kb2) {
                const bf16x8 a = *(const lds_bf16x8 *)(kb + k_off[kk] + kb2 * 32 * ROW_BYTES);
                sacc[kb2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qreg[kk], sacc[kb2], 0, 0, 0);
            }
        }
    };

    f32x16 oacc[DBLK];
#pragma unroll
    for (int db = 0; db < DBLK; ++db)
        for (int r = 0; r < 16; ++r) oacc[db][r] = 0.0f;
    // Online-softmax state of this lane's query row.  m_ref is the reference
    // maximum the exponents are taken against: set from the first tile's row
    // maximum and raised (O and l rescaled) only when a tile's exponentials
    // sum to more than 2^24 for some lane.  Any reference gives the same result
    // in exact arithmetic, because O and l are divided by the same factor.
    float m_ref = -__builtin_inff();
    float mb = -__builtin_inff();   // m_ref * scale_log2
    float l_run = 0.0f;             // partial sum over this lane's keys
    const float sl2 = p.scale_log2;

    // Prologue: K(0), V(0), K(1) in flight; scores of tile 0.
    copy_k(0, 0);
    copy_v(0, 0);
    if (n_tiles > 1) copy_k(1, 1);
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
    __syncthreads();
    f32x16 s_cur[2];
    scores(0, s_cur);

    // Iteration n (buffers fixed by the parity of n): softmax and P V of tile
    // n, scores of tile n+1.
    auto tile_step = [&](const int n, auto parity) __attribute__((always_inline)) {
        constexpr int PAR = decltype(parity)::value;   // n % 2
        __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
        __syncthreads();
        if (n + 2 < n_tiles) copy_k(n + 2, PAR);
        if (n + 1 < n_tiles) copy_v(n + 1, 1 - PAR);

        const int key0 = n * BN;
        // Mask keys past Skv and, when causal, keys after the query row.
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
        // more than 2^24 in the exp2 domain; only then is the row maximum
        // taken, O and l rescaled and the exponentials recomputed.
        // P is rounded to bf16 (the output product's B operand) as it is formed,
        // and the row sum is taken from the bf16 pairs, one v_dot2 against
        // (1, 1) per pair: half the vector instructions of fp32 adds, in a
        // kernel whose vector ALU, not its matrix core, sets the pace.  The
        // sum is then that of exactly the weights the output product uses.
        bf16x8 pb8[4];
        auto exps = [&]() __attribute__((always_inline)) {
            float ts[2] = {0.0f, 0.0f};
#pragma unroll
            for (int kc = 0; kc < 4; ++kc) {
                f32x8 p8;
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    p8[e] = exp2_hw(__builtin_fmaf(s_cur[kc >> 1][8 * (kc & 1) + e], sl2, -mb));
                pb8[kc] = __builtin_convertvector(p8, bf16x8);
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    ts[kc & 1] = sum_bf16_pair(pb8[kc][2 * e], pb8[kc][2 * e + 1], ts[kc & 1]);
            }
            return ts[0] + ts[1];
        };
        float tsum = exps();
        if (__any(!(tsum <= 16777216.0f))) {
            float mx = s_cur[0][0];
#pragma unroll
            for (int kb2 = 0; kb2 < 2; ++kb2)
#pragma unroll
                for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s_cur[kb2][r]);
            // Raise the reference to the row maximum (both lane halves agree).
            const float m_new = fmaxf(m_ref, fmaxf(mx, xor32(mx)));
            const float alpha = exp2_hw((m_ref - m_new) * sl2);   // 0 on the first tile
            l_run *= alpha;
#pragma unroll
            for (int db = 0; db < DBLK; ++db)
#pragma unroll
                for (int r = 0; r < 16; ++r) oacc[db][r] *= alpha;
            m_ref = m_new;
            mb = m_ref * sl2;
            tsum = exps();
        }
        l_run += tsum;

        // Scores of the next tile, independent of the work below so the two
        // interleave.  After the last tile this reads a stale (in-bounds)
        // buffer and the result is dropped; computing it unconditionally keeps
        // the loop body one basic block.
        f32x16 s_next[2];
        scores(1 - PAR, s_next);

        // Probabilities of tile n and O^T += V^T P^T over four 16-key chunks.
        lds_char *const vb = lds + (2 + PAR) * TILE_BYTES;
#pragma unroll
        for (int kb2 = 0; kb2 < 2; ++kb2) {
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                const bf16x8 pb = pb8[2 * kb2 + u];
                const int chunk = (16 * (2 * kb2 + u)) * ROW_BYTES;
#pragma unroll
                for (int db = 0; db < DBLK; ++db) {
                    const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
                        (lds_bf16x4 *)(vb + v_off[db] + chunk));
                    const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
                        (lds_bf16x4 *)(vb + v_off[db] + chunk + 8 * ROW_BYTES));
                    const bf16x8 a = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
                    oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb, oacc[db], 0, 0, 0);
                }
            }
        }
        s_cur[0] = s_next[0];
        s_cur[1] = s_next[1];
    };

    // Two tiles per trip so that each LDS buffer has a fixed offset.
    for (int n = 0; n < n_tiles; n += 2) {
        tile_step(n, Int<0>{});
        if (n + 1 < n_tiles) tile_step(n + 1, Int<1>{});
    }

    // O = acc / l, rounded to bf16; lane holds d = 32db + 8j + 4h + 0..3 of its row.
    const float l_tot = l_run + xor32(l_run);
    const float inv = 1.0f / l_tot;
    store_lse(p.lse == nullptr ? nullptr : p.lse + ((int64_t)t.b * p.Hq + t.hq) * p.Sq, p.Sq, my_q,
              lane, mb, l_tot);
#pragma unroll
    for (int db = 0; db < DBLK; ++db) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const f32x4 o4 = {oacc[db][4 * j + 0] * inv, oacc[db][4 * j + 1] * inv,
                              oacc[db][4 * j + 2] * inv, oacc[db][4 * j + 3] * inv};
            const bf16x4 ob = __builtin_convertvector(o4, bf16x4);
            const int col = 32 * db + 8 * j + 4 * h;   // 4 columns, all < DG or all >= DG
            if (col >= DG) continue;
            const uint32_t off = (uint32_t)(my_q * DG + col) * 2u;
            __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2, ob), ro, (int)off, 0, 0);
        }
    }
}

template <int D, int DG, bool CAUSAL, int MAPPING, int ORDER>
hipError_t launch_order(const KernelArgs &a, int grid, hipStream_t stream) {
    hipLaunchKernelGGL((attn_fwd_kernel<D, DG, CAUSAL, MAPPING, ORDER>), dim3(grid), dim3(kThreads),
                       0, stream, a);
    return hipGetLastError();
}

// The block-major order inside an XCD's piece exists for mapping 2 only.
template <int D, int DG, bool CAUSAL, int MAPPING>
hipError_t launch_one(const KernelArgs &a, int grid, hipStream_t stream) {
    switch (MAPPING == ATTN_MAP_SWIZZLED_HEAD_FIRST ? a.order : (a.order & kOrderHeavyFirst)) {
        case 0: return launch_order<D, DG, CAUSAL, MAPPING, 0>(a, grid, stream);
        case 1: return launch_order<D, DG, CAUSAL, MAPPING, 1>(a, grid, stream);
        case 2: return launch_order<D, DG, CAUSAL, MAPPING, (MAPPING == 2 ? 2 : 0)>(a, grid, stream);
        default: return launch_order<D, DG, CAUSAL, MAPPING, (MAPPING == 2 ? 3 : 1)>(a, grid, stream);
    }
}

template <int D, int DG, bool CAUSAL>
hipError_t launch_mapping(const KernelArgs &a, int mapping, int grid, hipStream_t stream) {
    switch (mapping) {
        case ATTN_MAP_NAIVE_BLOCK_FIRST: return launch_one<D, DG, CAUSAL, 0>(a, grid, stream);
        case ATTN_MAP_NAIVE_HEAD_FIRST: return launch_one<D, DG, CAUSAL, 1>(a, grid, stream);
        case ATTN_MAP_SWIZZLED_HEAD_FIRST: return launch_one<D, DG, CAUSAL, 2>(a, grid, stream);
        default: return launch_one<D, DG, CAUSAL, 3>(a, grid, stream);
    }
}

}  // namespace

hipError_t launch_attn_fwd(const KernelArgs &a, int d, bool causal, int mapping, int grid,
                           hipStream_t stream) {
    if (d == 128) return launch_attn_fwd_d128(a, causal, mapping, grid, stream);
    if (d == 56)
        return causal ? launch_mapping<64, 56, true>(a, mapping, grid, stream)
                      : launch_mapping<64, 56, false>(a, mapping, grid, stream);
    return causal ? launch_mapping<64, 64, true>(a, mapping, grid, stream)
                  : launch_mapping<64, 64, false>(a, mapping, grid, stream);
}

}  // namespace attn
