// attn_fwd.hip -- fused attention forward for gfx950 (MI355X) with a selectable
// workgroup -> XCD mapping.
//
// Computes O = softmax(scale * Q K^T [causal mask]) V (Section 2.3, Eq. "eq:fa")
// with the FlashAttention-2 partition of Section 2.3.1: one workgroup (WG) per
// (batch b, query head hq, block m of BLOCK_M = 128 query rows), each WG
// streaming every BLOCK_N = 64-key tile of its K/V head through LDS and
// keeping an online-softmax state (running max, running sum, fp32
// accumulator) per query row, rescaled whenever the running max grows (the
// cross-tile "fix-up" of Section 2.3.1).  With GQA, query head hq reads K/V
// head hq / (Hq / Hkv).
//
// Placement (Sections 2.2, 3.2, 3.3): the hardware dispatches WG id `wid` to XCD
// `wid mod NX`; the prologue turns `wid` into the tile (b, hq, m) by one of
// three permutations, so the mapping alone decides which XCD's private L2 a
// head's K/V stream goes through:
//   0 naive block-first:   (b, m, hq) = digits of wid, heads fastest
//   1 naive head-first:    (b, hq, m) = digits of wid, blocks fastest
//   2 swizzled head-first: (b, hq, m) = digits of L, where L is the rank of wid
//     in the XCD-major listing of the grid: with x = wid mod NX,
//     k = wid div NX and (q, r) = divmod(N, NX), L = x*q + min(x, r) + k.
//     XCD x then runs one contiguous piece of the head-major order, i.e. whole
//     heads (whole K/V groups under GQA), one after another.
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
// so the softmax row reductions are lane-local except one exchange between
// lanes l and l^32 per tile.
//
// LDS (double-buffered K and V tiles, 2 x 2 x 64 x d bf16): rows of K are
// stored with 16-byte chunk c at position c ^ (row & 7), rows of V with
// 32-byte segment s at position s ^ (row & 3); both make the MFMA operand reads
// free of bank conflicts.  Global loads are 16-byte buffer loads whose
// out-of-range lanes read zero (ragged Sq / Skv tails); stores out of range
// are dropped.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "attn_numa.h"
#include "attn_internal.h"

namespace attn {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

typedef __attribute__((address_space(3))) char lds_char;
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
typedef __attribute__((address_space(3))) bf16x8 lds_bf16x8;
typedef __attribute__((address_space(3))) u32x4 lds_u32x4;

constexpr int kThreads = 256;
// Word 3 of a gfx9 buffer resource: 32-bit data format, raw (stride 0) access.
constexpr int kBufferFlags = 0x00020000;

__device__ __forceinline__ u32x4 load16(__amdgpu_buffer_rsrc_t rsrc, uint32_t byte_off) {
    return __builtin_amdgcn_raw_buffer_load_b128(rsrc, (int)byte_off, 0, 0);
}

__device__ __forceinline__ float xor32(float x) {
    // value held by lane l ^ 32
    return __shfl_xor(x, 32, 64);
}

__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }

template <int D, bool CAUSAL>
__global__ __launch_bounds__(kThreads, 2) void attn_fwd_kernel(const KernelArgs p) {
    constexpr int BM = kBlockM;
    constexpr int BN = kBlockN;
    constexpr int KSTEPS = D / 16;             // MFMA k-steps of S^T = K Q^T
    constexpr int DBLK = D / 32;               // 32-row blocks of O^T
    constexpr int CHUNKS_PER_ROW = D / 8;      // 16-byte chunks per K/V row
    constexpr int CPT = BN * CHUNKS_PER_ROW / kThreads;  // chunks per thread per tile
    constexpr int ROW_BYTES = D * 2;
    constexpr int TILE_BYTES = BN * ROW_BYTES;
    static_assert(CPT * kThreads == BN * CHUNKS_PER_ROW, "tile not divisible");

    __shared__ __attribute__((aligned(1024))) char smem[4 * TILE_BYTES];
    lds_char *const lds = (lds_char *)smem;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int w = tid >> 6;
    const int c = lane & 31;   // query column of the MFMA tiles
    const int h = lane >> 5;   // which half of the 64 lanes

    const Tile t = map_wid(p.mapping, blockIdx.x, p.B, p.Hq, p.NB, p.NX);
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

    const int64_t q_head = ((int64_t)t.b * p.Hq + t.hq) * p.Sq * D;
    const int64_t kv_head = ((int64_t)t.b * p.Hkv + g) * p.Skv * D;
    const __amdgpu_buffer_rsrc_t rq = __builtin_amdgcn_make_buffer_rsrc(
        (void *)((const char *)p.q + q_head * 2), 0, p.Sq * ROW_BYTES, kBufferFlags);
    const __amdgpu_buffer_rsrc_t rk = __builtin_amdgcn_make_buffer_rsrc(
        (void *)((const char *)p.k + kv_head * 2), 0, p.Skv * ROW_BYTES, kBufferFlags);
    const __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc(
        (void *)((const char *)p.v + kv_head * 2), 0, p.Skv * ROW_BYTES, kBufferFlags);
    const __amdgpu_buffer_rsrc_t ro = __builtin_amdgcn_make_buffer_rsrc(
        (void *)((char *)p.o + q_head * 2), 0, p.Sq * ROW_BYTES, kBufferFlags);

    // Q^T as the B operand: lane holds Q[row][16kk + 8h .. +7] for each k-step.
    const int q_wave0 = t.m * BM + 32 * w;   // first query row of this wave
    const int my_q = q_wave0 + c;
    bf16x8 qreg[KSTEPS];
#pragma unroll
    for (int kk = 0; kk < KSTEPS; ++kk)
        qreg[kk] = __builtin_bit_cast(
            bf16x8, load16(rq, (uint32_t)(my_q * D + 16 * kk + 8 * h) * 2u));

    // Per-thread share of a K/V tile copy: global offsets and swizzled LDS slots.
    uint32_t g_off[CPT], k_slot[CPT], v_slot[CPT];
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
        const int ci = tid + kThreads * i;
        const int row = ci / CHUNKS_PER_ROW;
        const int cc = ci % CHUNKS_PER_ROW;
        g_off[i] = (uint32_t)(row * D + cc * 8) * 2u;
        k_slot[i] = row * ROW_BYTES + ((cc ^ (row & 7)) * 16);
        v_slot[i] = row * ROW_BYTES + ((((cc >> 1) ^ (row & 3)) * 2 + (cc & 1)) * 16);
    }

    const int kv_end = CAUSAL ? min((t.m + 1) * BM, p.Skv) : p.Skv;
    const int n_tiles = (kv_end + BN - 1) / BN;

    u32x4 kpre[CPT], vpre[CPT];
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
        kpre[i] = load16(rk, g_off[i]);
        vpre[i] = load16(rv, g_off[i]);
    }

    // Per-lane LDS read offsets.
    //   K operand: row 32kb + c, logical chunk 2kk + h -> slot (2kk + h) ^ (c & 7).
    const uint32_t k_row_off = c * ROW_BYTES;
    const int k_x = h ^ (c & 7);
    //   V operand (transposing read, 16-lane groups): lane i = l%16 of group
    //   gsel = (l%32)/16 addresses row base + 4h + i/4, columns 32db + 16gsel + 4(i%4).
    const int li = lane & 15;
    const int gsel = (lane >> 4) & 1;
    const uint32_t v_lane_off = (4 * h + (li >> 2)) * ROW_BYTES + 8 * (li & 3);
    const int v_x = gsel ^ (li >> 2);

    f32x16 oacc[DBLK];
#pragma unroll
    for (int db = 0; db < DBLK; ++db)
        for (int r = 0; r < 16; ++r) oacc[db][r] = 0.0f;
    float m_run = -__builtin_inff();
    float l_run = 0.0f;   // partial sum over this lane's keys
    const float sl2 = p.scale_log2;

    for (int n = 0; n < n_tiles; ++n) {
        lds_char *const kb = lds + (n & 1) * 2 * TILE_BYTES;
        lds_char *const vb = kb + TILE_BYTES;
#pragma unroll
        for (int i = 0; i < CPT; ++i) {
            *(lds_u32x4 *)(kb + k_slot[i]) = kpre[i];
            *(lds_u32x4 *)(vb + v_slot[i]) = vpre[i];
        }
        __syncthreads();
        if (n + 1 < n_tiles) {
            const uint32_t next = (uint32_t)(n + 1) * TILE_BYTES;
#pragma unroll
            for (int i = 0; i < CPT; ++i) {
                kpre[i] = load16(rk, next + g_off[i]);
                vpre[i] = load16(rv, next + g_off[i]);
            }
        }
        const int key0 = n * BN;
        if (CAUSAL && key0 > q_wave0 + 31) continue;   // every key after every row of this wave

        // S^T = K Q^T
        f32x16 sacc[2];
#pragma unroll
        for (int kb2 = 0; kb2 < 2; ++kb2)
            for (int r = 0; r < 16; ++r) sacc[kb2][r] = 0.0f;
#pragma unroll
        for (int kk = 0; kk < KSTEPS; ++kk) {
#pragma unroll
            for (int kb2 = 0; kb2 < 2; ++kb2) {
                const bf16x8 a = *(const lds_bf16x8 *)(kb + k_row_off + kb2 * 32 * ROW_BYTES +
                                                       (((2 * kk) ^ k_x) * 16));
                sacc[kb2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qreg[kk], sacc[kb2], 0, 0, 0);
            }
        }

        // Mask keys past Skv and, when causal, keys after the query row.
        const bool need_mask = (key0 + BN > p.Skv) || (CAUSAL && key0 + BN - 1 > q_wave0);
        if (need_mask) {
#pragma unroll
            for (int kb2 = 0; kb2 < 2; ++kb2)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int key = key0 + 32 * kb2 + 8 * (r >> 2) + 4 * h + (r & 3);
                    const bool dead = key >= p.Skv || (CAUSAL && key > my_q);
                    sacc[kb2][r] = dead ? -__builtin_inff() : sacc[kb2][r];
                }
        }

        // Online softmax: new running max, rescale factor, probabilities.
        float mx = sacc[0][0];
#pragma unroll
        for (int kb2 = 0; kb2 < 2; ++kb2)
#pragma unroll
            for (int r = 0; r < 16; ++r) mx = fmaxf(mx, sacc[kb2][r]);
        mx = fmaxf(mx, xor32(mx));
        const float m_new = fmaxf(m_run, mx);
        const float alpha = exp2_hw((m_run - m_new) * sl2);
        const float mb = m_new * sl2;
        float lsum = 0.0f;
#pragma unroll
        for (int kb2 = 0; kb2 < 2; ++kb2)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const float pr = exp2_hw(__builtin_fmaf(sacc[kb2][r], sl2, -mb));
                sacc[kb2][r] = pr;
                lsum += pr;
            }
        l_run = l_run * alpha + lsum;
        m_run = m_new;
#pragma unroll
        for (int db = 0; db < DBLK; ++db)
#pragma unroll
            for (int r = 0; r < 16; ++r) oacc[db][r] *= alpha;

        // O^T += V^T P^T over four 16-key chunks.
#pragma unroll
        for (int kb2 = 0; kb2 < 2; ++kb2) {
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                f32x8 p8;
#pragma unroll
                for (int e = 0; e < 8; ++e) p8[e] = sacc[kb2][8 * u + e];
                const bf16x8 pb = __builtin_convertvector(p8, bf16x8);
                const uint32_t chunk_off = (uint32_t)(16 * (2 * kb2 + u)) * ROW_BYTES + v_lane_off;
#pragma unroll
                for (int db = 0; db < DBLK; ++db) {
                    const uint32_t off = chunk_off + (((2 * db) ^ v_x) * 32);
                    const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
                        (lds_bf16x4 *)(vb + off));
                    const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
                        (lds_bf16x4 *)(vb + off + 8 * ROW_BYTES));
                    const bf16x8 a = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
                    oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb, oacc[db], 0, 0, 0);
                }
            }
        }
    }

    // O = acc / l, rounded to bf16; lane holds d = 32db + 8j + 4h + 0..3 of its row.
    const float l_tot = l_run + xor32(l_run);
    const float inv = 1.0f / l_tot;
#pragma unroll
    for (int db = 0; db < DBLK; ++db) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const f32x4 o4 = {oacc[db][4 * j + 0] * inv, oacc[db][4 * j + 1] * inv,
                              oacc[db][4 * j + 2] * inv, oacc[db][4 * j + 3] * inv};
            const bf16x4 ob = __builtin_convertvector(o4, bf16x4);
            const uint32_t off = (uint32_t)(my_q * D + 32 * db + 8 * j + 4 * h) * 2u;
            __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2, ob), ro, (int)off, 0, 0);
        }
    }
}

template <int D, bool CAUSAL>
hipError_t launch_one(const KernelArgs &a, int grid, hipStream_t stream) {
    hipLaunchKernelGGL((attn_fwd_kernel<D, CAUSAL>), dim3(grid), dim3(kThreads), 0, stream, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_attn_fwd(const KernelArgs &a, int d, bool causal, int grid, hipStream_t stream) {
    if (d == 64) return causal ? launch_one<64, true>(a, grid, stream) : launch_one<64, false>(a, grid, stream);
    return causal ? launch_one<128, true>(a, grid, stream) : launch_one<128, false>(a, grid, stream);
}

}  // namespace attn
