// attn_device.h -- device-side helpers shared by the attention kernels of
// libattn_numa.so (types, buffer resources, LDS copies and swizzles).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace attn {
namespace dev {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef int i32x4 __attribute__((ext_vector_type(4)));

typedef __attribute__((address_space(3))) char lds_char;
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
typedef __attribute__((address_space(3))) bf16x8 lds_bf16x8;
typedef __attribute__((address_space(3))) u32x4 lds_u32x4;
typedef __attribute__((address_space(3))) u32x2 lds_u32x2;
typedef __attribute__((address_space(3))) f32x4 lds_f32x4;

constexpr int kThreads = 256;
// Word 3 of a gfx9 buffer resource: 32-bit data format, raw (stride 0) access.
constexpr int kBufferFlags = 0x00020000;

// Buffer resource as four scalar words (gfx9 layout): base address, stride 0,
// size in bytes (accesses at or past it read zero / are dropped), flags.
// The values must be uniform across the wave; they are read from the first
// lane so that they live in scalar registers.
__device__ __forceinline__ i32x4 buffer_words(const void *base, uint32_t bytes) {
    const uint64_t a = (uint64_t)base;
    i32x4 r;
    r[0] = __builtin_amdgcn_readfirstlane((int)(uint32_t)a);
    r[1] = __builtin_amdgcn_readfirstlane((int)(uint32_t)(a >> 32) & 0xffff);
    r[2] = __builtin_amdgcn_readfirstlane((int)bytes);
    r[3] = kBufferFlags;
    return r;
}

// 16 bytes per lane from global memory straight into LDS: lane j's bytes land
// at lds_addr + 16*j.  Issued from inline assembly so that the compiler does
// not order later LDS reads of the other buffer behind it; the kernel waits for
// these copies itself (vmcnt) before the barrier that publishes a tile.
// M0 is a register the compiler reserves; these kernels give it no other use
// (a CPU test compiles them and checks that every instruction reading M0 is one
// of these copies, each right after its own M0 write).  The compiler's hazard
// pass does not look inside the assembly, so the wait states are explicit: one
// between the M0 write and the load that reads it, and at least five between
// a vector-ALU write of a descriptor word (v_readfirstlane) and the load that
// reads it -- the s_mov and the s_nop 4 supply six.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void lds_copy16(i32x4 rsrc, uint32_t voffset, uint32_t lds_addr) {
    asm volatile("s_mov_b32 m0, %2\n\ts_nop 4\n\tbuffer_load_dwordx4 %0, %1, 0 offen lds"
                 :
                 : "v"(voffset), "s"(rsrc), "s"(lds_addr)
                 : "memory", "m0");
}
#pragma clang diagnostic pop

__device__ __forceinline__ u32x4 load16(__amdgpu_buffer_rsrc_t rsrc, uint32_t byte_off) {
    return __builtin_amdgcn_raw_buffer_load_b128(rsrc, (int)byte_off, 0, 0);
}

__device__ __forceinline__ float xor32(float x) {
    // value held by lane l ^ 32
    return __shfl_xor(x, 32, 64);
}

__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float log2_hw(float x) { return __builtin_amdgcn_logf(x); }
constexpr float kLn2 = 0.69314718055994530942f;

// Row log-sum-exp (natural log of sum_j exp(scale * s_ij)) of a finished row:
// mb = scale * log2(e) * m_ref and l = sum_j exp2(scale * log2(e) * s_ij - mb),
// so the natural-log value is (mb + log2 l) * ln 2.  Written by lane `lane` < 32
// (lanes l and l+32 own the same row) with a bounded store: rows past the end
// are dropped.
__device__ __forceinline__ void store_lse(float *lse_head, int rows, int row, int lane, float mb,
                                          float l) {
    if (lse_head == nullptr || lane >= 32) return;
    const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(
        (void *)lse_head, 0, rows * 4, kBufferFlags);
    const float v = (mb + log2_hw(l)) * kLn2;
    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), r, row * 4, 0, 0);
}

// s_waitcnt operand: vmcnt(0), expcnt and lgkmcnt not waited for.
constexpr int kWaitVmcnt0 = 0x0f70;

// LDS swizzles.  gfx950 serves 16 lanes of a 16-byte read (or of the 8-byte
// transposing read) from 64 four-byte banks, a 256-byte window; sixteen
// consecutive rows must therefore land in sixteen distinct 16-byte bank groups.
//   K rows (read as 16-byte chunks by 16 consecutive rows): chunk c of row r is
//   stored at c ^ k_swizzle(r); for 128-byte rows two rows share a window.
template <int D>
__device__ __forceinline__ int k_swizzle(int row) {
    return D == 128 ? (row & 15) : ((row >> 1) & 7);
}
//   V rows (read 4 rows x 32 bytes per 16 lanes, two such groups on adjacent
//   segments per 32 lanes): 32-byte segment s of row r is stored at
//   s ^ v_swizzle(r), which keeps all 8 (row, segment) pairs of 32 lanes apart.
template <int D>
__device__ __forceinline__ int v_swizzle(int row) {
    return D == 128 ? 2 * (row & 3) : 2 * ((row >> 1) & 1);
}

template <int V>
struct Int {
    static constexpr int value = V;
};

}  // namespace dev
}  // namespace attn
