// Host-only harness for the C ABI source (paper_2511_02132_amd/csrc/attn_abi.cpp):
// argument validation, alias checks, the launch arguments each entry point
// derives, and attn_map_tiles, built for the CPU with AddressSanitizer and
// UBSan (tests/test_abi_host_sanitize_cpu.py).  The kernel launchers and the
// three HIP runtime calls the ABI makes are stubs that record their
// arguments: no GPU, no HIP runtime and no device code are involved.
//
// Usage: abi_host_harness OUT.bin
//   Runs every check (exit status 1 and a message on the first failure) and
//   writes, for each mapping-table case, the int32 table attn_map_tiles
//   produced, so the test can compare it with the oracle enumeration.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <vector>

#include "attn_calib.h"
#include "attn_internal.h"
#include "attn_numa.h"

namespace {

bool g_fail_device = false;   // the stub hipGetDevice fails while set
int g_fwd_launches = 0, g_bwd_launches = 0, g_calib_launches = 0, g_clears = 0;
attn::KernelArgs g_fwd{};
int g_fwd_d = 0, g_fwd_mapping = -1, g_fwd_grid = 0;
bool g_fwd_causal = false;
attn::BwdArgs g_bwd{};
int g_bwd_mapping = -1;
bool g_bwd_causal = false;
int g_calib_grid = 0, g_calib_iters = 0;
int *g_cleared = nullptr;
alignas(256) int g_static_queue[attn::kQueueInts];

int g_checks = 0;

void check(bool ok, const char *what, int line) {
    ++g_checks;
    if (!ok) {
        std::fprintf(stderr, "FAILED line %d: %s\n", line, what);
        std::exit(1);
    }
}
#define CHECK(cond) check((cond), #cond, __LINE__)

}  // namespace

// ---- stubs of the HIP runtime calls attn_abi.cpp makes
extern "C" hipError_t hipGetDevice(int *device) {
    if (g_fail_device) return hipErrorNoDevice;
    *device = 0;
    return hipSuccess;
}

extern "C" hipError_t hipDeviceGetAttribute(int *value, hipDeviceAttribute_t attr, int device) {
    if (device != 0) return hipErrorInvalidDevice;
    if (attr == hipDeviceAttributeNumberOfXccs) *value = 8;
    else if (attr == hipDeviceAttributeMultiprocessorCount) *value = 256;
    else return hipErrorInvalidValue;
    return hipSuccess;
}

extern "C" const char *hipGetErrorString(hipError_t e) {
    return e == hipSuccess ? "hipSuccess" : "stubbed HIP error";
}

// ---- stubs of the kernel launchers
namespace attn {

hipError_t launch_attn_fwd(const KernelArgs &args, int d, bool causal, int mapping, int grid,
                           hipStream_t) {
    ++g_fwd_launches;
    g_fwd = args;
    g_fwd_d = d;
    g_fwd_causal = causal;
    g_fwd_mapping = mapping;
    g_fwd_grid = grid;
    return hipSuccess;
}

hipError_t launch_attn_bwd(const BwdArgs &args, bool causal, int mapping, hipStream_t) {
    ++g_bwd_launches;
    g_bwd = args;
    g_bwd_causal = causal;
    g_bwd_mapping = mapping;
    return hipSuccess;
}

hipError_t launch_calib_mfma(int grid, int iters, int64_t *, float *, hipStream_t) {
    ++g_calib_launches;
    g_calib_grid = grid;
    g_calib_iters = iters;
    return hipSuccess;
}

hipError_t static_queue(int **queue) {
    *queue = g_static_queue;
    return hipSuccess;
}

hipError_t launch_clear_queue(int *queue, hipStream_t) {
    ++g_clears;
    g_cleared = queue;
    return hipSuccess;
}

}  // namespace attn

namespace {

// Fake device addresses: 256-byte aligned, far apart, never dereferenced.
const uintptr_t kQ = 0x100000000ull, kK = 0x200000000ull, kV = 0x300000000ull,
                kO = 0x400000000ull, kL = 0x500000000ull, kP = 0x600000000ull,
                kW = 0x700000000ull, kX = 0x800000000ull, kY = 0x900000000ull,
                kZ = 0xa00000000ull, kD = 0xb00000000ull, kG = 0xc00000000ull;
void *P(uintptr_t a) { return (void *)a; }

int fwd(uintptr_t q, uintptr_t k, uintptr_t v, uintptr_t o, int B, int Hq, int Hkv, int Sq,
        int Skv, int d, int causal, float scale, int mapping) {
    return attn_fwd(P(q), P(k), P(v), P(o), B, Hq, Hkv, Sq, Skv, d, causal, scale, mapping);
}

void check_validation() {
    // {q, k, v, o, B, Hq, Hkv, Sq, Skv, d, mapping, expected}; scale 0.088, causal 0
    struct Case {
        uintptr_t q, k, v, o;
        int B, Hq, Hkv, Sq, Skv, d, mapping, want;
    };
    const Case cases[] = {
        {0, kK, kV, kO, 1, 4, 2, 256, 256, 128, 2, ATTN_ERR_NULL},
        {kQ, 0, kV, kO, 1, 4, 2, 256, 256, 128, 2, ATTN_ERR_NULL},
        {kQ, kK, 0, kO, 1, 4, 2, 256, 256, 128, 2, ATTN_ERR_NULL},
        {kQ, kK, kV, 0, 1, 4, 2, 256, 256, 128, 2, ATTN_ERR_NULL},
        {kQ, kK, kV, kO, 0, 4, 2, 256, 256, 128, 2, ATTN_ERR_SHAPE},
        {kQ, kK, kV, kO, 1, -4, 2, 256, 256, 128, 2, ATTN_ERR_SHAPE},
        {kQ, kK, kV, kO, 1, 4, 0, 256, 256, 128, 2, ATTN_ERR_SHAPE},
        {kQ, kK, kV, kO, 1, 6, 4, 256, 256, 128, 2, ATTN_ERR_SHAPE},
        {kQ, kK, kV, kO, 1, 4, 2, 0, 256, 128, 2, ATTN_ERR_SHAPE},
        {kQ, kK, kV, kO, 1, 4, 2, 256, -1, 128, 2, ATTN_ERR_SHAPE},
        {kQ, kK, kV, kO, 1, 4, 2, 1 << 23, 256, 128, 2, ATTN_ERR_SHAPE},
        {kQ, kK, kV, kO, 1, 4, 2, 256, 1 << 23, 128, 2, ATTN_ERR_SHAPE},
        {kQ, kK, kV, kO, 1, 4, 2, INT32_MAX, INT32_MAX, 128, 2, ATTN_ERR_SHAPE},
        {kQ, kK, kV, kO, 65536, 65536, 1, 65536, 64, 64, 2, ATTN_ERR_SHAPE},
        {kQ, kK, kV, kO, 1, 4, 2, 256, 256, 96, 2, ATTN_ERR_UNSUPPORTED},
        {kQ, kK, kV, kO, 1, 4, 2, 256, 256, 0, 2, ATTN_ERR_SHAPE},
        {kQ, kK, kV, kO, 1, 4, 2, 256, 256, 128, 4, ATTN_ERR_MAPPING},
        {kQ, kK, kV, kO, 1, 4, 2, 256, 256, 128, -1, ATTN_ERR_MAPPING},
        {kQ, kK, kV, kO, 1, 4, 2, 256, 256, 128, 0x82, ATTN_ERR_MAPPING},
        {kQ, kK, kV, kO, 1, 4, 2, 256, 256, 128, 0x100, ATTN_ERR_MAPPING},
        {kQ, kK, kV, kO, 1, 4, 2, 256, 256, 128, 0x61, ATTN_ERR_MAPPING},
        // paired row blocks: head dimension 128 only
        {kQ, kK, kV, kO, 1, 4, 2, 256, 256, 64, 0x42, ATTN_ERR_UNSUPPORTED},
        {kQ, kK, kV, kO, 1, 4, 2, 256, 256, 56, 0x52, ATTN_ERR_UNSUPPORTED},
        {kQ, kK, kV, kO, 1, 4, 2, 256, 256, 128, 0x20, ATTN_ERR_MAPPING},
        {kQ, kK, kV, kO, 1, 4, 2, 256, 256, 128, 0x33, ATTN_ERR_MAPPING},
        {kQ + 8, kK, kV, kO, 1, 4, 2, 256, 256, 128, 2, ATTN_ERR_ALIGN},
        {kQ, kK, kV, kO + 2, 1, 4, 2, 256, 256, 128, 2, ATTN_ERR_ALIGN},
        {kQ, kK, kV, kQ, 1, 4, 2, 256, 256, 128, 2, ATTN_ERR_ALIAS},
        {kQ, kK, kV, kK + 256, 1, 4, 2, 256, 256, 128, 2, ATTN_ERR_ALIAS},
        // o ends exactly where v starts: no overlap
        {kQ, kK, kV, kV - 4 * 256 * 128 * 2, 1, 4, 2, 256, 256, 128, 2, ATTN_OK},
        // o starts one element before the end of v: overlap
        {kQ, kK, kV, kV + 2 * 256 * 128 * 2 - 16, 1, 4, 2, 256, 256, 128, 2, ATTN_ERR_ALIAS},
    };
    for (const Case &c : cases) {
        const int got = fwd(c.q, c.k, c.v, c.o, c.B, c.Hq, c.Hkv, c.Sq, c.Skv, c.d, 0, 0.088f,
                            c.mapping);
        if (got != c.want)
            std::fprintf(stderr, "case B%d Hq%d Hkv%d Sq%d Skv%d d%d map %#x: %d, want %d\n", c.B,
                         c.Hq, c.Hkv, c.Sq, c.Skv, c.d, c.mapping, got, c.want);
        CHECK(got == c.want);
        CHECK(std::strlen(attn_strerror(got)) > 0);
    }
    const float bad_scales[] = {NAN, INFINITY, -INFINITY, 0.0f, -1.0f};
    for (float s : bad_scales) CHECK(fwd(kQ, kK, kV, kO, 1, 4, 2, 256, 256, 128, 0, s, 2) == ATTN_ERR_SCALE);
    for (int code = -8; code <= 0; ++code) CHECK(std::strcmp(attn_strerror(code), "unknown status code") != 0);
    CHECK(std::strcmp(attn_strerror(-9), "unknown status code") == 0);
    CHECK(std::strcmp(attn_strerror(1), "unknown status code") == 0);
}

// The launch arguments attn_fwd derives, on ragged shapes and every head dimension.
void check_forward_launch() {
    struct Shape {
        int B, Hq, Hkv, Sq, Skv, d, causal, mapping;
    };
    const Shape shapes[] = {
        {1, 4, 4, 256, 256, 64, 0, 2},     {2, 8, 2, 384, 384, 128, 1, 0x12},
        {1, 8, 1, 200, 200, 128, 0, 3},    {1, 2, 2, 333, 517, 128, 0, 0x11},
        {1, 2, 2, 517, 333, 56, 1, 0x32},  {2, 6, 3, 129, 65, 64, 0, 0x13},
        {1, 1, 1, 1, 1, 128, 0, 1},        {3, 5, 5, 1000, 64, 56, 1, 0x22},
        {1, 16, 16, 131072, 131072, 128, 1, 0x12},
        // paired row blocks: ceil(NB/2) slots per head
        {1, 16, 16, 131072, 131072, 128, 1, 0x52}, {2, 8, 2, 384, 384, 128, 1, 0x40},
        {1, 3, 1, 1300, 1300, 128, 1, 0x53},       {1, 2, 2, 1, 1, 128, 0, 0x41},
        {2, 4, 4, 700, 900, 128, 0, 0x62},
    };
    for (const Shape &s : shapes) {
        const int before = g_fwd_launches;
        const float scale = 1.0f / std::sqrt((float)s.d);
        CHECK(fwd(kQ, kK, kV, kO, s.B, s.Hq, s.Hkv, s.Sq, s.Skv, s.d, s.causal, scale, s.mapping) ==
              ATTN_OK);
        CHECK(g_fwd_launches == before + 1);
        const int bm = s.d == 128 ? 256 : 128;
        const int nb = (s.Sq + bm - 1) / bm;
        CHECK(attn_block_m(s.d) == bm);
        CHECK(g_fwd.NB == nb);
        const bool paired = (s.mapping & 0x40) != 0;
        CHECK(g_fwd_grid == s.B * s.Hq * (paired ? (nb + 1) / 2 : nb));
        CHECK(attn_grid_size(s.B, s.Hq, s.Sq, s.d) == (int64_t)s.B * s.Hq * nb);
        CHECK(g_fwd.B == s.B && g_fwd.Hq == s.Hq && g_fwd.Hkv == s.Hkv);
        CHECK(g_fwd.Sq == s.Sq && g_fwd.Skv == s.Skv);
        CHECK(g_fwd_d == s.d && g_fwd_causal == (s.causal != 0));
        CHECK(g_fwd_mapping == (s.mapping & 0xf));
        CHECK(g_fwd.order == (((s.mapping & 0x10) ? attn::kOrderHeavyFirst : 0) |
                              ((s.mapping & 0x20) ? attn::kOrderXcdBlockMajor : 0) |
                              (paired ? attn::kOrderPaired : 0)));
        CHECK(g_fwd.NX == 8);
        CHECK(std::fabs(g_fwd.scale_log2 - scale * 1.44269504f) <= 1e-6f * scale);
        CHECK(g_fwd.q == P(kQ) && g_fwd.k == P(kK) && g_fwd.v == P(kV) && g_fwd.o == P(kO));
        CHECK(g_fwd.probe == nullptr && g_fwd.lse == nullptr && g_fwd.queue == nullptr);
    }
}

void check_lse_probe() {
    float *lse = (float *)P(kL);
    CHECK(attn_fwd_lse(P(kQ), P(kK), P(kV), P(kO), nullptr, 1, 4, 2, 300, 300, 128, 1, 0.088f, 2) ==
          ATTN_ERR_NULL);
    CHECK(attn_fwd_lse(P(kQ), P(kK), P(kV), P(kO), (float *)P(kL + 2), 1, 4, 2, 300, 300, 128, 1,
                       0.088f, 2) == ATTN_ERR_ALIGN);
    CHECK(attn_fwd_lse(P(kQ), P(kK), P(kV), P(kO), (float *)P(kO + 64), 1, 4, 2, 300, 300, 128, 1,
                       0.088f, 2) == ATTN_ERR_ALIAS);
    CHECK(attn_fwd_lse(P(kQ), P(kK), P(kV), P(kO), (float *)P(kK), 1, 4, 2, 300, 300, 128, 1,
                       0.088f, 2) == ATTN_ERR_ALIAS);
    CHECK(attn_fwd_lse(P(kQ), P(kK), P(kV), P(kO), lse, 1, 4, 2, 300, 300, 128, 1, 0.088f, 2) ==
          ATTN_OK);
    CHECK(g_fwd.lse == lse && g_fwd.probe == nullptr);
    int32_t *probe = (int32_t *)P(kP);
    CHECK(attn_fwd_probe(P(kQ), P(kK), P(kV), P(kO), 1, 4, 2, 300, 300, 64, 0, 0.1f, 3, nullptr) ==
          ATTN_ERR_NULL);
    CHECK(attn_fwd_probe(P(kQ), P(kK), P(kV), P(kO), 1, 4, 2, 300, 300, 64, 0, 0.1f, 3,
                         (int32_t *)P(kP + 1)) == ATTN_ERR_ALIGN);
    CHECK(attn_fwd_probe(P(kQ), P(kK), P(kV), P(kO), 1, 4, 3, 300, 300, 64, 0, 0.1f, 3, probe) ==
          ATTN_ERR_SHAPE);
    CHECK(attn_fwd_probe(P(kQ), P(kK), P(kV), P(kO), 1, 4, 2, 300, 300, 64, 0, 0.1f, 3, probe) ==
          ATTN_OK);
    CHECK(g_fwd.probe == probe && g_fwd.lse == nullptr && g_fwd_grid == 4 * 3);
    // paired: the probe covers the ceil(NB/2) slots of each head
    CHECK(attn_fwd_probe(P(kQ), P(kK), P(kV), P(kO), 1, 4, 2, 1300, 1300, 128, 1, 0.1f, 0x52,
                         probe) == ATTN_OK);
    CHECK(g_fwd.probe == probe && g_fwd_grid == 4 * 3 && g_fwd.NB == 6);
    CHECK(attn_fwd_lse(P(kQ), P(kK), P(kV), P(kO), lse, 1, 4, 2, 300, 300, 64, 1, 0.1f, 0x42) ==
          ATTN_ERR_UNSUPPORTED);
}

void check_persistent() {
    int32_t *queue = (int32_t *)P(kW);
    float *lse = (float *)P(kL);
    auto pers = [&](int32_t *qu, int32_t *probe, int B, int Hq, int Hkv, int S, int d) {
        return attn_fwd_persistent(P(kQ), P(kK), P(kV), P(kO), lse, qu, probe, B, Hq, Hkv, S, S, d,
                                   1, 0.088f, 0x12);
    };
    CHECK(pers(nullptr, nullptr, 1, 4, 4, 512, 128) == ATTN_ERR_NULL);
    CHECK(pers((int32_t *)P(kW + 2), nullptr, 1, 4, 4, 512, 128) == ATTN_ERR_ALIGN);
    CHECK(pers(queue, (int32_t *)P(kP + 2), 1, 4, 4, 512, 128) == ATTN_ERR_ALIGN);
    CHECK(pers(queue, nullptr, 1, 4, 4, 512, 64) == ATTN_ERR_UNSUPPORTED);
    // paired row blocks are for the dispatched grid only
    CHECK(attn_fwd_persistent(P(kQ), P(kK), P(kV), P(kO), lse, queue, nullptr, 1, 4, 4, 512, 512,
                              128, 1, 0.088f, 0x52) == ATTN_ERR_UNSUPPORTED);
    CHECK(pers((int32_t *)P(kO + 1024), nullptr, 1, 4, 4, 512, 128) == ATTN_ERR_ALIAS);
    CHECK(pers((int32_t *)P(kL), nullptr, 1, 4, 4, 512, 128) == ATTN_ERR_ALIAS);
    // the queue ends exactly where q starts: no overlap
    CHECK(pers((int32_t *)P(kQ - ATTN_QUEUE_INTS * 4), nullptr, 1, 4, 4, 512, 128) == ATTN_OK);
    // fewer tiles than compute units: one workgroup per tile
    CHECK(pers(queue, nullptr, 1, 3, 1, 257, 128) == ATTN_OK);
    CHECK(g_fwd_grid == 3 * 2 && g_fwd.queue == queue && g_fwd.lse == lse);
    // more tiles than compute units: one workgroup per compute unit
    CHECK(pers(queue, nullptr, 1, 32, 32, 8192, 128) == ATTN_OK);
    CHECK(g_fwd_grid == 256 && g_fwd.NB == 32);
    // the queue holds at most 32 XCD counters
    setenv("ATTN_NUM_XCD", "33", 1);
    CHECK(pers(queue, nullptr, 1, 4, 4, 512, 128) == ATTN_ERR_UNSUPPORTED);
    unsetenv("ATTN_NUM_XCD");

    // the entry point that allocates nothing: the library's queue, cleared first
    auto noalloc = [&](int32_t *probe, int B, int Hq, int Hkv, int S, int d, uintptr_t o) {
        return attn_fwd_persistent_noalloc(P(kQ), P(kK), P(kV), P(o), lse, probe, B, Hq, Hkv, S, S,
                                           d, 1, 0.088f, 0x12);
    };
    const int clears = g_clears, launches = g_fwd_launches;
    CHECK(noalloc(nullptr, 1, 4, 4, 512, 64, kO) == ATTN_ERR_UNSUPPORTED);
    CHECK(noalloc((int32_t *)P(kP + 2), 1, 4, 4, 512, 128, kO) == ATTN_ERR_ALIGN);
    CHECK(noalloc(nullptr, 1, 4, 4, 512, 128, kQ) == ATTN_ERR_ALIAS);
    CHECK(noalloc(nullptr, 1, 4, 3, 512, 128, kO) == ATTN_ERR_SHAPE);
    CHECK(attn_fwd_persistent_noalloc(P(kQ), P(kK), P(kV), P(kO), lse, nullptr, 1, 4, 4, 512, 512,
                                      128, 1, 0.088f, 0x42) == ATTN_ERR_UNSUPPORTED);
    setenv("ATTN_NUM_XCD", "33", 1);
    CHECK(noalloc(nullptr, 1, 4, 4, 512, 128, kO) == ATTN_ERR_UNSUPPORTED);
    unsetenv("ATTN_NUM_XCD");
    CHECK(g_clears == clears && g_fwd_launches == launches);   // rejected before any launch
    CHECK(noalloc((int32_t *)P(kP), 2, 16, 4, 700, 128, kO) == ATTN_OK);
    CHECK(g_clears == clears + 1 && g_fwd_launches == launches + 1);
    CHECK(g_cleared == g_static_queue && g_fwd.queue == g_static_queue);
    CHECK(g_fwd_grid == 2 * 16 * 3 && g_fwd.probe == (int32_t *)P(kP) && g_fwd.lse == lse);
}

void check_backward() {
    const uintptr_t ins[6] = {kQ, kK, kV, kO, kD, kL};      // q k v o dout lse
    const uintptr_t outs[4] = {kX, kY, kZ, kG};             // dq dk dv delta
    auto bwd = [&](const uintptr_t *in, const uintptr_t *out, int d, int B, int Hq, int Hkv,
                   int Sq, int Skv) {
        return attn_bwd(P(in[0]), P(in[1]), P(in[2]), P(in[3]), P(in[4]), (const float *)P(in[5]),
                        (float *)P(out[3]), P(out[0]), P(out[1]), P(out[2]), B, Hq, Hkv, Sq, Skv, d,
                        1, 0.088f, 0x12);
    };
    CHECK(bwd(ins, outs, 128, 2, 8, 2, 300, 500) == ATTN_OK);
    CHECK(g_bwd.NBQ == 3 && g_bwd.NKV == 4 && g_bwd.NX == 8 && g_bwd_mapping == 2 && g_bwd_causal);
    CHECK(g_bwd.order == attn::kOrderHeavyFirst && g_bwd.delta == (float *)P(kG));
    CHECK(bwd(ins, outs, 64, 2, 8, 2, 300, 500) == ATTN_ERR_UNSUPPORTED);
    // paired row blocks: a forward-only order
    CHECK(attn_bwd(P(kQ), P(kK), P(kV), P(kO), P(kD), (const float *)P(kL), (float *)P(kG), P(kX),
                   P(kY), P(kZ), 2, 8, 2, 300, 500, 128, 1, 0.088f, 0x52) == ATTN_ERR_MAPPING);
    for (int i = 0; i < 6; ++i) {   // a null input
        uintptr_t in[6];
        std::memcpy(in, ins, sizeof in);
        in[i] = 0;
        CHECK(bwd(in, outs, 128, 1, 4, 4, 256, 256) == ATTN_ERR_NULL);
    }
    for (int i = 0; i < 4; ++i) {   // a null output, a misaligned output
        uintptr_t out[4];
        std::memcpy(out, outs, sizeof out);
        out[i] = 0;
        CHECK(bwd(ins, out, 128, 1, 4, 4, 256, 256) == ATTN_ERR_NULL);
        out[i] = outs[i] + 2;
        CHECK(bwd(ins, out, 128, 1, 4, 4, 256, 256) == ATTN_ERR_ALIGN);
    }
    for (int i = 0; i < 4; ++i) {   // every output overlapping every input and output
        for (int j = 0; j < 6; ++j) {
            uintptr_t out[4];
            std::memcpy(out, outs, sizeof out);
            out[i] = ins[j] + 16;
            CHECK(bwd(ins, out, 128, 1, 4, 4, 256, 256) == ATTN_ERR_ALIAS);
        }
        for (int j = 0; j < 4; ++j) {
            if (j == i) continue;
            uintptr_t out[4];
            std::memcpy(out, outs, sizeof out);
            out[i] = outs[j] + 16;
            CHECK(bwd(ins, out, 128, 1, 4, 4, 256, 256) == ATTN_ERR_ALIAS);
        }
    }
}

void check_calib_and_misc() {
    int64_t *rec = (int64_t *)P(kX);
    float *sink = (float *)P(kY);
    CHECK(attn_calib_mfma(256, 20000, nullptr, sink) == ATTN_ERR_NULL);
    CHECK(attn_calib_mfma(0, 20000, rec, sink) == ATTN_ERR_SHAPE);
    CHECK(attn_calib_mfma(65537, 4, rec, sink) == ATTN_ERR_SHAPE);
    CHECK(attn_calib_mfma(256, 6, rec, sink) == ATTN_ERR_SHAPE);
    CHECK(attn_calib_mfma(256, (1 << 24) + 4, rec, sink) == ATTN_ERR_SHAPE);
    CHECK(attn_calib_mfma(256, 4, (int64_t *)P(kX + 4), sink) == ATTN_ERR_ALIGN);
    CHECK(attn_calib_mfma(256, 4, rec, (float *)P(kX + 8)) == ATTN_ERR_ALIAS);
    CHECK(attn_calib_mfma(256, 20000, rec, sink) == ATTN_OK);
    CHECK(g_calib_launches == 1 && g_calib_grid == 256 && g_calib_iters == 20000);

    CHECK(attn_grid_size(0, 1, 1, 128) == ATTN_ERR_SHAPE);
    CHECK(attn_grid_size(1, 1, 1, 96) == ATTN_ERR_UNSUPPORTED);
    CHECK(attn_grid_size(65536, 65536, 65536, 64) == (int64_t)65536 * 65536 * 512);
    CHECK(attn_block_n(56) == 64 && attn_block_m(96) == ATTN_ERR_UNSUPPORTED);

    CHECK(attn_set_stream(P(0x1234)) == ATTN_OK && attn_get_stream() == P(0x1234));
    CHECK(attn_set_stream(nullptr) == ATTN_OK && attn_get_stream() == nullptr);

    // the XCD count: environment override, else the device attribute
    setenv("ATTN_NUM_XCD", "4", 1);
    CHECK(attn_num_xcd() == 4);
    setenv("ATTN_NUM_XCD", "4x", 1);   // not a number: ignored
    CHECK(attn_num_xcd() == 8);
    setenv("ATTN_NUM_XCD", "65", 1);   // out of range: ignored
    CHECK(attn_num_xcd() == 8);
    unsetenv("ATTN_NUM_XCD");
    CHECK(attn_num_xcd() == 8);
}

// A failing HIP call surfaces as ATTN_ERR_HIP with its text; nothing launches.
void check_hip_failure() {
    CHECK(std::strcmp(attn_last_hip_error(), "") == 0);
    g_fail_device = true;
    const int launches = g_fwd_launches;
    // the persistent form asks for the compute-unit count of the current device
    CHECK(attn_fwd_persistent(P(kQ), P(kK), P(kV), P(kO), nullptr, (int32_t *)P(kW), nullptr, 1, 4,
                              4, 512, 512, 128, 1, 0.088f, 2) == ATTN_ERR_HIP);
    CHECK(std::strstr(attn_last_hip_error(), "stubbed HIP error") != nullptr);
    CHECK(g_fwd_launches == launches);
    g_fail_device = false;
}

struct MapCase {
    int mapping, B, Hq, Sq, d, NX;
};

void write_map_tables(const char *path) {
    const int shapes[][5] = {
        // B, Hq, Sq, d, NX
        {1, 4, 256, 64, 8},   {1, 32, 8192, 128, 8}, {2, 12, 300, 128, 8}, {3, 5, 1000, 64, 4},
        {1, 1, 1, 128, 8},    {2, 3, 129, 64, 1},    {1, 7, 1700, 128, 3}, {2, 128, 2048, 56, 8},
        {4, 6, 513, 128, 8},  {1, 64, 2176, 64, 8},  {3, 9, 4000, 128, 5},
    };
    // each value also with paired row blocks (head dimension 128 only)
    const int values[] = {0,    1,    2,    3,    0x10, 0x11, 0x12, 0x13, 0x22, 0x32,
                          0x40, 0x41, 0x42, 0x43, 0x50, 0x51, 0x52, 0x53, 0x62, 0x72};
    FILE *f = std::fopen(path, "wb");
    CHECK(f != nullptr);
    for (const auto &s : shapes) {
        for (int value : values) {
            const int64_t n = attn_grid_size(s[0], s[1], s[2], s[3]);
            CHECK(n > 0);
            // a sentinel no entry can hold: every row must be written
            std::vector<int32_t> out((size_t)n * 3, 0x7eadbeef);
            if ((value & 0x40) && s[3] != 128) {
                CHECK(attn_map_tiles(value, s[0], s[1], s[2], s[3], s[4], out.data()) ==
                      ATTN_ERR_UNSUPPORTED);
                continue;
            }
            CHECK(attn_map_tiles(value, s[0], s[1], s[2], s[3], s[4], out.data()) == ATTN_OK);
            const int32_t hdr[6] = {value, s[0], s[1], s[2], s[3], s[4]};
            CHECK(std::fwrite(hdr, sizeof hdr, 1, f) == 1);
            CHECK(std::fwrite(out.data(), sizeof(int32_t), out.size(), f) == out.size());
        }
    }
    CHECK(std::fclose(f) == 0);
    int32_t one[3];
    CHECK(attn_map_tiles(2, 1, 4, 256, 64, 8, nullptr) == ATTN_ERR_NULL);
    CHECK(attn_map_tiles(5, 1, 4, 256, 64, 8, one) == ATTN_ERR_MAPPING);
    CHECK(attn_map_tiles(0x21, 1, 4, 256, 64, 8, one) == ATTN_ERR_MAPPING);
    CHECK(attn_map_tiles(2, 1, 4, 256, 64, 0, one) == ATTN_ERR_SHAPE);
    CHECK(attn_map_tiles(2, 0, 4, 256, 64, 8, one) == ATTN_ERR_SHAPE);
    CHECK(attn_map_tiles(2, 65536, 65536, 65536, 64, 8, one) == ATTN_ERR_SHAPE);
}

}  // namespace

int main(int argc, char **argv) {
    if (argc != 2) {
        std::fprintf(stderr, "usage: %s OUT.bin\n", argv[0]);
        return 2;
    }
    unsetenv("ATTN_NUM_XCD");
    check_hip_failure();
    check_validation();
    check_forward_launch();
    check_lse_probe();
    check_persistent();
    check_backward();
    check_calib_and_misc();
    write_map_tables(argv[1]);
    std::printf("ok %d\n", g_checks);
    return 0;
}
