// attn_abi.cpp -- the C ABI of libattn_numa.so: argument validation, status
// codes, per-thread stream, XCD count, and the launch of the forward kernel.
// Every check runs on the host before the first HIP call, so invalid calls
// fail the same way with or without a GPU.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>

#include "attn_calib.h"
#include "attn_internal.h"
#include "attn_numa.h"

namespace {

thread_local hipStream_t t_stream = nullptr;
thread_local char t_hip_error[256] = "";

constexpr int kMaxDevices = 64;
std::atomic<int> g_nx_cache[kMaxDevices];   // 0 = not yet queried
std::atomic<int> g_cu_cache[kMaxDevices];   // compute units per device, 0 = not yet queried

int hip_fail(hipError_t e);

// Compute units of the current device (cached), or a negative ATTN_ERR_*.
static_assert(ATTN_QUEUE_INTS == attn::kQueueInts && attn::kQueueDone < ATTN_QUEUE_INTS,
              "queue layout");

int num_cu() {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e);
    if (dev < 0 || dev >= kMaxDevices) return ATTN_ERR_UNSUPPORTED;
    int n = g_cu_cache[dev].load(std::memory_order_relaxed);
    if (n > 0) return n;
    e = hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return hip_fail(e);
    if (n <= 0) return ATTN_ERR_UNSUPPORTED;
    g_cu_cache[dev].store(n, std::memory_order_relaxed);
    return n;
}

int hip_fail(hipError_t e) {
    std::snprintf(t_hip_error, sizeof t_hip_error, "%s (%d)", hipGetErrorString(e), (int)e);
    return ATTN_ERR_HIP;
}

bool supported_d(int d) { return d == 56 || d == 64 || d == 128; }

// Shape checks shared by every entry point.  Offsets inside one head are
// 32-bit byte offsets, so a head (plus one tile of slack) must stay below 2^31.
int check_shape(int B, int Hq, int Hkv, int Sq, int Skv, int d) {
    if (B <= 0 || Hq <= 0 || Hkv <= 0 || Sq <= 0 || Skv <= 0 || d <= 0) return ATTN_ERR_SHAPE;
    if (Hq % Hkv != 0) return ATTN_ERR_SHAPE;
    if (!supported_d(d)) return ATTN_ERR_UNSUPPORTED;
    const int64_t lim = INT32_MAX;
    if (((int64_t)Sq + attn::kMaxBlockM) * d * 2 > lim) return ATTN_ERR_SHAPE;
    if (((int64_t)Skv + 2 * attn::kBlockN) * d * 2 > lim) return ATTN_ERR_SHAPE;
    const int bm = attn::block_m_for(d);
    const int64_t nb = ((int64_t)Sq + bm - 1) / bm;
    if ((int64_t)B * Hq * nb > lim) return ATTN_ERR_SHAPE;
    return ATTN_OK;
}

// Base mapping in the low 4 bits, optional order flag above them.
bool valid_mapping(int mapping) {
    const int base = mapping & 0xf;
    const int flags = mapping & ~0xf;
    if (base < ATTN_MAP_NAIVE_BLOCK_FIRST || base > ATTN_MAP_SWIZZLED_BLOCK_FIRST) return false;
    if ((flags & ~(ATTN_ORDER_HEAVY_FIRST | ATTN_ORDER_XCD_BLOCK_MAJOR | ATTN_ORDER_PAIRED)) != 0)
        return false;
    // the block-major order inside an XCD's piece is defined for mapping 2 only
    return (flags & ATTN_ORDER_XCD_BLOCK_MAJOR) == 0 || base == ATTN_MAP_SWIZZLED_HEAD_FIRST;
}

int order_bits(int mapping) {
    return ((mapping & ATTN_ORDER_HEAVY_FIRST) ? attn::kOrderHeavyFirst : 0) |
           ((mapping & ATTN_ORDER_XCD_BLOCK_MAJOR) ? attn::kOrderXcdBlockMajor : 0) |
           ((mapping & ATTN_ORDER_PAIRED) ? attn::kOrderPaired : 0);
}

// Row blocks of a head that one workgroup's grid slot stands for: NB, or the
// pair slots of the paired order.
int slots_per_head(int NB, int mapping) {
    return (mapping & ATTN_ORDER_PAIRED) ? attn::pair_slots(NB) : NB;
}

bool overlaps(const void *a, int64_t a_bytes, const void *b, int64_t b_bytes) {
    const uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
    return a0 < b0 + (uintptr_t)b_bytes && b0 < a0 + (uintptr_t)a_bytes;
}

int validate(const void *q, const void *k, const void *v, const void *o, int B, int Hq, int Hkv,
             int Sq, int Skv, int d, float scale, int mapping) {
    if (!q || !k || !v || !o) return ATTN_ERR_NULL;
    int rc = check_shape(B, Hq, Hkv, Sq, Skv, d);
    if (rc) return rc;
    if (!valid_mapping(mapping)) return ATTN_ERR_MAPPING;
    if (!std::isfinite(scale) || !(scale > 0.0f)) return ATTN_ERR_SCALE;
    if (((uintptr_t)q | (uintptr_t)k | (uintptr_t)v | (uintptr_t)o) & 15u) return ATTN_ERR_ALIGN;
    const int64_t qo_bytes = (int64_t)B * Hq * Sq * d * 2;
    const int64_t kv_bytes = (int64_t)B * Hkv * Skv * d * 2;
    if (overlaps(o, qo_bytes, q, qo_bytes) || overlaps(o, qo_bytes, k, kv_bytes) ||
        overlaps(o, qo_bytes, v, kv_bytes))
        return ATTN_ERR_ALIAS;
    return ATTN_OK;
}

int env_num_xcd() {
    const char *s = std::getenv("ATTN_NUM_XCD");
    if (!s || !*s) return 0;
    char *end = nullptr;
    const long v = std::strtol(s, &end, 10);
    if (end == s || *end != '\0' || v <= 0 || v > 64) return 0;
    return (int)v;
}

// queue: the persistent form's caller-owned tile queues, or NULL; with
// use_static_queue the persistent form runs on the library's own queue array,
// cleared by a kernel on the stream right before the launch.
int run(const void *q, const void *k, const void *v, void *o, int B, int Hq, int Hkv, int Sq,
        int Skv, int d, int causal, float scale, int mapping, int32_t *probe, float *lse,
        int32_t *queue = nullptr, bool use_static_queue = false) {
    int rc = validate(q, k, v, o, B, Hq, Hkv, Sq, Skv, d, scale, mapping);
    if (rc) return rc;
    // pairs exist for the dispatched head-dimension-128 kernel only
    if ((mapping & ATTN_ORDER_PAIRED) && (d != 128 || queue || use_static_queue))
        return ATTN_ERR_UNSUPPORTED;
    if (lse) {
        if (((uintptr_t)lse) & 3u) return ATTN_ERR_ALIGN;
        const int64_t lse_bytes = (int64_t)B * Hq * Sq * 4;
        const int64_t qo_bytes = (int64_t)B * Hq * Sq * d * 2;
        const int64_t kv_bytes = (int64_t)B * Hkv * Skv * d * 2;
        if (overlaps(lse, lse_bytes, q, qo_bytes) || overlaps(lse, lse_bytes, k, kv_bytes) ||
            overlaps(lse, lse_bytes, v, kv_bytes) || overlaps(lse, lse_bytes, o, qo_bytes))
            return ATTN_ERR_ALIAS;
    }
    const int nx = attn_num_xcd();
    if (nx < 0) return nx;
    attn::KernelArgs a{};   // every field zero (no probe, lse or queue) unless set below
    a.q = q;
    a.k = k;
    a.v = v;
    a.o = o;
    a.probe = probe;
    a.lse = lse;
    a.queue = queue;
    a.B = B;
    a.Hq = Hq;
    a.Hkv = Hkv;
    a.Sq = Sq;
    a.Skv = Skv;
    a.NB = (Sq + attn::block_m_for(d) - 1) / attn::block_m_for(d);
    a.NX = nx;
    a.order = order_bits(mapping);
    a.scale_log2 = (float)((double)scale * 1.4426950408889634073599246810019);  // log2(e)
    int grid = B * Hq * slots_per_head(a.NB, mapping);
    if (queue || use_static_queue) {   // persistent form: one workgroup per compute unit, or per tile if fewer
        const int ncu = num_cu();
        if (ncu < 0) return ncu;
        if (nx > attn::kQueueMaxXcd) return ATTN_ERR_UNSUPPORTED;
        // With more workgroups than tiles the idle ones would take other XCDs'
        // tiles before those XCDs' own workgroups start.
        grid = grid < ncu ? grid : ncu;
    }
    if (use_static_queue) {
        int *sq = nullptr;
        hipError_t e = attn::static_queue(&sq);
        if (e != hipSuccess) return hip_fail(e);
        e = attn::launch_clear_queue(sq, t_stream);
        if (e != hipSuccess) return hip_fail(e);
        a.queue = sq;
    }
    hipError_t e = attn::launch_attn_fwd(a, d, causal != 0, mapping & 0xf, grid, t_stream);
    if (e != hipSuccess) return hip_fail(e);
    return ATTN_OK;
}

}  // namespace

extern "C" {

int attn_fwd(const void *q, const void *k, const void *v, void *o, int B, int Hq, int Hkv, int Sq,
             int Skv, int d, int causal, float scale, int mapping) {
    return run(q, k, v, o, B, Hq, Hkv, Sq, Skv, d, causal, scale, mapping, nullptr, nullptr);
}

int attn_fwd_lse(const void *q, const void *k, const void *v, void *o, float *lse, int B, int Hq,
                 int Hkv, int Sq, int Skv, int d, int causal, float scale, int mapping) {
    if (!lse) return ATTN_ERR_NULL;
    return run(q, k, v, o, B, Hq, Hkv, Sq, Skv, d, causal, scale, mapping, nullptr, lse);
}

int attn_bwd(const void *q, const void *k, const void *v, const void *o, const void *dout,
             const float *lse, float *delta, void *dq, void *dk, void *dv, int B, int Hq, int Hkv,
             int Sq, int Skv, int d, int causal, float scale, int mapping) {
    if (!dout || !lse || !delta || !dq || !dk || !dv) return ATTN_ERR_NULL;
    int rc = validate(q, k, v, o, B, Hq, Hkv, Sq, Skv, d, scale, mapping);
    if (rc) return rc;
    if (mapping & ATTN_ORDER_PAIRED) return ATTN_ERR_MAPPING;   // a forward-only order
    if (d != 128) return ATTN_ERR_UNSUPPORTED;
    if ((((uintptr_t)dout | (uintptr_t)dq | (uintptr_t)dk | (uintptr_t)dv) & 15u) ||
        (((uintptr_t)lse | (uintptr_t)delta) & 3u))
        return ATTN_ERR_ALIGN;
    if ((((int64_t)Skv + 128) * d * 2) > INT32_MAX) return ATTN_ERR_SHAPE;
    const int64_t qo = (int64_t)B * Hq * Sq * d * 2;
    const int64_t kv = (int64_t)B * Hkv * Skv * d * 2;
    const int64_t st = (int64_t)B * Hq * Sq * 4;
    const void *in[6] = {q, k, v, o, dout, lse};
    const int64_t in_bytes[6] = {qo, kv, kv, qo, qo, st};
    void *out[4] = {dq, dk, dv, delta};
    const int64_t out_bytes[4] = {qo, kv, kv, st};
    for (int i = 0; i < 4; ++i) {
        for (int j = 0; j < 6; ++j)
            if (overlaps(out[i], out_bytes[i], in[j], in_bytes[j])) return ATTN_ERR_ALIAS;
        for (int j = i + 1; j < 4; ++j)
            if (overlaps(out[i], out_bytes[i], out[j], out_bytes[j])) return ATTN_ERR_ALIAS;
    }
    const int nx = attn_num_xcd();
    if (nx < 0) return nx;
    attn::BwdArgs a{};
    a.q = q;
    a.k = k;
    a.v = v;
    a.o = o;
    a.dout = dout;
    a.lse = lse;
    a.delta = delta;
    a.dq = dq;
    a.dk = dk;
    a.dv = dv;
    a.B = B;
    a.Hq = Hq;
    a.Hkv = Hkv;
    a.Sq = Sq;
    a.Skv = Skv;
    a.NBQ = (Sq + 127) / 128;
    a.NKV = (Skv + 127) / 128;
    if ((int64_t)B * Hkv * a.NKV > INT32_MAX || (int64_t)B * Hq * a.NBQ > INT32_MAX ||
        ((int64_t)B * Hq * Sq + 15) / 16 > INT32_MAX)
        return ATTN_ERR_SHAPE;
    a.NX = nx;
    a.order = order_bits(mapping);
    a.scale = scale;
    a.scale_log2 = (float)((double)scale * 1.4426950408889634073599246810019);
    hipError_t e = attn::launch_attn_bwd(a, causal != 0, mapping & 0xf, t_stream);
    if (e != hipSuccess) return hip_fail(e);
    return ATTN_OK;
}

int attn_fwd_persistent(const void *q, const void *k, const void *v, void *o, float *lse,
                        int32_t *queue, int32_t *probe, int B, int Hq, int Hkv, int Sq, int Skv,
                        int d, int causal, float scale, int mapping) {
    if (!queue) return ATTN_ERR_NULL;
    if (((uintptr_t)queue & 3u) || ((uintptr_t)probe & 3u)) return ATTN_ERR_ALIGN;
    if (d != 128) return ATTN_ERR_UNSUPPORTED;
    const int64_t qo_bytes = (int64_t)B * Hq * Sq * d * 2;
    const int64_t kv_bytes = (int64_t)B * Hkv * Skv * d * 2;
    const int64_t qb = (int64_t)ATTN_QUEUE_INTS * 4;
    if (overlaps(queue, qb, q, qo_bytes) || overlaps(queue, qb, k, kv_bytes) ||
        overlaps(queue, qb, v, kv_bytes) || overlaps(queue, qb, o, qo_bytes) ||
        (lse && overlaps(queue, qb, lse, (int64_t)B * Hq * Sq * 4)))
        return ATTN_ERR_ALIAS;
    return run(q, k, v, o, B, Hq, Hkv, Sq, Skv, d, causal, scale, mapping, probe, lse, queue);
}

int attn_fwd_persistent_noalloc(const void *q, const void *k, const void *v, void *o, float *lse,
                                int32_t *probe, int B, int Hq, int Hkv, int Sq, int Skv, int d,
                                int causal, float scale, int mapping) {
    if (((uintptr_t)probe & 3u)) return ATTN_ERR_ALIGN;
    if (d != 128) return ATTN_ERR_UNSUPPORTED;
    return run(q, k, v, o, B, Hq, Hkv, Sq, Skv, d, causal, scale, mapping, probe, lse, nullptr,
               true);
}

int attn_fwd_probe(const void *q, const void *k, const void *v, void *o, int B, int Hq, int Hkv,
                   int Sq, int Skv, int d, int causal, float scale, int mapping, int32_t *probe) {
    if (!probe) return ATTN_ERR_NULL;
    if (((uintptr_t)probe) & 3u) return ATTN_ERR_ALIGN;
    return run(q, k, v, o, B, Hq, Hkv, Sq, Skv, d, causal, scale, mapping, probe, nullptr);
}

int attn_calib_mfma(int grid, int iters, int64_t *rec, float *sink) {
    if (!rec || !sink) return ATTN_ERR_NULL;
    if (grid <= 0 || grid > attn::kCalibMaxGrid || iters <= 0 || iters % 4 != 0 ||
        iters > attn::kCalibMaxIters)
        return ATTN_ERR_SHAPE;
    if (((uintptr_t)rec & 7u) || ((uintptr_t)sink & 3u)) return ATTN_ERR_ALIGN;
    if (overlaps(rec, (int64_t)grid * 4 * 8, sink, (int64_t)grid * attn::kCalibThreads * 4))
        return ATTN_ERR_ALIAS;
    const hipError_t e = attn::launch_calib_mfma(grid, iters, rec, sink, t_stream);
    return e == hipSuccess ? ATTN_OK : hip_fail(e);
}

int64_t attn_grid_size(int B, int Hq, int Sq, int d) {
    if (B <= 0 || Hq <= 0 || Sq <= 0 || d <= 0) return ATTN_ERR_SHAPE;
    if (!supported_d(d)) return ATTN_ERR_UNSUPPORTED;
    const int bm = attn::block_m_for(d);
    return (int64_t)B * Hq * (((int64_t)Sq + bm - 1) / bm);
}

int attn_map_tiles(int mapping, int B, int Hq, int Sq, int d, int NX, int32_t *out) {
    if (!out) return ATTN_ERR_NULL;
    if (!valid_mapping(mapping)) return ATTN_ERR_MAPPING;
    if (NX <= 0) return ATTN_ERR_SHAPE;
    const int64_t n = attn_grid_size(B, Hq, Sq, d);
    if (n < 0) return (int)n;
    if (n > INT32_MAX) return ATTN_ERR_SHAPE;
    const int nb = (Sq + attn::block_m_for(d) - 1) / attn::block_m_for(d);
    const bool paired = (mapping & ATTN_ORDER_PAIRED) != 0;
    if (paired && d != 128) return ATTN_ERR_UNSUPPORTED;
    // the four-wave kernel (128-row blocks) uses the 16-head groups for short heads
    const bool short_groups = attn::block_m_for(d) == attn::kBlockM;
    const int64_t slots = (int64_t)B * Hq * slots_per_head(nb, mapping);
    for (int64_t wid = 0; wid < n; ++wid) {
        if (wid >= slots) {   // past the paired grid: no workgroup
            out[3 * wid + 0] = out[3 * wid + 1] = out[3 * wid + 2] = -1;
            continue;
        }
        attn::Tile t = attn::map_wid(mapping & 0xf, order_bits(mapping), (int)wid, B, Hq,
                                     slots_per_head(nb, mapping), NX, short_groups);
        if (paired) t.m = nb - 1 - t.m;   // the slot's first row block
        out[3 * wid + 0] = t.b;
        out[3 * wid + 1] = t.hq;
        out[3 * wid + 2] = t.m;
    }
    return ATTN_OK;
}

int attn_block_m(int d) { return supported_d(d) ? attn::block_m_for(d) : ATTN_ERR_UNSUPPORTED; }

int attn_block_n(int d) { return supported_d(d) ? attn::kBlockN : ATTN_ERR_UNSUPPORTED; }

int attn_num_xcd(void) {
    const int env = env_num_xcd();
    if (env > 0) return env;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e);
    if (dev < 0 || dev >= kMaxDevices) return ATTN_ERR_UNSUPPORTED;
    int nx = g_nx_cache[dev].load(std::memory_order_relaxed);
    if (nx > 0) return nx;
    e = hipDeviceGetAttribute(&nx, hipDeviceAttributeNumberOfXccs, dev);
    if (e != hipSuccess) return hip_fail(e);
    if (nx <= 0) nx = 1;
    g_nx_cache[dev].store(nx, std::memory_order_relaxed);
    return nx;
}

int attn_set_stream(void *hip_stream) {
    t_stream = (hipStream_t)hip_stream;
    return ATTN_OK;
}

void *attn_get_stream(void) { return (void *)t_stream; }

const char *attn_strerror(int code) {
    switch (code) {
        case ATTN_OK: return "ok";
        case ATTN_ERR_NULL: return "null pointer argument";
        case ATTN_ERR_SHAPE: return "invalid shape (non-positive dimension, Hq % Hkv != 0, or size limit)";
        case ATTN_ERR_UNSUPPORTED: return "unsupported head dimension (forward: 56, 64, 128; backward and persistent forward: 128)";
        case ATTN_ERR_MAPPING: return "unknown mapping (0 naive block-first, 1 naive head-first, 2 swizzled head-first, 3 swizzled block-first, optionally | ATTN_ORDER_HEAVY_FIRST, for 2 | ATTN_ORDER_XCD_BLOCK_MAJOR, and in the forward | ATTN_ORDER_PAIRED)";
        case ATTN_ERR_SCALE: return "scale must be finite and > 0";
        case ATTN_ERR_ALIGN: return "pointer not aligned (bf16 tensors: 16 bytes; fp32 and int32 buffers: 4 bytes; int64 buffers: 8 bytes)";
        case ATTN_ERR_HIP: return "HIP runtime error";
        case ATTN_ERR_ALIAS: return "output overlaps an input";
        default: return "unknown status code";
    }
}

const char *attn_last_hip_error(void) { return t_hip_error; }

}  // extern "C"
