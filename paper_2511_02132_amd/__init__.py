"""Python binding of libattn_numa.so: NUMA-aware fused attention on MI355X.

Argument marshalling only.  Every step of the computation runs in the HIP
kernels of ``csrc/``; there is no CPU fallback, and a missing library is an
error.  Torch provides device memory and streams.

    from paper_2511_02132_amd import attn_fwd, SWIZZLED_HEAD_FIRST
    o = attn_fwd(q, k, v, causal=True, mapping=SWIZZLED_HEAD_FIRST)
    o, lse = attn_fwd_lse(q, k, v, causal=True)            # training forward
    dq, dk, dv = attn_bwd(q, k, v, o, do, lse, causal=True)  # d = 128

q: [B, Hq, Sq, d], k/v: [B, Hkv, Skv, d], bf16, contiguous, on the GPU;
d in {56, 64, 128} (the backward and the persistent form: d = 128); Hq a
multiple of Hkv (grouped-query attention).
"""

from __future__ import annotations

import ctypes
import math
import os

import numpy as np

NAIVE_BLOCK_FIRST = 0
NAIVE_HEAD_FIRST = 1
SWIZZLED_HEAD_FIRST = 2
SWIZZLED_BLOCK_FIRST = 3
# Flag OR-ed into a mapping: dispatch each head's row blocks last-to-first.
HEAVY_FIRST = 0x10
# Flag for SWIZZLED_HEAD_FIRST: dispatch each XCD's piece of whole heads block-major
# within groups of four heads (heads of at most 64 row blocks; longer ones keep
# head-major order).
XCD_BLOCK_MAJOR = 0x20
# Flag for the dispatched forward with d = 128: one workgroup per pair of row
# blocks (NB-1-p, then p) of a head, ceil(NB/2) slots per head placed by the
# mapping; under a causal mask every pair costs the same.
PAIRED = 0x40
MAPPINGS = {"naive_block_first": NAIVE_BLOCK_FIRST, "naive_head_first": NAIVE_HEAD_FIRST,
            "swizzled_head_first": SWIZZLED_HEAD_FIRST, "swizzled_block_first": SWIZZLED_BLOCK_FIRST}
MAPPING_NAMES = ["naive_block_first", "naive_head_first", "swizzled_head_first",
                 "swizzled_block_first"]


def variant_name(mapping: int) -> str:
    """Name of a mapping value with its order flags, e.g. 'swizzled_head_first+heavy_first'."""
    name = MAPPING_NAMES[mapping & 0xF]
    if mapping & HEAVY_FIRST:
        name += "+heavy_first"
    if mapping & XCD_BLOCK_MAJOR:
        name += "+xcd_block_major"
    if mapping & PAIRED:
        name += "+paired"
    return name


def variants(causal: bool, d: int = 128, backward: bool = False):
    """(name, mapping value) of every variant the measurements compare: the four
    mappings; under a causal mask each also with the heavy-first order;
    swizzled head-first with the block-major order inside each XCD; and, for the
    d = 128 forward under a causal mask, the three mappings that keep heads or
    KV groups together (naive block-first, swizzled head-first, swizzled
    block-first) with heavy-first paired row blocks."""
    vals = list(range(4)) + [SWIZZLED_HEAD_FIRST | XCD_BLOCK_MAJOR]
    if causal:
        vals = list(range(4)) + [m | HEAVY_FIRST for m in range(4)] + \
            [SWIZZLED_HEAD_FIRST | HEAVY_FIRST | XCD_BLOCK_MAJOR]
        if d == 128 and not backward:
            vals += [m | HEAVY_FIRST | PAIRED for m in (NAIVE_BLOCK_FIRST, SWIZZLED_HEAD_FIRST,
                                                        SWIZZLED_BLOCK_FIRST)]
    return [(variant_name(v), v) for v in vals]


def method_variant(causal: bool) -> int:
    """The mapping value the headline uses: the paper's swizzled head-first
    placement (each XCD serves one (batch, KV head) at a time); under a causal
    mask each head's row blocks are dispatched heaviest first."""
    if causal:
        return SWIZZLED_HEAD_FIRST | HEAVY_FIRST
    return SWIZZLED_HEAD_FIRST

ATTN_OK = 0
ATTN_ERR = {-1: "ATTN_ERR_NULL", -2: "ATTN_ERR_SHAPE", -3: "ATTN_ERR_UNSUPPORTED",
            -4: "ATTN_ERR_MAPPING", -5: "ATTN_ERR_SCALE", -6: "ATTN_ERR_ALIGN",
            -7: "ATTN_ERR_HIP", -8: "ATTN_ERR_ALIAS"}

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libattn_numa.so")

# Every symbol include/attn_numa.h declares, with its ctypes signature.
_vp, _ci, _cf = ctypes.c_void_p, ctypes.c_int, ctypes.c_float
_i32p = ctypes.POINTER(ctypes.c_int32)
SIGNATURES = {
    "attn_fwd": ([_vp, _vp, _vp, _vp, _ci, _ci, _ci, _ci, _ci, _ci, _ci, _cf, _ci], _ci),
    "attn_fwd_probe": ([_vp, _vp, _vp, _vp, _ci, _ci, _ci, _ci, _ci, _ci, _ci, _cf, _ci, _vp],
                       _ci),
    "attn_fwd_lse": ([_vp, _vp, _vp, _vp, _vp, _ci, _ci, _ci, _ci, _ci, _ci, _ci, _cf, _ci], _ci),
    "attn_fwd_persistent": ([_vp] * 7 + [_ci, _ci, _ci, _ci, _ci, _ci, _ci, _cf, _ci], _ci),
    "attn_fwd_persistent_noalloc": ([_vp] * 6 + [_ci, _ci, _ci, _ci, _ci, _ci, _ci, _cf, _ci],
                                    _ci),
    "attn_bwd": ([_vp] * 10 + [_ci, _ci, _ci, _ci, _ci, _ci, _ci, _cf, _ci], _ci),
    "attn_calib_mfma": ([_ci, _ci, _vp, _vp], _ci),
    "attn_grid_size": ([_ci, _ci, _ci, _ci], ctypes.c_int64),
    "attn_map_tiles": ([_ci, _ci, _ci, _ci, _ci, _ci, _i32p], _ci),
    "attn_block_m": ([_ci], _ci),
    "attn_block_n": ([_ci], _ci),
    "attn_num_xcd": ([], _ci),
    "attn_set_stream": ([_vp], _ci),
    "attn_get_stream": ([], _vp),
    "attn_strerror": ([_ci], ctypes.c_char_p),
    "attn_last_hip_error": ([], ctypes.c_char_p),
}

_lib = None


class AttnError(RuntimeError):
    def __init__(self, code: int, what: str):
        self.code = code
        super().__init__(what)


def lib() -> ctypes.CDLL:
    """The loaded, typed library.  Raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError("%s is missing: build it with `python -m paper_2511_02132_amd.build`"
                              % LIB_PATH)
        handle = ctypes.CDLL(LIB_PATH)
        for name, (argtypes, restype) in SIGNATURES.items():
            fn = getattr(handle, name)
            fn.argtypes = argtypes
            fn.restype = restype
        _lib = handle
    return _lib


def strerror(code: int) -> str:
    return lib().attn_strerror(code).decode()


def _check(rc: int, what: str) -> int:
    if rc < 0:
        msg = "%s failed: %s (%s)" % (what, ATTN_ERR.get(rc, rc), strerror(rc))
        if rc == -7:
            msg += ": " + lib().attn_last_hip_error().decode()
        raise AttnError(rc, msg)
    return rc


def block_m(d: int) -> int:
    return _check(lib().attn_block_m(d), "attn_block_m")


def block_n(d: int) -> int:
    return _check(lib().attn_block_n(d), "attn_block_n")


def grid_size(B: int, Hq: int, Sq: int, d: int) -> int:
    return _check(lib().attn_grid_size(B, Hq, Sq, d), "attn_grid_size")


def num_xcd() -> int:
    return _check(lib().attn_num_xcd(), "attn_num_xcd")


def map_tiles(mapping: int, B: int, Hq: int, Sq: int, d: int, NX: int) -> np.ndarray:
    """[N, 3] int32 (b, hq, m) per workgroup id, from the library's own mapping code."""
    n = grid_size(B, Hq, Sq, d)
    out = np.empty((n, 3), dtype=np.int32)
    _check(lib().attn_map_tiles(mapping, B, Hq, Sq, d, NX, out.ctypes.data_as(_i32p)),
           "attn_map_tiles")
    return out


def _shapes(q, k, v, o):
    import torch
    for name, t in (("q", q), ("k", k), ("v", v), ("o", o)):
        if not isinstance(t, torch.Tensor):
            raise TypeError("%s must be a torch.Tensor" % name)
        if t.dtype != torch.bfloat16:
            raise TypeError("%s must be bfloat16, got %s" % (name, t.dtype))
        if t.device.type != "cuda":
            raise ValueError("%s must be on the GPU, got %s" % (name, t.device))
        if not t.is_contiguous():
            raise ValueError("%s must be contiguous (BHSD)" % name)
        if t.dim() != 4:
            raise ValueError("%s must be 4-D [B, H, S, d]" % name)
    B, Hq, Sq, d = q.shape
    Bk, Hkv, Skv, dk = k.shape
    if tuple(v.shape) != tuple(k.shape) or Bk != B or dk != d:
        raise ValueError("k and v must be [B, Hkv, Skv, d] matching q")
    if tuple(o.shape) != tuple(q.shape):
        raise ValueError("o must have q's shape")
    if not (q.device == k.device == v.device == o.device):
        raise ValueError("all tensors must be on one device")
    return B, Hq, Hkv, Sq, Skv, d


def _prepare(q, k, v, o, scale, stream):
    import torch
    if o is None:
        o = torch.empty_like(q)
    B, Hq, Hkv, Sq, Skv, d = _shapes(q, k, v, o)
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    if stream is None:
        stream = torch.cuda.current_stream(q.device)
    torch.cuda.set_device(q.device)
    lib().attn_set_stream(ctypes.c_void_p(stream.cuda_stream))
    return o, (B, Hq, Hkv, Sq, Skv, d), float(scale)


def attn_fwd(q, k, v, o=None, *, causal: bool = False, scale: float | None = None,
             mapping: int = SWIZZLED_HEAD_FIRST, stream=None):
    """O = softmax(scale * Q K^T [causal]) V on the GPU; returns o (enqueued, not synced)."""
    o, (B, Hq, Hkv, Sq, Skv, d), scale = _prepare(q, k, v, o, scale, stream)
    _check(lib().attn_fwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                          B, Hq, Hkv, Sq, Skv, d, int(bool(causal)), scale, int(mapping)),
           "attn_fwd")
    return o


def attn_fwd_probe(q, k, v, o=None, probe=None, *, causal: bool = False,
                   scale: float | None = None, mapping: int = SWIZZLED_HEAD_FIRST, stream=None):
    """attn_fwd plus the per-workgroup record [N, 4] int32 = (b, hq, m, xcc)."""
    import torch
    o, (B, Hq, Hkv, Sq, Skv, d), scale = _prepare(q, k, v, o, scale, stream)
    n = grid_size(B, Hq, Sq, d)
    if probe is None:
        probe = torch.full((n, 4), -1, dtype=torch.int32, device=q.device)
    if probe.dtype != torch.int32 or probe.numel() < 4 * n or not probe.is_contiguous() \
            or probe.device != q.device:
        raise ValueError("probe must be a contiguous int32 GPU tensor with >= 4*N elements")
    _check(lib().attn_fwd_probe(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                                B, Hq, Hkv, Sq, Skv, d, int(bool(causal)), scale, int(mapping),
                                probe.data_ptr()),
           "attn_fwd_probe")
    return o, probe


def attn_fwd_lse(q, k, v, o=None, lse=None, *, causal: bool = False, scale: float | None = None,
                 mapping: int = SWIZZLED_HEAD_FIRST, stream=None):
    """attn_fwd that also returns the row log-sum-exp lse [B, Hq, Sq] fp32."""
    import torch
    o, (B, Hq, Hkv, Sq, Skv, d), scale = _prepare(q, k, v, o, scale, stream)
    if lse is None:
        lse = torch.empty((B, Hq, Sq), dtype=torch.float32, device=q.device)
    _check_stat(lse, (B, Hq, Sq), q.device, "lse")
    _check(lib().attn_fwd_lse(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                              lse.data_ptr(), B, Hq, Hkv, Sq, Skv, d, int(bool(causal)), scale,
                              int(mapping)),
           "attn_fwd_lse")
    return o, lse


QUEUE_INTS = 64   # ATTN_QUEUE_INTS


def new_queue(device):
    """A zeroed tile-queue buffer for attn_fwd_persistent (reusable on one stream)."""
    import torch
    return torch.zeros(QUEUE_INTS, dtype=torch.int32, device=device)


def attn_fwd_persistent(q, k, v, o=None, *, lse=None, queue=None, probe=None,
                        causal: bool = False, scale: float | None = None,
                        mapping: int = SWIZZLED_HEAD_FIRST, stream=None):
    """attn_fwd in the persistent form (one workgroup per CU pulling tiles from
    per-XCD queues; d = 128).  Returns o (and writes lse / probe when given)."""
    import torch
    o, (B, Hq, Hkv, Sq, Skv, d), scale = _prepare(q, k, v, o, scale, stream)
    if queue is None:
        queue = new_queue(q.device)
    if queue.dtype != torch.int32 or queue.numel() < QUEUE_INTS or not queue.is_contiguous() \
            or queue.device != q.device:
        raise ValueError("queue must be a contiguous int32 GPU tensor of %d zeros" % QUEUE_INTS)
    if lse is not None:
        _check_stat(lse, (B, Hq, Sq), q.device, "lse")
    if probe is not None and (probe.dtype != torch.int32 or not probe.is_contiguous()
                              or probe.numel() < 4 * grid_size(B, Hq, Sq, d)
                              or probe.device != q.device):
        raise ValueError("probe must be a contiguous int32 GPU tensor with >= 4*N elements")
    _check(lib().attn_fwd_persistent(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                                     None if lse is None else lse.data_ptr(), queue.data_ptr(),
                                     None if probe is None else probe.data_ptr(),
                                     B, Hq, Hkv, Sq, Skv, d, int(bool(causal)), scale,
                                     int(mapping)),
           "attn_fwd_persistent")
    return o


def attn_fwd_persistent_noalloc(q, k, v, o, *, lse=None, probe=None, causal: bool = False,
                                scale: float | None = None, mapping: int = SWIZZLED_HEAD_FIRST,
                                stream=None):
    """attn_fwd_persistent on the library's own tile-queue array: the call
    allocates nothing (o, and lse / probe when wanted, come from the caller).
    Calls that may overlap on one GPU race on that array; order them on one
    stream."""
    import torch
    if o is None:
        raise ValueError("o must be given: this call allocates nothing")
    o, (B, Hq, Hkv, Sq, Skv, d), scale = _prepare(q, k, v, o, scale, stream)
    if lse is not None:
        _check_stat(lse, (B, Hq, Sq), q.device, "lse")
    if probe is not None and (probe.dtype != torch.int32 or not probe.is_contiguous()
                              or probe.numel() < 4 * grid_size(B, Hq, Sq, d)
                              or probe.device != q.device):
        raise ValueError("probe must be a contiguous int32 GPU tensor with >= 4*N elements")
    _check(lib().attn_fwd_persistent_noalloc(q.data_ptr(), k.data_ptr(), v.data_ptr(),
                                             o.data_ptr(),
                                             None if lse is None else lse.data_ptr(),
                                             None if probe is None else probe.data_ptr(),
                                             B, Hq, Hkv, Sq, Skv, d, int(bool(causal)), scale,
                                             int(mapping)),
           "attn_fwd_persistent_noalloc")
    return o


def _check_stat(t, shape, device, name):
    import torch
    if not isinstance(t, torch.Tensor) or t.dtype != torch.float32 or tuple(t.shape) != shape \
            or not t.is_contiguous() or t.device != device:
        raise ValueError("%s must be a contiguous float32 GPU tensor of shape %s" % (name, shape))


def attn_bwd(q, k, v, o, dout, lse, dq=None, dk=None, dv=None, delta=None, *,
             causal: bool = False, scale: float | None = None,
             mapping: int = SWIZZLED_HEAD_FIRST, stream=None):
    """Gradients (dq, dk, dv) of attn_fwd for dL/dO = dout (bf16; d = 128).

    o and lse come from attn_fwd_lse with the same causal/scale; delta is a
    float32 [B, Hq, Sq] workspace (allocated here when not given)."""
    import torch
    _, (B, Hq, Hkv, Sq, Skv, d), scale = _prepare(q, k, v, o, scale, stream)
    _shapes(q, k, v, dout)
    if dq is None:
        dq = torch.empty_like(q)
    if dk is None:
        dk = torch.empty_like(k)
    if dv is None:
        dv = torch.empty_like(v)
    if delta is None:
        delta = torch.empty((B, Hq, Sq), dtype=torch.float32, device=q.device)
    _shapes(dq, dk, dv, dq)
    _check_stat(lse, (B, Hq, Sq), q.device, "lse")
    _check_stat(delta, (B, Hq, Sq), q.device, "delta")
    _check(lib().attn_bwd(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(),
                          dout.data_ptr(), lse.data_ptr(), delta.data_ptr(), dq.data_ptr(),
                          dk.data_ptr(), dv.data_ptr(), B, Hq, Hkv, Sq, Skv, d,
                          int(bool(causal)), scale, int(mapping)),
           "attn_bwd")
    return dq, dk, dv


CALIB_THREADS = 512


def calib_mfma(device=None, *, grid: int | None = None, iters: int = 20000, launches: int = 8,
               stream=None) -> list:
    """Matrix-core calibration (attn_calib_mfma), `launches` launches back to back.

    Per launch: its time from HIP events on the stream (ms), the dense bf16
    rate (TFLOP/s) and the median shader clock of its workgroups (MHz).  The
    grid defaults to one workgroup per compute unit."""
    import torch
    device = torch.device(device if device is not None else "cuda")
    torch.cuda.set_device(device)
    if grid is None:
        grid = torch.cuda.get_device_properties(device).multi_processor_count
    if stream is None:
        stream = torch.cuda.current_stream(device)
    lib().attn_set_stream(ctypes.c_void_p(stream.cuda_stream))
    rec = torch.zeros((launches, grid, 4), dtype=torch.int64, device=device)
    sink = torch.empty(grid * CALIB_THREADS, dtype=torch.float32, device=device)
    flop = 32768.0 * 4 * iters * 8 * grid
    events = [torch.cuda.Event(enable_timing=True) for _ in range(launches + 1)]
    events[0].record(stream)
    for i in range(launches):
        _check(lib().attn_calib_mfma(grid, iters, rec[i].data_ptr(), sink.data_ptr()),
               "attn_calib_mfma")
        events[i + 1].record(stream)
    torch.cuda.synchronize(device)
    r = rec.cpu().numpy().astype(np.float64)
    out = []
    for i in range(launches):
        ms = events[i].elapsed_time(events[i + 1])
        mhz = (r[i, :, 3] - r[i, :, 2]) / (r[i, :, 1] - r[i, :, 0]) * 100.0
        out.append({"ms": ms, "tflops": flop / ms / 1e9, "clock_mhz": float(np.median(mhz))})
    return out


def attention_flops(B: int, Hq: int, Sq: int, Skv: int, d: int, causal: bool) -> float:
    """FlashAttention convention: 4*B*Hq*Sq*Skv*d, halved when causal."""
    f = 4.0 * B * Hq * Sq * Skv * d
    return f / 2 if causal else f


def attention_bwd_flops(B: int, Hq: int, Sq: int, Skv: int, d: int, causal: bool) -> float:
    """FlashAttention convention for the backward: 2.5x the forward (five products)."""
    return 2.5 * attention_flops(B, Hq, Sq, Skv, d, causal)
