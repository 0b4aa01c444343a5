"""Python binding of libhyq, the MI355X (gfx950) HyQuant hybrid-precision
attention library (prefill operator, and the decode cache with its
attention).

The functions here carry the C ABI's names (``include/hyq.h``) and only
marshal arguments: torch tensors (device memory) become pointers, the
current torch stream becomes the HIP stream.  Every step of the path runs in
the library's HIP kernels; there is no fallback.  Before any call the
binding checks that every buffer has the dtype, device, contiguity and byte
size the shape requires, so a kernel never sees a buffer smaller than its
grid assumes.
"""
from __future__ import annotations

import ctypes
import dataclasses
import math
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libhyq.so")

HYQ_OK, HYQ_EINVAL, HYQ_EUNSUPPORTED, HYQ_EHIP = 0, -1, -2, -3
KQ_POS_PAD = 0x7FFFFFFF
FMT_INT, FMT_FP8, FMT_FP4, FMT_FP4Q6 = 0, 1, 2, 3   # hyq_shape.kv_format
WIN_FIXED, WIN_BAND = 0, 1    # hyq_shape.window_mode
SEL_PROXY, SEL_COLMASS = 0, 1  # hyq_shape.selector
DECODE_WS = 64                # HYQ_DECODE_WS: staging buffer capacity
EXPORTED = ("hyq_sizes_for", "hyq_select_vertical", "hyq_quantize", "hyq_attn_prefill",
            "hyq_prefill", "hyq_strerror", "hyq_last_error", "hyq_dcache_init", "hyq_freeze",
            "hyq_decode_append", "hyq_decode_attn", "hyq_decode_attn_noalloc")


class HyqError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"libhyq error {code}: {msg}")
        self.code = code


class _Shape(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in
                ("B", "Hq", "Hkv", "L", "D", "window", "budget_ppm", "bits_kv", "block",
                 "kv_format", "window_mode", "selector", "staging")]


class _Sizes(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in ("P", "k", "nQ", "n_qblk", "n_kvblk", "kv_row_bytes")] + \
               [(n, ctypes.c_size_t) for n in ("idx_bytes", "kq_pos_bytes", "q_codes_bytes",
                                               "q_scale_bytes", "k_codes_bytes", "v_codes_bytes",
                                               "kv_scale_bytes", "scores_bytes", "select_ws_bytes")]


_DCACHE_INTS = ("B", "Hq", "Hkv", "D", "window", "bits_kv", "kv_format", "n_vl", "vl_rows",
                "ring_rows", "n_frozen", "cap_blocks", "n_merged", "ring_head", "n_staged",
                "staging")
_DCACHE_PTRS = ("k_codes", "v_codes", "k_scale", "v_scale", "q_pos", "fp_k", "fp_v", "vl_pos")


class _DCache(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in _DCACHE_INTS] + [("t", ctypes.c_int64)] + \
               [(n, ctypes.c_void_p) for n in _DCACHE_PTRS]


_DSIZES = ("k_codes_bytes", "v_codes_bytes", "k_scale_bytes", "v_scale_bytes", "q_pos_bytes",
           "fp_k_bytes", "fp_v_bytes", "vl_pos_bytes", "freeze_ws_bytes", "attn_ws_bytes")


class _DCacheSizes(ctypes.Structure):
    _fields_ = [(n, ctypes.c_size_t) for n in _DSIZES]


@dataclasses.dataclass(frozen=True)
class Shape:
    """Problem shape (mirrors ``hyq_shape``)."""
    B: int
    Hq: int
    Hkv: int
    L: int
    D: int = 128
    window: int = 0
    budget_ppm: int = 0
    bits_kv: int = 8
    block: int = 64
    kv_format: int = 0      # FMT_INT, FMT_FP8 (bits 8), FMT_FP4 or FMT_FP4Q6 (bits 4)
    window_mode: int = 0    # WIN_FIXED or WIN_BAND
    selector: int = 0       # SEL_PROXY (Algorithm 1) or SEL_COLMASS (eq. vl_score)
    staging: int = 0        # decode staging capacity W_s: 0 = DECODE_WS, else a multiple of 64

    def c(self) -> _Shape:
        return _Shape(*[int(getattr(self, f.name)) for f in dataclasses.fields(self)])


_lib = None


def lib():
    """The loaded libhyq (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(
                f"{LIB_PATH} is missing: build it with `python -m paper_2608_27875_amd.build` "
                "(the HIP library is required; there is no fallback)")
        L = ctypes.CDLL(LIB_PATH)
        P = ctypes.c_void_p
        L.hyq_sizes_for.argtypes = [ctypes.POINTER(_Shape), ctypes.POINTER(_Sizes)]
        L.hyq_select_vertical.argtypes = [ctypes.POINTER(_Shape), P, P, P, P, P, ctypes.c_size_t, P]
        L.hyq_quantize.argtypes = [ctypes.POINTER(_Shape)] + [P] * 12
        L.hyq_attn_prefill.argtypes = [ctypes.POINTER(_Shape)] + [P] * 11 + \
            [ctypes.c_float, P, ctypes.c_int32, P]
        L.hyq_prefill.argtypes = [ctypes.POINTER(_Shape)] + [P] * 11 + \
            [ctypes.c_float, P, ctypes.c_int32, P, ctypes.c_size_t, P]
        L.hyq_strerror.restype = ctypes.c_char_p
        L.hyq_strerror.argtypes = [ctypes.c_int]
        L.hyq_last_error.restype = ctypes.c_char_p
        L.hyq_last_error.argtypes = []
        DC = ctypes.POINTER(_DCache)
        L.hyq_dcache_init.argtypes = [ctypes.POINTER(_Shape), ctypes.c_int64, DC,
                                      ctypes.POINTER(_DCacheSizes)]
        L.hyq_freeze.argtypes = [ctypes.POINTER(_Shape), P, P, P, DC, P, ctypes.c_size_t, P]
        L.hyq_decode_append.argtypes = [DC, P, P, P]
        L.hyq_decode_attn.argtypes = [DC, P, ctypes.c_float, P, ctypes.c_int32, P,
                                      ctypes.c_size_t, P]
        L.hyq_decode_attn_noalloc.argtypes = [DC, P, ctypes.c_float, P, ctypes.c_int32, P]
        for f in ("hyq_sizes_for", "hyq_select_vertical", "hyq_quantize", "hyq_attn_prefill",
                  "hyq_prefill", "hyq_dcache_init", "hyq_freeze", "hyq_decode_append", "hyq_decode_attn",
                  "hyq_decode_attn_noalloc"):
            getattr(L, f).restype = ctypes.c_int
        _lib = L
    return _lib


def _check(rc: int):
    if rc != HYQ_OK:
        raise HyqError(rc, lib().hyq_last_error().decode() or lib().hyq_strerror(rc).decode())


def hyq_sizes_for(shape: Shape) -> dict:
    z = _Sizes()
    _check(lib().hyq_sizes_for(ctypes.byref(shape.c()), ctypes.byref(z)))
    return {n: getattr(z, n) for n, _ in _Sizes._fields_}


def hyq_strerror(code: int) -> str:
    return lib().hyq_strerror(code).decode()


def hyq_last_error() -> str:
    return lib().hyq_last_error().decode()


# --------------------------------------------------------------------------
# argument marshalling
# --------------------------------------------------------------------------

def _torch():
    import torch
    return torch


def _stream(stream):
    torch = _torch()
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def _ptr(t, name, nbytes, dtypes, device, allow_none=False):
    """Pointer of tensor ``t`` after checking dtype, device, contiguity and size."""
    if t is None:
        if allow_none or nbytes == 0:
            return None
        raise ValueError(f"{name} is required")
    if t.dtype not in dtypes:
        raise TypeError(f"{name}: dtype {t.dtype} not in {dtypes}")
    if t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    have = t.numel() * t.element_size()
    if have < nbytes:
        raise ValueError(f"{name} holds {have} bytes, needs {nbytes}")
    return ctypes.c_void_p(t.data_ptr()) if t.numel() else None


def _io(shape: Shape, Q, K, V=None):
    torch = _torch()
    B, Hq, Hkv, L, D = shape.B, shape.Hq, shape.Hkv, shape.L, shape.D
    if Q.device.type != "cuda":
        raise ValueError("tensors must be on a GPU")
    dev = Q.device
    bf = (torch.bfloat16,)
    want = {"Q": (B, Hq, L, D), "K": (B, Hkv, L, D), "V": (B, Hkv, L, D)}
    for n, t in (("Q", Q), ("K", K), ("V", V)):
        if t is None:
            continue
        if tuple(t.shape) != want[n]:
            raise ValueError(f"{n} has shape {tuple(t.shape)}, expected {want[n]}")
    return dev, bf


def hyq_select_vertical(shape: Shape, Q, K, idx, scores=None, ws=None, stream=None):
    """Algorithm 1 (see include/hyq.h); writes idx [B,Hkv,k] (and scores)."""
    torch = _torch()
    z = hyq_sizes_for(shape)
    dev, bf = _io(shape, Q, K)
    args = [
        _ptr(Q, "Q", Q.numel() * 2, bf, dev),
        _ptr(K, "K", K.numel() * 2, bf, dev),
        _ptr(idx, "idx", z["idx_bytes"], (torch.int32,), dev),
        _ptr(scores, "scores", z["scores_bytes"], (torch.float32,), dev, allow_none=True),
        _ptr(ws, "ws", z["select_ws_bytes"], (torch.uint8, torch.int8, torch.float32), dev),
    ]
    wsb = 0 if ws is None else ws.numel() * ws.element_size()
    _check(lib().hyq_select_vertical(ctypes.byref(shape.c()), args[0], args[1], args[2], args[3],
                                     args[4], ctypes.c_size_t(wsb), _stream(stream)))


def hyq_quantize(shape: Shape, Q, K, V, idx, q_codes, q_scale, k_codes, k_scale, v_codes,
                 v_scale, kq_pos, stream=None):
    """Algorithm 2, Stages 1-2 (see include/hyq.h)."""
    torch = _torch()
    z = hyq_sizes_for(shape)
    if shape.bits_kv == 16:
        return
    dev, bf = _io(shape, Q, K, V)
    u8 = (torch.uint8, torch.int8)
    f32 = (torch.float32,)
    i32 = (torch.int32,)
    a = [
        _ptr(Q, "Q", Q.numel() * 2, bf, dev), _ptr(K, "K", K.numel() * 2, bf, dev),
        _ptr(V, "V", V.numel() * 2, bf, dev),
        _ptr(idx, "idx", z["idx_bytes"], i32, dev),
        _ptr(q_codes, "q_codes", z["q_codes_bytes"], u8, dev),
        _ptr(q_scale, "q_scale", z["q_scale_bytes"], f32, dev),
        _ptr(k_codes, "k_codes", z["k_codes_bytes"], u8, dev),
        _ptr(k_scale, "k_scale", z["kv_scale_bytes"], f32, dev),
        _ptr(v_codes, "v_codes", z["v_codes_bytes"], u8, dev),
        _ptr(v_scale, "v_scale", z["kv_scale_bytes"], f32, dev),
        _ptr(kq_pos, "kq_pos", z["kq_pos_bytes"], i32, dev),
    ]
    _check(lib().hyq_quantize(ctypes.byref(shape.c()), *a, _stream(stream)))


def hyq_attn_prefill(shape: Shape, Q, K, V, idx, q_codes, q_scale, k_codes, k_scale, v_codes,
                     v_scale, kq_pos, softmax_scale, out, out_dtype=0, stream=None):
    """Algorithm 2, Stage 3 / eq. (prefill_hybrid) (see include/hyq.h)."""
    torch = _torch()
    z = hyq_sizes_for(shape)
    dev, bf = _io(shape, Q, K, V)
    u8 = (torch.uint8, torch.int8)
    f32 = (torch.float32,)
    i32 = (torch.int32,)
    quant = shape.bits_kv != 16
    out_bytes = shape.B * shape.Hq * shape.L * shape.D * (4 if out_dtype == 0 else 2)
    odt = (torch.float32,) if out_dtype == 0 else (torch.bfloat16,)
    a = [
        _ptr(Q, "Q", Q.numel() * 2, bf, dev), _ptr(K, "K", K.numel() * 2, bf, dev),
        _ptr(V, "V", V.numel() * 2, bf, dev),
        _ptr(idx, "idx", z["idx_bytes"] if quant else 0, i32, dev, allow_none=not quant),
        _ptr(q_codes, "q_codes", z["q_codes_bytes"], u8, dev, allow_none=not quant),
        _ptr(q_scale, "q_scale", z["q_scale_bytes"], f32, dev, allow_none=not quant),
        _ptr(k_codes, "k_codes", z["k_codes_bytes"], u8, dev, allow_none=not quant),
        _ptr(k_scale, "k_scale", z["kv_scale_bytes"], f32, dev, allow_none=not quant),
        _ptr(v_codes, "v_codes", z["v_codes_bytes"], u8, dev, allow_none=not quant),
        _ptr(v_scale, "v_scale", z["kv_scale_bytes"], f32, dev, allow_none=not quant),
        _ptr(kq_pos, "kq_pos", z["kq_pos_bytes"], i32, dev, allow_none=not quant),
    ]
    o = _ptr(out, "out", out_bytes, odt, dev)
    _check(lib().hyq_attn_prefill(ctypes.byref(shape.c()), *a, ctypes.c_float(softmax_scale), o,
                                  ctypes.c_int32(out_dtype), _stream(stream)))


def hyq_prefill(shape: Shape, Q, K, V, idx, q_codes, q_scale, k_codes, k_scale, v_codes,
                v_scale, kq_pos, softmax_scale, out, out_dtype=0, ws=None, stream=None):
    """Algorithm 2 as one call: selection, quantization and attention
    (see include/hyq.h); the library checks all three before launching."""
    torch = _torch()
    z = hyq_sizes_for(shape)
    dev, bf = _io(shape, Q, K, V)
    u8 = (torch.uint8, torch.int8)
    f32 = (torch.float32,)
    i32 = (torch.int32,)
    quant = shape.bits_kv != 16
    sel = z["k"] > 0
    out_bytes = shape.B * shape.Hq * shape.L * shape.D * (4 if out_dtype == 0 else 2)
    odt = (torch.float32,) if out_dtype == 0 else (torch.bfloat16,)
    a = [
        _ptr(Q, "Q", Q.numel() * 2, bf, dev), _ptr(K, "K", K.numel() * 2, bf, dev),
        _ptr(V, "V", V.numel() * 2, bf, dev),
        _ptr(idx, "idx", z["idx_bytes"], i32, dev, allow_none=not sel),
        _ptr(q_codes, "q_codes", z["q_codes_bytes"], u8, dev, allow_none=not quant),
        _ptr(q_scale, "q_scale", z["q_scale_bytes"], f32, dev, allow_none=not quant),
        _ptr(k_codes, "k_codes", z["k_codes_bytes"], u8, dev, allow_none=not quant),
        _ptr(k_scale, "k_scale", z["kv_scale_bytes"], f32, dev, allow_none=not quant),
        _ptr(v_codes, "v_codes", z["v_codes_bytes"], u8, dev, allow_none=not quant),
        _ptr(v_scale, "v_scale", z["kv_scale_bytes"], f32, dev, allow_none=not quant),
        _ptr(kq_pos, "kq_pos", z["kq_pos_bytes"], i32, dev, allow_none=not quant),
    ]
    o = _ptr(out, "out", out_bytes, odt, dev)
    w = _ptr(ws, "ws", z["select_ws_bytes"], (torch.uint8, torch.int8, torch.float32), dev,
             allow_none=not sel)
    wsb = 0 if ws is None else ws.numel() * ws.element_size()
    _check(lib().hyq_prefill(ctypes.byref(shape.c()), *a, ctypes.c_float(softmax_scale), o,
                             ctypes.c_int32(out_dtype), w, ctypes.c_size_t(wsb), _stream(stream)))


# --------------------------------------------------------------------------
# convenience: buffers and the chained path
# --------------------------------------------------------------------------

def alloc_buffers(shape: Shape, device, out_dtype: int = 0) -> dict:
    """Every intermediate and output buffer of one prefill call (torch tensors)."""
    torch = _torch()
    z = hyq_sizes_for(shape)

    def u8(n):
        return torch.empty(max(n, 0), dtype=torch.uint8, device=device)

    B, Hq, Hkv, L, D = shape.B, shape.Hq, shape.Hkv, shape.L, shape.D
    return dict(
        sizes=z,
        idx=torch.empty((B, Hkv, z["k"]), dtype=torch.int32, device=device),
        ws=u8(z["select_ws_bytes"]),
        q_codes=torch.empty(z["q_codes_bytes"], dtype=torch.int8, device=device),
        q_scale=torch.empty(z["q_scale_bytes"] // 4, dtype=torch.float32, device=device),
        k_codes=u8(z["k_codes_bytes"]),
        k_scale=torch.empty(z["kv_scale_bytes"] // 4, dtype=torch.float32, device=device),
        v_codes=u8(z["v_codes_bytes"]),
        v_scale=torch.empty(z["kv_scale_bytes"] // 4, dtype=torch.float32, device=device),
        kq_pos=torch.empty(z["kq_pos_bytes"] // 4, dtype=torch.int32, device=device),
        out=torch.empty((B, Hq, L, D), dtype=torch.float32 if out_dtype == 0 else torch.bfloat16,
                        device=device),
    )


def prefill(shape: Shape, Q, K, V, bufs: dict, out_dtype: int = 0, stream=None,
            softmax_scale: float | None = None):
    """select -> quantize -> attention (Algorithm 2, one hyq_prefill call)
    into ``bufs['out']``."""
    scale = 1.0 / math.sqrt(shape.D) if softmax_scale is None else softmax_scale
    b = bufs
    hyq_prefill(shape, Q, K, V, b["idx"], b["q_codes"], b["q_scale"], b["k_codes"], b["k_scale"],
                b["v_codes"], b["v_scale"], b["kq_pos"], scale, b["out"], out_dtype, b["ws"],
                stream)
    return b["out"]


# --------------------------------------------------------------------------
# decode: Algorithm 4 (Freeze) and Algorithm 3 (decode attention)
# --------------------------------------------------------------------------

def hyq_dcache_init(shape: Shape, max_tokens: int):
    """Geometry of the decode cache of a prefill (see include/hyq.h):
    returns (ctypes hyq_dcache with NULL buffers, dict of buffer sizes)."""
    c = _DCache()
    z = _DCacheSizes()
    _check(lib().hyq_dcache_init(ctypes.byref(shape.c()), ctypes.c_int64(max_tokens),
                                 ctypes.byref(c), ctypes.byref(z)))
    return c, {n: getattr(z, n) for n in _DSIZES}


class DecodeCache:
    """A hybrid KV cache on one device: the ``hyq_dcache`` struct (geometry
    and host-side state) and the torch tensors that own its buffers."""

    def __init__(self, shape: Shape, max_tokens: int, device):
        torch = _torch()
        self.shape = shape
        self.c, self.sizes = hyq_dcache_init(shape, max_tokens)
        dev = torch.device(device)
        if dev.type == "cuda" and dev.index is None:
            dev = torch.device("cuda", torch.cuda.current_device())
        self.device = dev
        z = self.sizes

        def u8(n):
            return torch.zeros(max(n, 1), dtype=torch.uint8, device=self.device)

        self.bufs = {
            "k_codes": u8(z["k_codes_bytes"]), "v_codes": u8(z["v_codes_bytes"]),
            "k_scale": torch.zeros(max(z["k_scale_bytes"] // 4, 1), dtype=torch.float32,
                                   device=self.device),
            "v_scale": torch.zeros(max(z["v_scale_bytes"] // 4, 1), dtype=torch.float32,
                                   device=self.device),
            "q_pos": torch.zeros(max(z["q_pos_bytes"] // 4, 1), dtype=torch.int32,
                                 device=self.device),
            "fp_k": torch.zeros(max(z["fp_k_bytes"] // 2, 1), dtype=torch.bfloat16,
                                device=self.device),
            "fp_v": torch.zeros(max(z["fp_v_bytes"] // 2, 1), dtype=torch.bfloat16,
                                device=self.device),
            "vl_pos": torch.zeros(max(z["vl_pos_bytes"] // 4, 1), dtype=torch.int32,
                                  device=self.device),
        }
        for n in _DCACHE_PTRS:
            t = self.bufs[n]
            have = t.numel() * t.element_size()
            if have < z[n + "_bytes"]:
                raise ValueError(f"{n}: {have} bytes < {z[n + '_bytes']}")
            setattr(self.c, n, t.data_ptr())
        self.freeze_ws = u8(z["freeze_ws_bytes"])
        self.attn_ws = u8(z["attn_ws_bytes"])

    @property
    def state(self) -> dict:
        return {n: getattr(self.c, n) for n in ("n_merged", "ring_head", "n_staged", "t")}

    def geometry(self) -> dict:
        return {n: getattr(self.c, n) for n in _DCACHE_INTS}


def _decode_rows_ok(cache: DecodeCache, t, name, heads):
    torch = _torch()
    want = (cache.c.B, heads, cache.c.D)
    if tuple(t.shape) != want:
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {want}")
    return _ptr(t, name, t.numel() * 2, (torch.bfloat16,), cache.device)


def hyq_freeze(shape: Shape, Q, K, V, cache: DecodeCache, stream=None):
    """Algorithm 4: fill ``cache`` from the prefill's bf16 Q, K, V."""
    dev, bf = _io(shape, Q, K, V)
    if dev != cache.device:
        raise ValueError("Q, K, V must be on the cache's device")
    a = [_ptr(Q, "Q", Q.numel() * 2, bf, dev), _ptr(K, "K", K.numel() * 2, bf, dev),
         _ptr(V, "V", V.numel() * 2, bf, dev)]
    ws = cache.freeze_ws
    _check(lib().hyq_freeze(ctypes.byref(shape.c()), *a, ctypes.byref(cache.c),
                            ctypes.c_void_p(ws.data_ptr()),
                            ctypes.c_size_t(ws.numel()), _stream(stream)))


def hyq_decode_append(cache: DecodeCache, k_new, v_new, stream=None):
    """One decode step's K and V rows (bf16 [B, Hkv, D]) into the cache."""
    k = _decode_rows_ok(cache, k_new, "k_new", cache.c.Hkv)
    v = _decode_rows_ok(cache, v_new, "v_new", cache.c.Hkv)
    _check(lib().hyq_decode_append(ctypes.byref(cache.c), k, v, _stream(stream)))


def hyq_decode_attn(cache: DecodeCache, q, out, softmax_scale: float | None = None,
                    out_dtype: int = 0, stream=None):
    """Algorithm 3: out[b, h] = attention of q[b, h] (bf16 [B, Hq, D]) over the cache."""
    torch = _torch()
    qp = _decode_rows_ok(cache, q, "q", cache.c.Hq)
    scale = 1.0 / math.sqrt(cache.c.D) if softmax_scale is None else softmax_scale
    odt = (torch.float32,) if out_dtype == 0 else (torch.bfloat16,)
    nb = cache.c.B * cache.c.Hq * cache.c.D * (4 if out_dtype == 0 else 2)
    o = _ptr(out, "out", nb, odt, cache.device)
    ws = cache.attn_ws
    _check(lib().hyq_decode_attn(ctypes.byref(cache.c), qp, ctypes.c_float(scale), o,
                                 ctypes.c_int32(out_dtype), ctypes.c_void_p(ws.data_ptr()),
                                 ctypes.c_size_t(ws.numel()), _stream(stream)))


NOALLOC_SCRATCH_BYTES = 16 << 20   # HYQ_NOALLOC_SCRATCH_BYTES


def hyq_decode_attn_noalloc(cache: DecodeCache, q, out, softmax_scale: float | None = None,
                            out_dtype: int = 0, stream=None):
    """hyq_decode_attn with the library's own per-GPU scratch instead of a
    workspace (see include/hyq.h): allocates nothing."""
    torch = _torch()
    qp = _decode_rows_ok(cache, q, "q", cache.c.Hq)
    scale = 1.0 / math.sqrt(cache.c.D) if softmax_scale is None else softmax_scale
    odt = (torch.float32,) if out_dtype == 0 else (torch.bfloat16,)
    nb = cache.c.B * cache.c.Hq * cache.c.D * (4 if out_dtype == 0 else 2)
    o = _ptr(out, "out", nb, odt, cache.device)
    _check(lib().hyq_decode_attn_noalloc(ctypes.byref(cache.c), qp, ctypes.c_float(scale), o,
                                         ctypes.c_int32(out_dtype), _stream(stream)))
