"""EntQuant inference-time decoding on MI355X: thin ctypes binding of libeq.

Every function here has the name of the C entry point it wraps (include/eq.h,
include/eq_encode.h) and only marshals arguments: torch supplies device memory
and streams, all decoding runs in libeq's gfx950 kernels.  There is no CPU
fallback: if libeq.so is missing, loading fails loudly.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from ._build import LIB as _LIB_PATH
from ._build import build as _build_lib

EQ_OK, EQ_EINVAL, EQ_EFORMAT, EQ_EHIP, EQ_ECORRUPT, EQ_ESCRATCH = 0, -1, -2, -3, -4, -5
NOALLOC_SCRATCH_BYTES = 32 << 20
FMT_E4M3, FMT_INT8 = 1, 2  # base formats of the codes (container field base_format)

_lib = None
_vp = ctypes.c_void_p


class EqError(RuntimeError):
    def __init__(self, fn: str, code: int):
        super().__init__(f"{fn}: {eq_strerror(code)} ({code})")
        self.code = code


class eq_layer(ctypes.Structure):
    _fields_ = [("rows", ctypes.c_uint32), ("cols", ctypes.c_uint32),
                ("chunk_syms", ctypes.c_uint32), ("n_chunks", ctypes.c_uint32),
                ("lanes", ctypes.c_uint32), ("prob_bits", ctypes.c_uint32),
                ("n_syms", ctypes.c_uint32), ("base_format", ctypes.c_uint32),
                ("total_words", ctypes.c_uint64), ("padded_words", ctypes.c_uint64),
                ("scale", _vp), ("sym", _vp), ("freq", _vp), ("chunk_off", _vp),
                ("chunk_state", _vp), ("words", _vp), ("lut", _vp), ("status", _vp),
                ("version", ctypes.c_uint32), ("tile_cols", ctypes.c_uint32),
                ("n_quads", ctypes.c_uint32), ("n_pairs", ctypes.c_uint32),
                ("n_singles", ctypes.c_uint32), ("row_order", _vp)]


class eqe_params(ctypes.Structure):
    _fields_ = [("prob_bits", ctypes.c_uint32), ("chunk_syms", ctypes.c_uint32),
                ("lanes", ctypes.c_uint32), ("threads", ctypes.c_uint32),
                ("seed", ctypes.c_uint64), ("target_bits", ctypes.c_float),
                ("base_format", ctypes.c_uint32)]


class eqe_params2(ctypes.Structure):
    _fields_ = [("res_bits", ctypes.c_uint32), ("tile_rows", ctypes.c_uint32),
                ("tile_cols", ctypes.c_uint32), ("threads", ctypes.c_uint32),
                ("seed", ctypes.c_uint64), ("target_bits", ctypes.c_float),
                ("base_format", ctypes.c_uint32), ("row_order", ctypes.c_uint32)]


class eqe_rd_params(ctypes.Structure):
    _fields_ = [("lambda_", ctypes.c_double), ("lr", ctypes.c_double),
                ("iters", ctypes.c_uint32), ("history", ctypes.c_uint32),
                ("threads", ctypes.c_uint32), ("base_format", ctypes.c_uint32)]


# name -> (restype, argtypes): every symbol the public headers declare
SIGNATURES = {
    "eq_lut_bytes": (ctypes.c_size_t, []),
    "eq_layer_init": (ctypes.c_int, [ctypes.POINTER(eq_layer), _vp, ctypes.c_uint64, _vp, _vp,
                                     _vp]),
    "eq_layer_prepare": (ctypes.c_int, [ctypes.POINTER(eq_layer), _vp]),
    "eq_decode_codes": (ctypes.c_int, [ctypes.POINTER(eq_layer), _vp, _vp]),
    "eq_decode_bf16": (ctypes.c_int, [ctypes.POINTER(eq_layer), _vp, _vp]),
    "eq_gemv_workspace_bytes": (ctypes.c_size_t, [ctypes.POINTER(eq_layer), ctypes.c_uint32]),
    "eq_decode_gemv": (ctypes.c_int, [ctypes.POINTER(eq_layer), _vp, ctypes.c_uint32, _vp, _vp,
                                      _vp, ctypes.c_size_t, _vp]),
    "eq_decode_gemv_noalloc": (ctypes.c_int, [ctypes.POINTER(eq_layer), _vp, ctypes.c_uint32, _vp,
                                              _vp, _vp]),
    "eq_decode_bf16_multi": (ctypes.c_int, [_vp, _vp, ctypes.c_uint32, _vp]),
    "eq_decode_codes_multi": (ctypes.c_int, [_vp, _vp, ctypes.c_uint32, _vp]),
    "eq_gemv_multi_workspace_bytes": (ctypes.c_size_t, [_vp, ctypes.c_uint32, ctypes.c_uint32]),
    "eq_decode_gemv_multi": (ctypes.c_int, [_vp, ctypes.c_uint32, _vp, ctypes.c_uint32, _vp, _vp,
                                            _vp, ctypes.c_size_t, _vp]),
    "eq_gemm_codes_workspace_bytes": (ctypes.c_size_t, [ctypes.POINTER(eq_layer), ctypes.c_uint32]),
    "eq_gemm_workspace_bytes": (ctypes.c_size_t, [ctypes.POINTER(eq_layer), ctypes.c_uint32]),
    "eq_gemm_codes": (ctypes.c_int, [ctypes.POINTER(eq_layer), _vp, _vp, ctypes.c_uint32, _vp, _vp,
                                     _vp, ctypes.c_size_t, _vp]),
    "eq_decode_gemm": (ctypes.c_int, [ctypes.POINTER(eq_layer), _vp, ctypes.c_uint32, _vp, _vp,
                                      _vp, ctypes.c_size_t, _vp]),
    "eq_get_status": (ctypes.c_int, [ctypes.POINTER(eq_layer), _vp]),
    "eq_strerror": (ctypes.c_char_p, [ctypes.c_int]),
    "eqe_alpha_search": (ctypes.c_float, [_vp, ctypes.c_uint32, ctypes.c_uint32, ctypes.c_double,
                                          ctypes.c_uint32, ctypes.c_uint32, ctypes.c_uint32,
                                          ctypes.POINTER(ctypes.c_double)]),
    "eqe_encode": (ctypes.c_int, [_vp, ctypes.c_uint32, ctypes.c_uint32, ctypes.c_float,
                                  ctypes.POINTER(eqe_params), ctypes.POINTER(ctypes.c_void_p),
                                  ctypes.POINTER(ctypes.c_uint64)]),
    "eqe_encode2": (ctypes.c_int, [_vp, ctypes.c_uint32, ctypes.c_uint32, ctypes.c_float, _vp,
                                   ctypes.POINTER(eqe_params2), ctypes.POINTER(ctypes.c_void_p),
                                   ctypes.POINTER(ctypes.c_uint64)]),
    "eqe_encode_scaled": (ctypes.c_int, [_vp, ctypes.c_uint32, ctypes.c_uint32, _vp,
                                         ctypes.POINTER(eqe_params),
                                         ctypes.POINTER(ctypes.c_void_p),
                                         ctypes.POINTER(ctypes.c_uint64)]),
    "eqe_rd_objective": (ctypes.c_double, [_vp, ctypes.c_uint32, ctypes.c_uint32, ctypes.c_uint32,
                                           ctypes.c_double, _vp, ctypes.c_uint32, _vp, _vp]),
    "eqe_rd_scales": (ctypes.c_int, [_vp, ctypes.c_uint32, ctypes.c_uint32,
                                     ctypes.POINTER(eqe_rd_params), _vp, _vp, _vp]),
    "eqe_rd_lambda_search": (ctypes.c_int, [_vp, ctypes.c_uint32, ctypes.c_uint32,
                                            ctypes.c_double, ctypes.c_uint32,
                                            ctypes.POINTER(eqe_rd_params),
                                            ctypes.POINTER(ctypes.c_double),
                                            ctypes.POINTER(ctypes.c_double)]),
    "eqe_free": (None, [_vp]),
}


def build() -> str:
    """Compile libeq.so (gfx950) in place and reload it."""
    global _lib
    path = _build_lib()
    _lib = None
    return path


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(f"{_LIB_PATH} is not built; run __graft_entry__.build() first")
        L = ctypes.CDLL(_LIB_PATH)
        for name, (res, args) in SIGNATURES.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def _check(fn: str, rc: int) -> None:
    if rc != EQ_OK:
        raise EqError(fn, rc)


def _stream(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _dptr(t, dtype=None, numel=None):
    """Device pointer of a contiguous CUDA tensor, with optional checks."""
    if t is None:
        return None
    if not t.is_cuda or not t.is_contiguous():
        raise ValueError("expected a contiguous device tensor")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"expected dtype {dtype}, got {t.dtype}")
    if numel is not None and t.numel() < numel:
        raise ValueError(f"tensor too small: {t.numel()} < {numel}")
    return ctypes.c_void_p(t.data_ptr())


# ---------------------------------------------------------------- decode ABI
def eq_strerror(code: int) -> str:
    return lib().eq_strerror(code).decode()


def eq_lut_bytes() -> int:
    return lib().eq_lut_bytes()


def eq_layer_init(host_blob: np.ndarray, dev_blob, dev_lut, dev_status) -> eq_layer:
    host_blob = np.ascontiguousarray(host_blob, dtype=np.uint8)
    L = eq_layer()
    rc = lib().eq_layer_init(ctypes.byref(L), host_blob.ctypes.data, host_blob.size,
                             _dptr(dev_blob, numel=host_blob.size),
                             _dptr(dev_lut, numel=None), _dptr(dev_status))
    _check("eq_layer_init", rc)
    return L


def eq_layer_prepare(L, stream=None) -> None:
    _check("eq_layer_prepare", lib().eq_layer_prepare(ctypes.byref(_raw(L)), _stream(stream)))


def eq_decode_codes(L, codes, stream=None) -> None:
    import torch
    r = _raw(L)
    p = _dptr(codes, torch.uint8, r.rows * r.cols)
    _check("eq_decode_codes", lib().eq_decode_codes(ctypes.byref(r), p, _stream(stream)))


def eq_decode_bf16(L, w, stream=None) -> None:
    import torch
    r = _raw(L)
    if w.dtype not in (torch.bfloat16, torch.int16, torch.uint16):
        raise ValueError("w must hold 16-bit BF16 patterns")
    p = _dptr(w, None, r.rows * r.cols)
    _check("eq_decode_bf16", lib().eq_decode_bf16(ctypes.byref(r), p, _stream(stream)))


def eq_gemv_workspace_bytes(L, B: int) -> int:
    return lib().eq_gemv_workspace_bytes(ctypes.byref(_raw(L)), B)


def eq_decode_gemv(L, x, B: int, bias, y, ws, stream=None) -> None:
    import torch
    r = _raw(L)
    if x.dtype not in (torch.bfloat16, torch.int16, torch.uint16):
        raise ValueError("x must hold 16-bit BF16 patterns")
    px = _dptr(x, None, B * r.cols)
    pb = _dptr(bias, None, r.rows) if bias is not None else None
    py = _dptr(y, torch.float32, B * r.rows)
    pw = _dptr(ws)
    nbytes = ws.numel() * ws.element_size()
    _check("eq_decode_gemv", lib().eq_decode_gemv(ctypes.byref(r), px, B, pb, py, pw, nbytes,
                                                  _stream(stream)))


def eq_decode_gemv_noalloc(L, x, B: int, bias, y, stream=None) -> None:
    """eq_decode_gemv with the library's static per-device scratch as workspace."""
    import torch
    r = _raw(L)
    if x.dtype not in (torch.bfloat16, torch.int16, torch.uint16):
        raise ValueError("x must hold 16-bit BF16 patterns")
    px = _dptr(x, None, B * r.cols)
    pb = _dptr(bias, None, r.rows) if bias is not None else None
    py = _dptr(y, torch.float32, B * r.rows)
    _check("eq_decode_gemv_noalloc",
           lib().eq_decode_gemv_noalloc(ctypes.byref(r), px, B, pb, py, _stream(stream)))


def _layer_array(layers):
    """Host array of eq_layer pointers (the views must outlive the call)."""
    raws = [_raw(L) for L in layers]
    arr = (ctypes.POINTER(eq_layer) * len(raws))(*[ctypes.pointer(r) for r in raws])
    return arr, raws


def _ptr_array(ptrs):
    return (ctypes.c_void_p * len(ptrs))(*[p.value if p is not None else None for p in ptrs])


def eq_decode_bf16_multi(layers, outs, stream=None) -> None:
    """Block-wise decode of several layers: layer i to outs[i]."""
    import torch
    if len(layers) != len(outs):
        raise ValueError("one output per layer")
    arr, raws = _layer_array(layers)
    for w in outs:
        if w.dtype not in (torch.bfloat16, torch.int16, torch.uint16):
            raise ValueError("outputs must hold 16-bit BF16 patterns")
    ptrs = _ptr_array([_dptr(w, None, r.rows * r.cols) for w, r in zip(outs, raws)])
    _check("eq_decode_bf16_multi",
           lib().eq_decode_bf16_multi(arr, ptrs, len(raws), _stream(stream)))


def eq_decode_codes_multi(layers, outs, stream=None) -> None:
    """Block-wise decode of several layers to one-byte codes: layer i to outs[i]."""
    import torch
    if len(layers) != len(outs):
        raise ValueError("one output per layer")
    arr, raws = _layer_array(layers)
    ptrs = _ptr_array([_dptr(c, torch.uint8, r.rows * r.cols) for c, r in zip(outs, raws)])
    _check("eq_decode_codes_multi",
           lib().eq_decode_codes_multi(arr, ptrs, len(raws), _stream(stream)))


def eq_gemv_multi_workspace_bytes(layers, B: int) -> int:
    arr, raws = _layer_array(layers)
    return lib().eq_gemv_multi_workspace_bytes(arr, len(raws), B)


def eq_decode_gemv_multi(layers, x, B: int, biases, ys, ws, stream=None) -> None:
    """Fused decode-GEMV of several layers sharing the input x: ys[i] for
    layer i; biases is None or a list (entries may be None)."""
    import torch
    if len(layers) != len(ys) or (biases is not None and len(biases) != len(layers)):
        raise ValueError("one output (and bias) per layer")
    arr, raws = _layer_array(layers)
    if x.dtype not in (torch.bfloat16, torch.int16, torch.uint16):
        raise ValueError("x must hold 16-bit BF16 patterns")
    px = _dptr(x, None, B * raws[0].cols)
    py = _ptr_array([_dptr(y, torch.float32, B * r.rows) for y, r in zip(ys, raws)])
    pb = None
    if biases is not None:
        pb = _ptr_array([_dptr(b, None, r.rows) if b is not None else None
                         for b, r in zip(biases, raws)])
    nbytes = ws.numel() * ws.element_size()
    _check("eq_decode_gemv_multi",
           lib().eq_decode_gemv_multi(arr, len(raws), px, B, pb, py, _dptr(ws), nbytes,
                                      _stream(stream)))


def multi_workspace(layers, B: int):
    """A device workspace for eq_decode_gemv_multi over `layers`."""
    import torch
    return torch.empty(eq_gemv_multi_workspace_bytes(layers, B), dtype=torch.uint8,
                       device=layers[0].dev_blob.device)


def eq_gemm_codes_workspace_bytes(L, B: int) -> int:
    return lib().eq_gemm_codes_workspace_bytes(ctypes.byref(_raw(L)), B)


def eq_gemm_workspace_bytes(L, B: int) -> int:
    return lib().eq_gemm_workspace_bytes(ctypes.byref(_raw(L)), B)


def eq_gemm_codes(L, codes, x, B: int, bias, y, ws=None, stream=None) -> None:
    """Prefill GEMM from decoded codes: y[B][M] = x[B][N] W_hat^T + bias; ws:
    eq_gemm_codes_workspace_bytes(L, B) bytes (None when that is 0)."""
    import torch
    r = _raw(L)
    if x.dtype not in (torch.bfloat16, torch.int16, torch.uint16):
        raise ValueError("x must hold 16-bit BF16 patterns")
    pc = _dptr(codes, torch.uint8, r.rows * r.cols)
    px = _dptr(x, None, B * r.cols)
    pb = _dptr(bias, None, r.rows) if bias is not None else None
    py = _dptr(y, torch.float32, B * r.rows)
    pw = _dptr(ws) if ws is not None else None
    nbytes = ws.numel() * ws.element_size() if ws is not None else 0
    _check("eq_gemm_codes", lib().eq_gemm_codes(ctypes.byref(r), pc, px, B, pb, py, pw, nbytes,
                                                _stream(stream)))


def eq_decode_gemm(L, x, B: int, bias, y, ws, stream=None) -> None:
    """Prefill: decode the codes into ws, then the MFMA GEMM."""
    import torch
    r = _raw(L)
    if x.dtype not in (torch.bfloat16, torch.int16, torch.uint16):
        raise ValueError("x must hold 16-bit BF16 patterns")
    px = _dptr(x, None, B * r.cols)
    pb = _dptr(bias, None, r.rows) if bias is not None else None
    py = _dptr(y, torch.float32, B * r.rows)
    nbytes = ws.numel() * ws.element_size()
    _check("eq_decode_gemm", lib().eq_decode_gemm(ctypes.byref(r), px, B, pb, py, _dptr(ws),
                                                  nbytes, _stream(stream)))


def eq_get_status(L, stream=None) -> int:
    return lib().eq_get_status(ctypes.byref(_raw(L)), _stream(stream))


# ---------------------------------------------------------------- encoder ABI
def eqe_alpha_search(w: np.ndarray, target_bits: float, sample_rows: int = 0,
                     threads: int = 0, base_format: int = FMT_E4M3):
    w = np.ascontiguousarray(w, dtype=np.uint16)
    h = ctypes.c_double()
    a = lib().eqe_alpha_search(w.ctypes.data, w.shape[0], w.shape[1], target_bits, sample_rows,
                               threads, base_format, ctypes.byref(h))
    if a <= 0:
        raise EqError("eqe_alpha_search", EQ_EINVAL)
    return a, h.value


def eqe_encode(w: np.ndarray, alpha: float, *, prob_bits: int = 12, chunk_syms: int,
               lanes: int, threads: int = 0, seed: int = 0, target_bits: float = 0.0,
               base_format: int = FMT_E4M3, scale_bf16: np.ndarray | None = None) -> np.ndarray:
    """eqe_encode, or eqe_encode_scaled when scale_bf16 (uint16[M]) is given."""
    w = np.ascontiguousarray(w, dtype=np.uint16)
    prm = eqe_params(prob_bits, chunk_syms, lanes, threads, seed, target_bits, base_format)
    p = ctypes.c_void_p()
    nb = ctypes.c_uint64()
    if scale_bf16 is None:
        rc = lib().eqe_encode(w.ctypes.data, w.shape[0], w.shape[1], alpha, ctypes.byref(prm),
                              ctypes.byref(p), ctypes.byref(nb))
        _check("eqe_encode", rc)
    else:
        sc = np.ascontiguousarray(scale_bf16, dtype=np.uint16)
        if sc.size != w.shape[0]:
            raise ValueError("one scale per row")
        rc = lib().eqe_encode_scaled(w.ctypes.data, w.shape[0], w.shape[1], sc.ctypes.data,
                                     ctypes.byref(prm), ctypes.byref(p), ctypes.byref(nb))
        _check("eqe_encode_scaled", rc)
    try:
        out = np.empty(nb.value, dtype=np.uint8)
        ctypes.memmove(out.ctypes.data, p.value, nb.value)
    finally:
        lib().eqe_free(p)
    return out


def eqe_encode2(w: np.ndarray, alpha: float, *, tile_rows: int, tile_cols: int,
                res_bits: int = 12, threads: int = 0, seed: int = 0, target_bits: float = 0.0,
                base_format: int = FMT_E4M3, scale_bf16: np.ndarray | None = None,
                row_order: bool = False) -> np.ndarray:
    """A version-2 container (tile-ordered chunks, phrase alphabet); with
    row_order, the tiles are cut over the rows sorted by phrase count."""
    w = np.ascontiguousarray(w, dtype=np.uint16)
    prm = eqe_params2(res_bits, tile_rows, tile_cols, threads, seed, target_bits, base_format,
                      int(bool(row_order)))
    sc = None
    if scale_bf16 is not None:
        sc = np.ascontiguousarray(scale_bf16, dtype=np.uint16)
        if sc.size != w.shape[0]:
            raise ValueError("one scale per row")
    p = ctypes.c_void_p()
    nb = ctypes.c_uint64()
    rc = lib().eqe_encode2(w.ctypes.data, w.shape[0], w.shape[1], alpha,
                           None if sc is None else sc.ctypes.data, ctypes.byref(prm),
                           ctypes.byref(p), ctypes.byref(nb))
    _check("eqe_encode2", rc)
    try:
        out = np.empty(nb.value, dtype=np.uint8)
        ctypes.memmove(out.ctypes.data, p.value, nb.value)
    finally:
        lib().eqe_free(p)
    return out


def _rd_params(lam, iters, history, lr, threads, base_format):
    return eqe_rd_params(lam, lr, iters, history, threads, base_format)


def eqe_rd_objective(w: np.ndarray, scale: np.ndarray, lam: float, base_format: int = FMT_E4M3,
                     threads: int = 0):
    """(F, straight-through gradient, distortion term) at the given scales."""
    w = np.ascontiguousarray(w, dtype=np.uint16)
    sc = np.ascontiguousarray(scale, dtype=np.float64)
    g = np.empty(w.shape[0], dtype=np.float64)
    d = ctypes.c_double()
    f = lib().eqe_rd_objective(w.ctypes.data, w.shape[0], w.shape[1], base_format, lam,
                               sc.ctypes.data, threads, g.ctypes.data, ctypes.byref(d))
    if np.isnan(f):
        raise EqError("eqe_rd_objective", EQ_EINVAL)
    return f, g, d.value


def eqe_rd_scales(w: np.ndarray, lam: float, *, iters: int = 0, history: int = 0, lr: float = 0.0,
                  threads: int = 0, base_format: int = FMT_E4M3):
    """(scales as float64, scales as BF16 bit patterns, lowest F)."""
    w = np.ascontiguousarray(w, dtype=np.uint16)
    M = w.shape[0]
    prm = _rd_params(lam, iters, history, lr, threads, base_format)
    s64 = np.empty(M, dtype=np.float64)
    s16 = np.empty(M, dtype=np.uint16)
    f = ctypes.c_double()
    _check("eqe_rd_scales", lib().eqe_rd_scales(w.ctypes.data, M, w.shape[1], ctypes.byref(prm),
                                                 s64.ctypes.data, s16.ctypes.data, ctypes.byref(f)))
    return s64, s16, f.value


def eqe_rd_lambda_search(w: np.ndarray, target_bits: float, sample_rows: int = 0, *,
                         iters: int = 0, history: int = 0, lr: float = 0.0, threads: int = 0,
                         base_format: int = FMT_E4M3):
    """(lambda, entropy over the rows searched)."""
    w = np.ascontiguousarray(w, dtype=np.uint16)
    prm = _rd_params(0.0, iters, history, lr, threads, base_format)
    lam, h = ctypes.c_double(), ctypes.c_double()
    _check("eqe_rd_lambda_search",
           lib().eqe_rd_lambda_search(w.ctypes.data, w.shape[0], w.shape[1], target_bits,
                                      sample_rows, ctypes.byref(prm), ctypes.byref(lam),
                                      ctypes.byref(h)))
    return lam.value, h.value


# ---------------------------------------------------------------- layer object
class Layer:
    """One compressed layer resident on the device: the container bytes, the
    decode-table scratch and the status word, with its validated eq_layer."""

    def __init__(self, blob: np.ndarray, device="cuda", stream=None):
        import torch
        self.blob = np.ascontiguousarray(blob, dtype=np.uint8)
        self.dev_blob = torch.from_numpy(self.blob).to(device)
        self.lut = torch.empty(eq_lut_bytes(), dtype=torch.uint8, device=device)
        self.status = torch.zeros(1, dtype=torch.int32, device=device)
        self.raw = eq_layer_init(self.blob, self.dev_blob, self.lut, self.status)
        eq_layer_prepare(self, stream)

    @property
    def rows(self) -> int:
        return self.raw.rows

    @property
    def cols(self) -> int:
        return self.raw.cols

    @property
    def base_format(self) -> int:
        return self.raw.base_format

    def workspace(self, B: int):
        import torch
        return torch.empty(eq_gemv_workspace_bytes(self, B), dtype=torch.uint8,
                           device=self.dev_blob.device)

    def gemm_workspace(self, B: int):
        """Workspace of eq_decode_gemm for B tokens."""
        import torch
        return torch.empty(eq_gemm_workspace_bytes(self, B), dtype=torch.uint8,
                           device=self.dev_blob.device)


def _raw(L) -> eq_layer:
    return L.raw if isinstance(L, Layer) else L


def smoke() -> None:
    """One small decode (codes, BF16), fused GEMV (B = 3) and prefill (24
    tokens) on cuda:0, and the same codes in a version-2 container (codes and
    the batch-1 GEMV), checked against the CPU oracle."""
    import sys

    import torch

    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    if root not in sys.path:
        sys.path.insert(0, root)
    import oracle
    import synth
    from synth.configs import small_spec

    spec = small_spec(96, 320, bits=2.5, chunk=1024, lanes=64, seed=77)
    w = synth.weights(spec)
    alpha, _ = eqe_alpha_search(w, spec.target_bits)
    blob = eqe_encode(w, alpha, chunk_syms=spec.chunk_syms, lanes=spec.lanes)
    dev = torch.device("cuda:0")
    L = Layer(blob, dev)
    codes = torch.empty(spec.params, dtype=torch.uint8, device=dev)
    eq_decode_codes(L, codes)
    wb = torch.empty(spec.params, dtype=torch.int16, device=dev)
    eq_decode_bf16(L, wb)
    B = 3
    x = torch.from_numpy(synth.activations(spec, B).view(np.int16)).to(dev)
    y = torch.empty(B, spec.rows, dtype=torch.float32, device=dev)
    ws = L.workspace(B)
    eq_decode_gemv(L, x, B, None, y, ws)
    _check("eq_get_status", eq_get_status(L))

    rc, q_ref = oracle.container_decode(blob)
    assert rc == oracle.OK
    assert np.array_equal(codes.cpu().numpy().reshape(q_ref.shape), q_ref), "codes differ"
    w_ref = oracle.dequant(q_ref, oracle.container_scales(blob))
    assert np.array_equal(wb.cpu().numpy().view(np.uint16).reshape(w_ref.shape), w_ref), \
        "bf16 differs"
    y_ref = oracle.gemv(w_ref, synth.activations(spec, B))
    err = np.abs(y.cpu().numpy() - y_ref).max(axis=1) / np.abs(y_ref).max(axis=1)
    assert (err <= 1e-2).all(), f"gemv error {err}"
    # prefill: decode to codes + matrix-core GEMM over 24 tokens
    T = 24
    xt_bits = np.stack([synth.vector(spec.seed, 40 + t, spec.cols) for t in range(T)])
    xt = torch.from_numpy(xt_bits.view(np.int16)).to(dev)
    yt = torch.empty(T, spec.rows, dtype=torch.float32, device=dev)
    eq_decode_gemm(L, xt, T, None, yt, L.gemm_workspace(T))
    _check("eq_get_status", eq_get_status(L))
    yt_ref = oracle.gemv(w_ref, xt_bits)
    err_t = np.abs(yt.cpu().numpy() - yt_ref).max(axis=1) / np.abs(yt_ref).max(axis=1)
    assert (err_t <= 1e-2).all(), f"prefill error {err_t}"
    # version 2: tiles of 64 x 64, codes and the batch-1 GEMV
    blob2 = eqe_encode2(w, alpha, tile_rows=64, tile_cols=64)
    L2 = Layer(blob2, dev)
    codes2 = torch.empty(spec.params, dtype=torch.uint8, device=dev)
    eq_decode_codes(L2, codes2)
    x1 = x[:1].contiguous()
    y1 = torch.empty(1, spec.rows, dtype=torch.float32, device=dev)
    eq_decode_gemv(L2, x1, 1, None, y1, L2.workspace(1))
    _check("eq_get_status", eq_get_status(L2))
    rc, q2_ref = oracle.container2_decode(blob2)
    assert rc == oracle.OK
    assert np.array_equal(codes2.cpu().numpy().reshape(q2_ref.shape), q2_ref), "v2 codes differ"
    w2_ref = oracle.dequant(q2_ref, oracle.container_scales(blob2))
    y1_ref = oracle.gemv(w2_ref, synth.activations(spec, B)[:1])
    err2 = np.abs(y1.cpu().numpy() - y1_ref).max() / np.abs(y1_ref).max()
    assert err2 <= 1e-2, f"version-2 gemv error {err2}"
    print(f"smoke ok: codes/bf16 bit-exact, gemv max rel err {err.max():.2e}, "
          f"prefill max rel err {err_t.max():.2e}; version 2: codes bit-exact, "
          f"gemv rel err {err2:.2e}")
