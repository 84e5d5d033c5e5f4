"""EntQuant CPU oracle -- TEST INFRASTRUCTURE ONLY.

A plain, slow C implementation (``eq_oracle.c``) of what the decode path
computes, with ctypes wrappers.  Only the test suite, the package smoke check
and the CPU-baseline leg of the benchmark may import this module; the product
library never uses it.  ``build()`` compiles ``liboracle.so`` with gcc.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

OK, EINVAL, EFORMAT, ECORRUPT, ENOMEM = 0, -1, -2, -4, -5
E4M3, INT8 = 1, 2  # base formats (container header field base_format)

_u8p = ctypes.c_void_p
_vp = ctypes.c_void_p


class Info(ctypes.Structure):
    _fields_ = [(n, ctypes.c_uint32) for n in
                ("rows", "cols", "chunk_syms", "n_chunks", "lanes", "prob_bits", "n_syms",
                 "base_format")] + \
               [(n, ctypes.c_uint64) for n in
                ("total_words", "padded_words", "seed", "file_bytes")] + \
               [(n, ctypes.c_float) for n in ("alpha", "target_bits", "entropy_bits")] + \
               [(n, ctypes.c_uint64) for n in
                ("off_scale", "off_sym", "off_freq", "off_chunk_off", "off_chunk_state",
                 "off_words")]


class Info2(ctypes.Structure):
    _fields_ = [(n, ctypes.c_uint32) for n in
                ("rows", "cols", "chunk_syms", "n_chunks", "lanes", "prob_bits", "n_syms",
                 "base_format", "tile_cols", "n_quads", "n_pairs", "n_singles", "tau")] + \
               [(n, ctypes.c_uint64) for n in
                ("total_words", "padded_words", "seed", "file_bytes")] + \
               [(n, ctypes.c_float) for n in ("alpha", "target_bits", "entropy_bits")] + \
               [(n, ctypes.c_uint64) for n in
                ("off_scale", "off_phr", "off_freq", "off_chunk_off", "off_chunk_state",
                 "off_words")] + \
               [("flags", ctypes.c_uint32), ("off_order", ctypes.c_uint64)]


def build() -> str:
    """Compile liboracle.so (always recompiles)."""
    cmd = ["gcc", "-O2", "-std=c99", "-D_GNU_SOURCE", "-fPIC", "-shared", "-ffp-contract=off",
           "-fno-fast-math", os.path.join(_HERE, "eq_oracle.c"), os.path.join(_HERE, "eq_phrase.c"),
           "-o", _LIB_PATH + ".tmp", "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(_LIB_PATH + ".tmp", _LIB_PATH)
    return _LIB_PATH


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build()
        L = ctypes.CDLL(_LIB_PATH)
        sig = {
            "or_e4m3_value": (ctypes.c_double, [ctypes.c_uint8]),
            "or_e4m3_round": (ctypes.c_uint8, [ctypes.c_float]),
            "or_int8_value": (ctypes.c_double, [ctypes.c_uint8]),
            "or_int8_round": (ctypes.c_uint8, [ctypes.c_float]),
            "or_qmax": (ctypes.c_double, [ctypes.c_uint32]),
            "or_code_value": (ctypes.c_double, [ctypes.c_uint32, ctypes.c_uint8]),
            "or_bf16_value": (ctypes.c_double, [ctypes.c_uint16]),
            "or_bf16_round": (ctypes.c_uint16, [ctypes.c_double]),
            "or_entropy_counts": (ctypes.c_double, [_vp, ctypes.c_uint32]),
            "or_entropy_codes": (ctypes.c_double, [_vp, ctypes.c_uint64]),
            "or_sparsity_entropy": (ctypes.c_double, [ctypes.c_double, ctypes.c_double]),
            "or_row_scales": (None, [_vp, ctypes.c_uint32, ctypes.c_uint32, ctypes.c_float,
                                     ctypes.c_uint32, _vp]),
            "or_quantize": (None, [_vp, ctypes.c_uint32, ctypes.c_uint32, _vp, ctypes.c_uint32,
                                   _vp]),
            "or_dequant": (None, [_vp, ctypes.c_uint32, ctypes.c_uint32, _vp, ctypes.c_uint32,
                                  _vp]),
            "or_alpha_search": (ctypes.c_float, [_vp, ctypes.c_uint32, ctypes.c_uint32,
                                                 ctypes.c_double, ctypes.c_uint32,
                                                 ctypes.POINTER(ctypes.c_double)]),
            "or_freq_table": (ctypes.c_int, [_vp, ctypes.c_uint32, _vp, _vp,
                                             ctypes.POINTER(ctypes.c_uint32)]),
            "or_rans_encode": (ctypes.c_int, [_vp, ctypes.c_uint32, ctypes.c_uint32,
                                              ctypes.c_uint32, _vp, _vp, ctypes.c_uint32, _vp,
                                              ctypes.c_uint32, ctypes.POINTER(ctypes.c_uint32),
                                              _vp]),
            "or_rans_decode": (ctypes.c_int, [_vp, ctypes.c_uint32, _vp, ctypes.c_uint32,
                                              ctypes.c_uint32, ctypes.c_uint32, _vp, _vp,
                                              ctypes.c_uint32, _vp]),
            "or_container_build": (ctypes.c_int, [_vp, ctypes.c_uint32, ctypes.c_uint32,
                                                  ctypes.c_float, ctypes.c_uint32,
                                                  ctypes.c_uint32, ctypes.c_uint32,
                                                  ctypes.c_uint32,
                                                  ctypes.c_uint64, ctypes.c_float,
                                                  ctypes.POINTER(ctypes.c_void_p),
                                                  ctypes.POINTER(ctypes.c_uint64)]),
            "or_free": (None, [_vp]),
            "or_container_build_scaled": (ctypes.c_int, [_vp, ctypes.c_uint32, ctypes.c_uint32,
                                                         _vp, ctypes.c_uint32, ctypes.c_uint32,
                                                         ctypes.c_uint32, ctypes.c_uint32,
                                                         ctypes.c_uint64, ctypes.c_float,
                                                         ctypes.POINTER(ctypes.c_void_p),
                                                         ctypes.POINTER(ctypes.c_uint64)]),
            "or_rd_objective": (ctypes.c_double, [_vp, ctypes.c_uint32, ctypes.c_uint32,
                                                  ctypes.c_uint32, ctypes.c_double, _vp, _vp,
                                                  _vp]),
            "or_rd_scales": (ctypes.c_int, [_vp, ctypes.c_uint32, ctypes.c_uint32,
                                            ctypes.c_uint32, ctypes.c_double, ctypes.c_uint32,
                                            ctypes.c_uint32, ctypes.c_double, _vp, _vp]),
            "or_lbfgs_quadratic": (ctypes.c_int, [ctypes.c_uint32, _vp, ctypes.c_double, _vp,
                                                  ctypes.c_uint32, ctypes.c_uint32,
                                                  ctypes.c_double, _vp, _vp]),
            "or_container_info": (ctypes.c_int, [_vp, ctypes.c_uint64, ctypes.POINTER(Info)]),
            "or_container_decode_chunk": (ctypes.c_int, [_vp, ctypes.c_uint64, ctypes.c_uint32,
                                                         _vp]),
            "or_container_decode": (ctypes.c_int, [_vp, ctypes.c_uint64, _vp]),
            "or_gemv": (None, [_vp, ctypes.c_uint32, ctypes.c_uint32, _vp, ctypes.c_uint32, _vp,
                               _vp]),
            "or_freq_norm": (ctypes.c_int, [_vp, ctypes.c_uint32, ctypes.c_uint32, _vp]),
            "or_tile_geometry": (None, [ctypes.c_uint32] * 5 + [_vp] * 4),
            "or_phrase_dict": (ctypes.c_int, [_vp] + [ctypes.c_uint32] * 6 + [_vp] * 4),
            "or_phrase_parse": (ctypes.c_int, [_vp, ctypes.c_uint32, _vp, ctypes.c_uint32, _vp,
                                               ctypes.c_uint32, _vp, ctypes.c_uint32, _vp, _vp]),
            "or_prans_encode": (ctypes.c_int, [_vp, _vp, _vp, ctypes.c_uint32, _vp,
                                               ctypes.c_uint32, ctypes.c_uint32, _vp,
                                               ctypes.c_uint64, _vp, _vp]),
            "or_prans_decode": (ctypes.c_int, [_vp, ctypes.c_uint64, _vp, _vp, ctypes.c_uint32,
                                               _vp, _vp, ctypes.c_uint32, ctypes.c_uint32, _vp,
                                               _vp, _vp]),
            "or_container2_build": (ctypes.c_int, [_vp, ctypes.c_uint32, ctypes.c_uint32,
                                                   ctypes.c_float, _vp, ctypes.c_uint32,
                                                   ctypes.c_uint32, ctypes.c_uint32,
                                                   ctypes.c_uint32, ctypes.c_uint32,
                                                   ctypes.c_uint64, ctypes.c_float,
                                                   ctypes.POINTER(ctypes.c_void_p),
                                                   ctypes.POINTER(ctypes.c_uint64)]),
            "or_container2_info": (ctypes.c_int, [_vp, ctypes.c_uint64, ctypes.POINTER(Info2)]),
            "or_container2_decode_chunk": (ctypes.c_int, [_vp, ctypes.c_uint64, ctypes.c_uint32,
                                                          _vp]),
            "or_container2_decode": (ctypes.c_int, [_vp, ctypes.c_uint64, _vp]),
        }
        for name, (res, args) in sig.items():
            fn = getattr(L, name)
            fn.restype = res
            fn.argtypes = args
        _lib = L
    return _lib


def _ptr(a: np.ndarray | None):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data


# ---- number formats ----
def e4m3_value(code: int) -> float:
    return lib().or_e4m3_value(code)


def e4m3_round(v: float) -> int:
    return lib().or_e4m3_round(v)


def int8_value(code: int) -> float:
    return lib().or_int8_value(code)


def int8_round(v: float) -> int:
    return lib().or_int8_round(v)


def qmax(fmt: int) -> float:
    return lib().or_qmax(fmt)


def code_value(fmt: int, code: int) -> float:
    return lib().or_code_value(fmt, code)


def bf16_value(bits: int) -> float:
    return lib().or_bf16_value(bits)


def bf16_round(v: float) -> int:
    return lib().or_bf16_round(v)


# ---- entropy ----
def entropy_counts(counts) -> float:
    c = np.ascontiguousarray(counts, dtype=np.uint64)
    return lib().or_entropy_counts(_ptr(c), c.size)


def entropy_codes(q: np.ndarray) -> float:
    q = np.ascontiguousarray(q, dtype=np.uint8)
    return lib().or_entropy_codes(_ptr(q), q.size)


def sparsity_entropy(s: float, h_nz: float) -> float:
    return lib().or_sparsity_entropy(s, h_nz)


# ---- quantiser ----
def row_scales(w: np.ndarray, alpha: float, fmt: int = E4M3) -> np.ndarray:
    w = np.ascontiguousarray(w, dtype=np.uint16)
    M, N = w.shape
    out = np.empty(M, dtype=np.uint16)
    lib().or_row_scales(_ptr(w), M, N, alpha, fmt, _ptr(out))
    return out


def quantize(w: np.ndarray, scale: np.ndarray, fmt: int = E4M3) -> np.ndarray:
    w = np.ascontiguousarray(w, dtype=np.uint16)
    scale = np.ascontiguousarray(scale, dtype=np.uint16)
    M, N = w.shape
    out = np.empty((M, N), dtype=np.uint8)
    lib().or_quantize(_ptr(w), M, N, _ptr(scale), fmt, _ptr(out))
    return out


def dequant(q: np.ndarray, scale: np.ndarray, fmt: int = E4M3) -> np.ndarray:
    q = np.ascontiguousarray(q, dtype=np.uint8)
    scale = np.ascontiguousarray(scale, dtype=np.uint16)
    M, N = q.shape
    out = np.empty((M, N), dtype=np.uint16)
    lib().or_dequant(_ptr(q), M, N, _ptr(scale), fmt, _ptr(out))
    return out


def alpha_search(w: np.ndarray, target_bits: float, fmt: int = E4M3):
    w = np.ascontiguousarray(w, dtype=np.uint16)
    M, N = w.shape
    h = ctypes.c_double()
    a = lib().or_alpha_search(_ptr(w), M, N, target_bits, fmt, ctypes.byref(h))
    return a, h.value


# ---- frequency table / coder ----
def freq_table(counts, P: int):
    c = np.ascontiguousarray(counts, dtype=np.uint64)
    assert c.size == 256
    sym = np.zeros(256, dtype=np.uint8)
    freq = np.zeros(256, dtype=np.uint16)
    K = ctypes.c_uint32()
    rc = lib().or_freq_table(_ptr(c), P, _ptr(sym), _ptr(freq), ctypes.byref(K))
    if rc != OK:
        raise ValueError(f"or_freq_table: {rc}")
    return sym[:K.value].copy(), freq[:K.value].copy()


def rans_encode(q: np.ndarray, lanes: int, P: int, sym: np.ndarray, freq: np.ndarray):
    q = np.ascontiguousarray(q, dtype=np.uint8)
    sym = np.ascontiguousarray(sym, dtype=np.uint8)
    freq = np.ascontiguousarray(freq, dtype=np.uint16)
    words = np.zeros(max(q.size, 1), dtype=np.uint16)
    states = np.zeros(lanes, dtype=np.uint32)
    nw = ctypes.c_uint32()
    rc = lib().or_rans_encode(_ptr(q), q.size, lanes, P, _ptr(sym), _ptr(freq), sym.size,
                              _ptr(words), words.size, ctypes.byref(nw), _ptr(states))
    if rc != OK:
        raise ValueError(f"or_rans_encode: {rc}")
    return words[:nw.value].copy(), states


def rans_decode(words: np.ndarray, states: np.ndarray, n: int, lanes: int, P: int,
                sym: np.ndarray, freq: np.ndarray):
    words = np.ascontiguousarray(words, dtype=np.uint16)
    states = np.ascontiguousarray(states, dtype=np.uint32)
    sym = np.ascontiguousarray(sym, dtype=np.uint8)
    freq = np.ascontiguousarray(freq, dtype=np.uint16)
    q = np.zeros(max(n, 1), dtype=np.uint8)
    w = words if words.size else np.zeros(1, dtype=np.uint16)
    rc = lib().or_rans_decode(_ptr(w), words.size, _ptr(states), n, lanes, P, _ptr(sym),
                              _ptr(freq), sym.size, _ptr(q))
    return rc, q[:n]


# ---- container ----
def container_build(w: np.ndarray, alpha: float, P: int, chunk_syms: int, lanes: int,
                    seed: int = 0, target_bits: float = 0.0, fmt: int = E4M3) -> np.ndarray:
    w = np.ascontiguousarray(w, dtype=np.uint16)
    M, N = w.shape
    p = ctypes.c_void_p()
    nb = ctypes.c_uint64()
    rc = lib().or_container_build(_ptr(w), M, N, alpha, fmt, P, chunk_syms, lanes, seed,
                                  target_bits, ctypes.byref(p), ctypes.byref(nb))
    if rc != OK:
        raise ValueError(f"or_container_build: {rc}")
    try:
        out = np.frombuffer(ctypes.string_at(p.value, nb.value), dtype=np.uint8).copy()
    finally:
        lib().or_free(p)
    return out


def container_build_scaled(w: np.ndarray, scale: np.ndarray, P: int, chunk_syms: int,
                           lanes: int, seed: int = 0, target_bits: float = 0.0,
                           fmt: int = E4M3) -> np.ndarray:
    w = np.ascontiguousarray(w, dtype=np.uint16)
    scale = np.ascontiguousarray(scale, dtype=np.uint16)
    M, N = w.shape
    p = ctypes.c_void_p()
    nb = ctypes.c_uint64()
    rc = lib().or_container_build_scaled(_ptr(w), M, N, _ptr(scale), fmt, P, chunk_syms, lanes,
                                         seed, target_bits, ctypes.byref(p), ctypes.byref(nb))
    if rc != OK:
        raise ValueError(f"or_container_build_scaled: {rc}")
    try:
        out = np.frombuffer(ctypes.string_at(p.value, nb.value), dtype=np.uint8).copy()
    finally:
        lib().or_free(p)
    return out


# ---- scale optimisation (Sec. 2.2 eq. optimization) ----
def rd_objective(w: np.ndarray, scale: np.ndarray, lam: float, fmt: int = E4M3):
    """(F, straight-through gradient, distortion term)."""
    w = np.ascontiguousarray(w, dtype=np.uint16)
    s = np.ascontiguousarray(scale, dtype=np.float64)
    M, N = w.shape
    g = np.empty(M, dtype=np.float64)
    d = ctypes.c_double()
    f = lib().or_rd_objective(_ptr(w), M, N, fmt, lam, _ptr(s), _ptr(g), ctypes.byref(d))
    return f, g, d.value


def rd_scales(w: np.ndarray, lam: float, iters: int = 200, history: int = 20, lr: float = 0.0,
              fmt: int = E4M3):
    """(scales, lowest F); lr <= 0: 0.25 if lam > 30 else 1.0 (App. A.1)."""
    w = np.ascontiguousarray(w, dtype=np.uint16)
    M, N = w.shape
    if lr <= 0:
        lr = 0.25 if lam > 30 else 1.0
    s = np.empty(M, dtype=np.float64)
    f = ctypes.c_double()
    rc = lib().or_rd_scales(_ptr(w), M, N, fmt, lam, iters, history, lr, _ptr(s), ctypes.byref(f))
    if rc != OK:
        raise ValueError(f"or_rd_scales: {rc}")
    return s, f.value


def lbfgs_quadratic(a: np.ndarray, b: float, c: np.ndarray, x0: np.ndarray, iters: int,
                    history: int = 20, lr: float = 1.0):
    a = np.ascontiguousarray(a, dtype=np.float64)
    c = np.ascontiguousarray(c, dtype=np.float64)
    x = np.ascontiguousarray(x0, dtype=np.float64).copy()
    f = ctypes.c_double()
    rc = lib().or_lbfgs_quadratic(a.size, _ptr(a), b, _ptr(c), iters, history, lr, _ptr(x),
                                  ctypes.byref(f))
    if rc != OK:
        raise ValueError(f"or_lbfgs_quadratic: {rc}")
    return x, f.value


def container_info(blob: np.ndarray) -> Info:
    blob = np.ascontiguousarray(blob, dtype=np.uint8)
    info = Info()
    rc = lib().or_container_info(_ptr(blob), blob.size, ctypes.byref(info))
    if rc != OK:
        raise ValueError(f"or_container_info: {rc}")
    return info


def container_decode_chunk(blob: np.ndarray, c: int):
    blob = np.ascontiguousarray(blob, dtype=np.uint8)
    info = container_info(blob)
    n = info.rows * info.cols
    nc = min(info.chunk_syms, n - c * info.chunk_syms)
    q = np.zeros(info.chunk_syms, dtype=np.uint8)
    rc = lib().or_container_decode_chunk(_ptr(blob), blob.size, c, _ptr(q))
    return rc, q[:nc]


def container_decode(blob: np.ndarray):
    blob = np.ascontiguousarray(blob, dtype=np.uint8)
    info = container_info(blob)
    q = np.zeros(info.n_chunks * info.chunk_syms, dtype=np.uint8)
    rc = lib().or_container_decode(_ptr(blob), blob.size, _ptr(q))
    return rc, q[:info.rows * info.cols].reshape(info.rows, info.cols)


def container_scales(blob: np.ndarray) -> np.ndarray:
    """The BF16 row scales (either container version)."""
    info = container2_info(blob) if container_version(blob) == 2 else container_info(blob)
    return np.frombuffer(blob[info.off_scale:info.off_scale + 2 * info.rows].tobytes(),
                         dtype=np.uint16).copy()


# ---- linear layer ----
def gemv(w_hat: np.ndarray, x: np.ndarray, bias: np.ndarray | None = None) -> np.ndarray:
    w_hat = np.ascontiguousarray(w_hat, dtype=np.uint16)
    x = np.ascontiguousarray(np.atleast_2d(x), dtype=np.uint16)
    M, N = w_hat.shape
    B = x.shape[0]
    assert x.shape[1] == N
    if bias is not None:
        bias = np.ascontiguousarray(bias, dtype=np.uint16)
    y = np.empty((B, M), dtype=np.float64)
    lib().or_gemv(_ptr(w_hat), M, N, _ptr(x), B, _ptr(bias), _ptr(y))
    return y


# ---- the same routines over independent pieces on several host threads ----
# Chunks are independent decode units and rows independent dequantisation and
# GEMV units, so these give exactly the single-threaded results; ctypes
# releases the interpreter lock for the duration of each C call.
def _threads(threads: int) -> int:
    if threads > 0:
        return threads
    return max(1, min(16, os.cpu_count() or 1))


def _row_blocks(M: int, n: int):
    step = max(1, (M + n - 1) // n)
    return [(r, min(M, r + step)) for r in range(0, M, step)]


def container_decode_par(blob: np.ndarray, threads: int = 0):
    """container_decode, chunk by chunk on `threads` host threads; returns the
    worst return code (OK only if every chunk decoded cleanly) and the codes."""
    from concurrent.futures import ThreadPoolExecutor
    blob = np.ascontiguousarray(blob, dtype=np.uint8)
    info = container_info(blob)
    q = np.zeros(info.n_chunks * info.chunk_syms, dtype=np.uint8)
    L = lib()

    def one(c):
        return L.or_container_decode_chunk(_ptr(blob), blob.size, c,
                                           q.ctypes.data + c * info.chunk_syms)

    with ThreadPoolExecutor(_threads(threads)) as ex:
        rcs = list(ex.map(one, range(info.n_chunks)))
    bad = [rc for rc in rcs if rc != OK]
    return (bad[0] if bad else OK), q[:info.rows * info.cols].reshape(info.rows, info.cols)


def dequant_par(q: np.ndarray, scale: np.ndarray, fmt: int = E4M3, threads: int = 0):
    from concurrent.futures import ThreadPoolExecutor
    q = np.ascontiguousarray(q, dtype=np.uint8)
    scale = np.ascontiguousarray(scale, dtype=np.uint16)
    M, N = q.shape
    out = np.empty((M, N), dtype=np.uint16)
    L = lib()

    def one(rr):
        r0, r1 = rr
        L.or_dequant(q.ctypes.data + r0 * N, r1 - r0, N, scale.ctypes.data + 2 * r0, fmt,
                     out.ctypes.data + 2 * r0 * N)

    with ThreadPoolExecutor(_threads(threads)) as ex:
        list(ex.map(one, _row_blocks(M, 4 * _threads(threads))))
    return out


def gemv_par(w_hat: np.ndarray, x: np.ndarray, bias: np.ndarray | None = None,
             threads: int = 0) -> np.ndarray:
    """gemv over row blocks on several threads (each row's sum is the same)."""
    from concurrent.futures import ThreadPoolExecutor
    w_hat = np.ascontiguousarray(w_hat, dtype=np.uint16)
    x = np.ascontiguousarray(np.atleast_2d(x), dtype=np.uint16)
    M, N = w_hat.shape
    B = x.shape[0]
    if bias is not None:
        bias = np.ascontiguousarray(bias, dtype=np.uint16)
    y = np.empty((B, M), dtype=np.float64)
    L = lib()

    def one(rr):
        r0, r1 = rr
        part = np.empty((B, r1 - r0), dtype=np.float64)
        L.or_gemv(w_hat.ctypes.data + 2 * r0 * N, r1 - r0, N, _ptr(x), B,
                  None if bias is None else bias.ctypes.data + 2 * r0, _ptr(part))
        y[:, r0:r1] = part

    with ThreadPoolExecutor(_threads(threads)) as ex:
        list(ex.map(one, _row_blocks(M, 4 * _threads(threads))))
    return y


def quantize_par(w: np.ndarray, scale: np.ndarray, fmt: int = E4M3, threads: int = 0):
    from concurrent.futures import ThreadPoolExecutor
    w = np.ascontiguousarray(w, dtype=np.uint16)
    scale = np.ascontiguousarray(scale, dtype=np.uint16)
    M, N = w.shape
    out = np.empty((M, N), dtype=np.uint8)
    L = lib()

    def one(rr):
        r0, r1 = rr
        L.or_quantize(w.ctypes.data + 2 * r0 * N, r1 - r0, N, scale.ctypes.data + 2 * r0, fmt,
                      out.ctypes.data + r0 * N)

    with ThreadPoolExecutor(_threads(threads)) as ex:
        list(ex.map(one, _row_blocks(M, 4 * _threads(threads))))
    return out



# ---- container version 2: tiles and aligned phrases ----
V2_RES = 12      # frequency resolution R (a symbol's probability in multiples of 2^-R)


def freq_norm(counts, R: int) -> np.ndarray:
    c = np.ascontiguousarray(counts, dtype=np.uint64)
    f = np.zeros(c.size, dtype=np.uint16)
    rc = lib().or_freq_norm(_ptr(c), c.size, R, _ptr(f))
    if rc != OK:
        raise ValueError(f"or_freq_norm: {rc}")
    return f


def tile_geometry(M: int, N: int, TR: int, TC: int, c: int):
    """(row0, col0, rows, cols) of chunk c."""
    v = [ctypes.c_uint32() for _ in range(4)]
    lib().or_tile_geometry(M, N, TR, TC, c, *[ctypes.addressof(x) for x in v])
    return tuple(x.value for x in v)


def phrase_dict(q: np.ndarray, TR: int, TC: int, R: int = V2_RES, tau: int = 1):
    """(DQ, DP): quad and pair values (little-endian code bytes), ascending."""
    q = np.ascontiguousarray(q, dtype=np.uint8)
    M, N = q.shape
    quads = np.zeros(1 << (R - 1), dtype=np.uint32)
    pairs = np.zeros(1 << (R - 2), dtype=np.uint32)
    nq, np_ = ctypes.c_uint32(), ctypes.c_uint32()
    rc = lib().or_phrase_dict(_ptr(q), M, N, TR, TC, R, tau, _ptr(quads), ctypes.addressof(nq),
                              _ptr(pairs), ctypes.addressof(np_))
    if rc != OK:
        raise ValueError(f"or_phrase_dict: {rc}")
    return quads[:nq.value].copy(), pairs[:np_.value].copy()


def phrase_parse(u: np.ndarray, quads, pairs, singles) -> np.ndarray:
    u = np.ascontiguousarray(u, dtype=np.uint8)
    quads = np.ascontiguousarray(quads, dtype=np.uint32)
    pairs = np.ascontiguousarray(pairs, dtype=np.uint32)
    singles = np.ascontiguousarray(singles, dtype=np.uint8)
    out = np.zeros(max(u.size, 1), dtype=np.uint32)
    n = ctypes.c_uint32()
    rc = lib().or_phrase_parse(_ptr(u), u.size, _ptr(quads) if quads.size else None, quads.size,
                               _ptr(pairs) if pairs.size else None, pairs.size,
                               _ptr(singles) if singles.size else None, singles.size, _ptr(out),
                               ctypes.addressof(n))
    if rc != OK:
        raise ValueError(f"or_phrase_parse: {rc}")
    return out[:n.value].copy()


def prans_encode(tokens, freq, R: int):
    """tokens: one sequence of symbol indices per state.  Returns (words, states)."""
    W = len(tokens)
    lens = np.array([len(t) for t in tokens], dtype=np.uint32)
    off = np.zeros(W, dtype=np.uint64)
    off[1:] = np.cumsum(lens.astype(np.uint64))[:-1]
    flat = np.ascontiguousarray(np.concatenate([np.asarray(t, dtype=np.uint32) for t in tokens])
                                if lens.sum() else np.zeros(1, dtype=np.uint32))
    freq = np.ascontiguousarray(freq, dtype=np.uint16)
    cap = int(lens.sum()) + 16
    words = np.zeros(cap, dtype=np.uint16)
    states = np.zeros(W, dtype=np.uint32)
    nw = ctypes.c_uint64()
    rc = lib().or_prans_encode(_ptr(flat), _ptr(off), _ptr(lens), W, _ptr(freq), freq.size, R,
                               _ptr(words), cap, ctypes.addressof(nw), _ptr(states))
    if rc != OK:
        raise ValueError(f"or_prans_encode: {rc}")
    return words[:nw.value].copy(), states


def prans_decode(words, states, need, freq, plen, R: int):
    """Returns (rc, list of symbol sequences per state)."""
    words = np.ascontiguousarray(words, dtype=np.uint16)
    states = np.ascontiguousarray(states, dtype=np.uint32)
    need = np.ascontiguousarray(need, dtype=np.uint32)
    freq = np.ascontiguousarray(freq, dtype=np.uint16)
    plen = np.ascontiguousarray(plen, dtype=np.uint8)
    W = states.size
    off = np.zeros(W, dtype=np.uint64)
    off[1:] = np.cumsum(need.astype(np.uint64))[:-1]
    tok = np.zeros(int(need.sum()) + 1, dtype=np.uint32)
    got = np.zeros(W, dtype=np.uint32)
    wp = words if words.size else np.zeros(1, dtype=np.uint16)
    rc = lib().or_prans_decode(_ptr(wp), words.size, _ptr(states), _ptr(need), W, _ptr(freq),
                               _ptr(plen), freq.size, R, _ptr(tok), _ptr(off), _ptr(got))
    return rc, [tok[int(off[s]):int(off[s]) + int(got[s])].copy() for s in range(W)]


def container2_build(w: np.ndarray, alpha: float, TR: int, TC: int, R: int = V2_RES,
                     seed: int = 0, target_bits: float = 0.0, fmt: int = E4M3,
                     scale: np.ndarray | None = None, row_order: bool = False) -> np.ndarray:
    """Version-2 container; row_order: tiles cut over the rows sorted by their
    phrase count (eq_phrase.c, item 4)."""
    w = np.ascontiguousarray(w, dtype=np.uint16)
    M, N = w.shape
    if scale is not None:
        scale = np.ascontiguousarray(scale, dtype=np.uint16)
    p = ctypes.c_void_p()
    nb = ctypes.c_uint64()
    rc = lib().or_container2_build(_ptr(w), M, N, alpha, _ptr(scale), fmt, R, TR, TC,
                                   int(bool(row_order)), seed, target_bits, ctypes.byref(p),
                                   ctypes.byref(nb))
    if rc != OK:
        raise ValueError(f"or_container2_build: {rc}")
    try:
        out = np.frombuffer(ctypes.string_at(p.value, nb.value), dtype=np.uint8).copy()
    finally:
        lib().or_free(p)
    return out


def container2_info(blob: np.ndarray) -> Info2:
    blob = np.ascontiguousarray(blob, dtype=np.uint8)
    info = Info2()
    rc = lib().or_container2_info(_ptr(blob), blob.size, ctypes.byref(info))
    if rc != OK:
        raise ValueError(f"or_container2_info: {rc}")
    return info


def container_version(blob: np.ndarray) -> int:
    return int(np.frombuffer(np.ascontiguousarray(blob[4:8]).tobytes(), dtype=np.uint32)[0])


def container2_decode_chunk(blob: np.ndarray, c: int):
    """(rc, codes of tile c as a rows x cols array)."""
    blob = np.ascontiguousarray(blob, dtype=np.uint8)
    info = container2_info(blob)
    r0, c0, rows, cols = tile_geometry(info.rows, info.cols, info.lanes, info.tile_cols, c)
    t = np.zeros(max(rows * cols, 1), dtype=np.uint8)
    rc = lib().or_container2_decode_chunk(_ptr(blob), blob.size, c, _ptr(t))
    return rc, t[:rows * cols].reshape(rows, cols)


def container2_decode(blob: np.ndarray):
    blob = np.ascontiguousarray(blob, dtype=np.uint8)
    info = container2_info(blob)
    q = np.zeros((info.rows, info.cols), dtype=np.uint8)
    rc = lib().or_container2_decode(_ptr(blob), blob.size, _ptr(q))
    return rc, q


def container2_row_order(blob: np.ndarray) -> np.ndarray:
    """order[k]: the matrix row of stored row k (the identity without a row
    order section)."""
    info = container2_info(blob)
    if not info.flags & 1:
        return np.arange(info.rows, dtype=np.uint32)
    o = info.off_order
    return np.frombuffer(np.ascontiguousarray(blob[o:o + 4 * info.rows]).tobytes(),
                         dtype=np.uint32).copy()


def container2_decode_par(blob: np.ndarray, threads: int = 0):
    """container2_decode, tile by tile on several host threads."""
    from concurrent.futures import ThreadPoolExecutor
    blob = np.ascontiguousarray(blob, dtype=np.uint8)
    info = container2_info(blob)
    order = container2_row_order(blob)
    q = np.zeros((info.rows, info.cols), dtype=np.uint8)

    def one(c):
        rc, t = container2_decode_chunk(blob, c)
        r0, c0, rows, cols = tile_geometry(info.rows, info.cols, info.lanes, info.tile_cols, c)
        q[order[r0:r0 + rows], c0:c0 + cols] = t
        return rc

    with ThreadPoolExecutor(_threads(threads)) as ex:
        rcs = list(ex.map(one, range(info.n_chunks)))
    bad = [rc for rc in rcs if rc != OK]
    return (bad[0] if bad else OK), q


def container2_phrases(blob: np.ndarray):
    """(codes [n][4], lengths [n], freq [n]) of the container's alphabet."""
    info = container2_info(blob)
    n = info.n_syms
    codes = blob[info.off_phr:info.off_phr + 4 * n].reshape(n, 4).copy()
    plen = np.array([4] * info.n_quads + [2] * info.n_pairs + [1] * info.n_singles, dtype=np.uint8)
    freq = np.frombuffer(blob[info.off_freq:info.off_freq + 2 * n].tobytes(), dtype=np.uint16).copy()
    return codes, plen, freq
