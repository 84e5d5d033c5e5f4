"""Seeded synthetic inputs shared by the product encoder and the test oracle.

Only input synthesis lives here (weights and activation vectors with the
workloads' shapes and value distributions); none of the method's arithmetic.
The C source is ``synth.c``; ``build()`` compiles it to ``libsynth.so``.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

from .configs import CONFIGS, MatrixSpec, config_matrices, matrix_seed  # noqa: F401

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libsynth.so")
_lib = None

STUDENT_T = 1
GAUSS_OUTLIER = 2


class _WeightSpec(ctypes.Structure):
    _fields_ = [
        ("kind", ctypes.c_int32),
        ("nu", ctypes.c_int32),
        ("row_sigma", ctypes.c_double),
        ("outlier_p", ctypes.c_double),
        ("outlier_mag", ctypes.c_double),
    ]


def build() -> str:
    """Compile libsynth.so in place (always recompiles)."""
    cmd = ["gcc", "-O2", "-std=c99", "-D_GNU_SOURCE", "-fPIC", "-shared",
           "-ffp-contract=off", "-pthread", os.path.join(_HERE, "synth.c"),
           "-o", _LIB_PATH + ".tmp", "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(_LIB_PATH + ".tmp", _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build()
        lib = ctypes.CDLL(_LIB_PATH)
        lib.eqs_u64.restype = ctypes.c_uint64
        lib.eqs_u64.argtypes = [ctypes.c_uint64] * 3
        lib.eqs_uniform.restype = ctypes.c_double
        lib.eqs_uniform.argtypes = [ctypes.c_uint64] * 3
        lib.eqs_to_bf16.restype = ctypes.c_uint16
        lib.eqs_to_bf16.argtypes = [ctypes.c_double]
        lib.eqs_weights.restype = ctypes.c_int
        lib.eqs_weights.argtypes = [ctypes.POINTER(_WeightSpec), ctypes.c_uint64,
                                    ctypes.c_uint32, ctypes.c_uint32,
                                    ctypes.c_void_p, ctypes.c_int]
        lib.eqs_vector.restype = ctypes.c_int
        lib.eqs_vector.argtypes = [ctypes.c_uint64, ctypes.c_uint64, ctypes.c_uint64,
                                   ctypes.c_void_p]
        _lib = lib
    return _lib


def u64(seed: int, stream: int, ctr: int) -> int:
    return _load().eqs_u64(seed, stream, ctr)


def uniform(seed: int, stream: int, ctr: int) -> float:
    return _load().eqs_uniform(seed, stream, ctr)


def to_bf16(v: float) -> int:
    return _load().eqs_to_bf16(v)


def weights(spec: MatrixSpec, threads: int = 0) -> np.ndarray:
    """BF16 bit patterns, shape (rows, cols), dtype uint16."""
    ws = _WeightSpec(spec.kind, spec.nu, spec.row_sigma, spec.outlier_p, spec.outlier_mag)
    out = np.empty((spec.rows, spec.cols), dtype=np.uint16)
    rc = _load().eqs_weights(ctypes.byref(ws), spec.seed, spec.rows, spec.cols,
                             out.ctypes.data, threads)
    if rc != 0:
        raise ValueError("eqs_weights rejected the spec")
    return out


def vector(seed: int, stream: int, n: int) -> np.ndarray:
    """bf16(N(0,1)) draws as uint16 bit patterns."""
    out = np.empty(n, dtype=np.uint16)
    _load().eqs_vector(seed, stream, n, out.ctypes.data)
    return out


def activations(spec: MatrixSpec, batch: int) -> np.ndarray:
    """Activation rows x[b, :cols] for a matrix, as uint16 BF16 patterns."""
    return np.stack([vector(spec.seed, 16 + b, spec.cols) for b in range(batch)])


def bias(spec: MatrixSpec) -> np.ndarray:
    """A bf16 bias vector of length rows (stream 15)."""
    return vector(spec.seed, 15, spec.rows)


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    """Reinterpret uint16 BF16 patterns as float32 values (exact)."""
    return (bits.astype(np.uint32) << 16).view(np.float32)
