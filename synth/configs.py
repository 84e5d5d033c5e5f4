"""The five synthetic workloads: shapes, value distributions, target entropy.

Every matrix is [out features M, in features N], row-major, BF16.
Seeds: 0x260122787 + 1000*config + 16*layer + matrix_id.
"""
from __future__ import annotations

from dataclasses import dataclass, replace

BASE_SEED = 0x260122787

STUDENT_T = 1
GAUSS_OUTLIER = 2


@dataclass(frozen=True)
class MatrixSpec:
    name: str
    rows: int            # M (out features)
    cols: int            # N (in features)
    kind: int            # STUDENT_T or GAUSS_OUTLIER
    nu: int              # Student-t degrees of freedom
    row_sigma: float     # log-normal per-row scale parameter
    outlier_p: float
    outlier_mag: float
    target_bits: float   # target empirical entropy (bits/param)
    chunk_syms: int      # C, symbols per chunk
    lanes: int           # interleaved coder states per chunk
    seed: int

    @property
    def params(self) -> int:
        return self.rows * self.cols


def matrix_seed(config: int, layer: int, matrix_id: int) -> int:
    return BASE_SEED + 1000 * config + 16 * layer + matrix_id


def _t(name, M, N, nu, sigma, bits, C, lanes, cfg, layer, mid):
    return MatrixSpec(name, M, N, STUDENT_T, nu, sigma, 0.0, 0.0, bits, C, lanes,
                      matrix_seed(cfg, layer, mid))


def _g(name, M, N, sigma, bits, C, lanes, cfg, layer, mid):
    return MatrixSpec(name, M, N, GAUSS_OUTLIER, 0, sigma, 1e-3, 20.0, bits, C, lanes,
                      matrix_seed(cfg, layer, mid))


# Interleaved states per chunk: 64 (one per wavefront lane) for short chunks;
# 256 for 64Ki-symbol chunks so that a large matrix still has enough
# independent decode chains to keep every SIMD busy.
def _lanes(C: int) -> int:
    return 256 if C >= 65536 else 64


CONFIGS = {
    1: dict(desc="single 1024x1024 matrix, t(5) x LN(0,0.5), ~2.0 bits, 4096-symbol chunks",
            batches=(1,)),
    2: dict(desc="Llama-2-7B attention projection 4096x4096, t(5) x LN(0,0.5), ~3.0 bits, "
                 "16384-symbol chunks", batches=(1,)),
    3: dict(desc="Llama-2-7B MLP gate/up 11008x4096 and down 4096x11008, N(0,1)+0.1% "
                 "+-20 sigma outliers x LN(0,0.7), ~2.0 bits, 16384-symbol chunks",
            batches=(1,)),
    4: dict(desc="Llama-70B MLP 8192x28672 and 28672x8192, t(4) x LN(0,0.5), ~2.0 bits, "
                 "65536-symbol chunks", batches=(1, 8)),
    5: dict(desc="80-layer 70B-shaped stack (q,k,v,o,gate,up,down), t(5) x LN(0,0.5), "
                 "~2/3/4 bits by layer mod 3, 65536-symbol chunks", batches=(1,)),
}

_STACK = (("q", 8192, 8192), ("k", 1024, 8192), ("v", 1024, 8192), ("o", 8192, 8192),
          ("gate", 28672, 8192), ("up", 28672, 8192), ("down", 8192, 28672))


def config_matrices(config: int, layers=None):
    """List of MatrixSpec for a configuration (config 5: optionally a subset of layers)."""
    if config == 1:
        return [_t("w", 1024, 1024, 5, 0.5, 2.0, 4096, _lanes(4096), 1, 0, 0)]
    if config == 2:
        return [_t("attn", 4096, 4096, 5, 0.5, 3.0, 16384, _lanes(16384), 2, 0, 0)]
    if config == 3:
        return [_g("gate", 11008, 4096, 0.7, 2.0, 16384, _lanes(16384), 3, 0, 0),
                _g("up", 11008, 4096, 0.7, 2.0, 16384, _lanes(16384), 3, 0, 1),
                _g("down", 4096, 11008, 0.7, 2.0, 16384, _lanes(16384), 3, 0, 2)]
    if config == 4:
        return [_t("down", 8192, 28672, 4, 0.5, 2.0, 65536, _lanes(65536), 4, 0, 0),
                _t("up", 28672, 8192, 4, 0.5, 2.0, 65536, _lanes(65536), 4, 0, 1)]
    if config == 5:
        out = []
        for layer in (range(80) if layers is None else layers):
            bits = (2.0, 3.0, 4.0)[layer % 3]
            for mid, (nm, M, N) in enumerate(_STACK):
                out.append(_t(f"l{layer}.{nm}", M, N, 5, 0.5, bits, 65536, _lanes(65536),
                              5, layer, mid))
        return out
    raise ValueError(f"unknown config {config}")


def small_spec(rows: int, cols: int, *, bits: float = 2.0, chunk: int = 4096, lanes: int = 64,
               nu: int = 5, sigma: float = 0.5, seed: int = 1, outliers: bool = False) -> MatrixSpec:
    """A small ad-hoc matrix for tests (same distributions as the configs)."""
    if outliers:
        return MatrixSpec("small", rows, cols, GAUSS_OUTLIER, 0, sigma, 1e-3, 20.0, bits, chunk,
                          lanes, BASE_SEED + seed)
    return MatrixSpec("small", rows, cols, STUDENT_T, nu, sigma, 0.0, 0.0, bits, chunk, lanes,
                      BASE_SEED + seed)


def with_chunking(spec: MatrixSpec, chunk: int, lanes: int) -> MatrixSpec:
    return replace(spec, chunk_syms=chunk, lanes=lanes)
