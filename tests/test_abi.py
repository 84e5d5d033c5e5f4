"""The C-ABI library: loads without a GPU, exports every declared symbol, and
validates containers on the host (no device access in these calls)."""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
import paper_2601_22787_amd as eq
import synth
from synth.configs import small_spec

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    names = set()
    for h in ("eq.h", "eq_encode.h"):
        text = open(os.path.join(ROOT, "include", h)).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        names |= set(re.findall(r"\b(eqe?_\w+)\s*\(", text))
    return names


def test_every_declared_symbol_is_exported():
    names = _declared()
    assert {"eq_layer_init", "eq_layer_prepare", "eq_decode_codes", "eq_decode_bf16",
            "eq_decode_gemv", "eq_gemv_workspace_bytes", "eq_get_status", "eq_strerror",
            "eq_lut_bytes", "eqe_encode", "eqe_alpha_search", "eqe_free"} <= names
    L = ctypes.CDLL(eq._LIB_PATH)
    for n in names:
        assert hasattr(L, n), n
    assert names == set(eq.SIGNATURES)


def test_strerror():
    assert eq.eq_strerror(0) == "ok"
    for code in (-1, -2, -3, -4):
        assert eq.eq_strerror(code) and eq.eq_strerror(code) != "unknown error code"
    assert eq.eq_strerror(7) == "unknown error code"


@pytest.fixture(scope="module")
def blob():
    w = synth.weights(small_spec(40, 512, seed=21))
    return eq.eqe_encode(w, 300.0, chunk_syms=2048, lanes=128)


_FAKE = np.zeros(1024, dtype=np.uint8)


def _fake_ptr(offset=0):
    """A 256-byte aligned host address (plus offset) standing in for device
    pointers: eq_layer_init never dereferences them."""
    base = _FAKE.ctypes.data
    return (base + 255) // 256 * 256 + offset


def _init(b, dev_offset=0):
    b = np.ascontiguousarray(b, dtype=np.uint8)
    L = eq.eq_layer()
    rc = eq.lib().eq_layer_init(ctypes.byref(L), b.ctypes.data, b.size, _fake_ptr(dev_offset),
                                _fake_ptr(), _fake_ptr())
    return rc, L


def test_layer_init_accepts_valid(blob):
    rc, L = _init(blob)
    assert rc == eq.EQ_OK
    info = oracle.container_info(blob)
    assert (L.rows, L.cols, L.chunk_syms, L.n_chunks, L.lanes, L.prob_bits, L.n_syms) == \
        (info.rows, info.cols, info.chunk_syms, info.n_chunks, info.lanes, info.prob_bits,
         info.n_syms)
    assert L.total_words == info.total_words


def _patch(b, off, value, dtype):
    b = b.copy()
    b[off:off + np.dtype(dtype).itemsize] = np.frombuffer(np.array([value], dtype=dtype).tobytes(),
                                                          dtype=np.uint8)
    return b


def test_layer_init_rejects_bad_containers(blob):
    info = oracle.container_info(blob)
    bad = {
        "magic": _patch(blob, 0, 0x31435158, np.uint32),
        "version": _patch(blob, 4, 2, np.uint32),
        "format": _patch(blob, 12, 3, np.uint32),
        "lanes": _patch(blob, 32, 96, np.uint32),
        "chunks": _patch(blob, 28, info.n_chunks + 1, np.uint32),
        "prob_bits_small": _patch(blob, 36, 7, np.uint32),
        "freq_sum": _patch(blob, info.off_freq, 1 + int(blob[info.off_freq]), np.uint8),
        "sym_order": _patch(blob, info.off_sym, 0xFE, np.uint8),
        "offset_order": _patch(blob, info.off_chunk_off + 4, 0xFFFFFFF, np.uint32),
        "state_low": _patch(blob, info.off_chunk_state + 8, 5, np.uint32),
        "scale_zero": _patch(blob, info.off_scale + 6, 0, np.uint16),
        "scale_inf": _patch(blob, info.off_scale + 6, 0x7F80, np.uint16),
        "padding": _patch(blob, 56, info.total_words + 8, np.uint64),
        "section": _patch(blob, 128, 1 << 40, np.uint64),
        # M * N >= 2^32 (element indices are 32-bit), the chunk count adjusted
        "too_large": _patch(_patch(_patch(blob, 16, 65536, np.uint32), 20, 65536, np.uint32),
                            28, (1 << 32) // 2048, np.uint32),
        "empty": _patch(blob, 16, 0, np.uint32),
    }
    for name, b in bad.items():
        rc, _ = _init(b)
        assert rc == eq.EQ_EFORMAT, name
    rc, _ = _init(blob[:300])
    assert rc == eq.EQ_EFORMAT
    L = eq.eq_layer()
    assert eq.lib().eq_layer_init(ctypes.byref(L), None, 0, None, None, None) == eq.EQ_EINVAL


def test_layer_init_base_formats(blob):
    """Int8 containers validate and report their format; a symbol outside the
    base format (E4M3 NaN, Int8 -128) is rejected."""
    w = synth.weights(small_spec(24, 256, seed=8))
    b8 = eq.eqe_encode(w, 20.0, chunk_syms=1024, lanes=64, base_format=eq.FMT_INT8)
    rc, L = _init(b8)
    assert rc == eq.EQ_OK and L.base_format == eq.FMT_INT8
    rc, L = _init(blob)
    assert rc == eq.EQ_OK and L.base_format == eq.FMT_E4M3
    # the first negative code (sign bit set) can be lowered to 0x80 (Int8) or
    # to 0x7F (E4M3) without breaking the ascending order
    for cont, bad_code in ((b8, 0x80), (blob, 0x7F)):
        info = oracle.container_info(cont)
        syms = cont[info.off_sym:info.off_sym + info.n_syms]
        k = int(np.argmax(syms >= 0x80))
        assert syms[k] > bad_code and (k == 0 or syms[k - 1] < bad_code)
        rc, _ = _init(_patch(cont, info.off_sym + k, bad_code, np.uint8))
        assert rc == eq.EQ_EFORMAT


def test_workspace_size_and_argument_checks(blob):
    rc, L = _init(blob)
    assert rc == eq.EQ_OK
    assert eq.lib().eq_gemv_workspace_bytes(ctypes.byref(L), 0) == 0
    assert eq.lib().eq_gemv_workspace_bytes(ctypes.byref(L), 9) == 0
    assert eq.lib().eq_gemv_workspace_bytes(ctypes.byref(L), 8) >= 2 * L.n_chunks * 8 * 4
    # null outputs are rejected on the host, before any launch
    assert eq.lib().eq_decode_codes(ctypes.byref(L), None, None) == eq.EQ_EINVAL
    assert eq.lib().eq_decode_bf16(ctypes.byref(L), None, None) == eq.EQ_EINVAL
    fake = np.zeros(16, dtype=np.uint8)
    assert eq.lib().eq_decode_gemv(ctypes.byref(L), fake.ctypes.data, 9, None, fake.ctypes.data,
                                   fake.ctypes.data, 1 << 20, None) == eq.EQ_EINVAL
    assert eq.lib().eq_decode_gemv(ctypes.byref(L), fake.ctypes.data, 2, None, fake.ctypes.data,
                                   fake.ctypes.data, 4, None) == eq.EQ_EINVAL


def test_layer_init_requires_aligned_device_copy(blob):
    """Sections are read with dword and wider loads: a device copy that is not
    256-byte aligned is refused before any launch."""
    assert _init(blob)[0] == eq.EQ_OK
    for off in (2, 4, 128):
        assert _init(blob, dev_offset=off)[0] == eq.EQ_EINVAL, off


@pytest.mark.parametrize("P", [8, 12])
def test_probability_precision_edges(P):
    """The container format takes 8 <= P <= 12 (the kernels multiply f by
    x >> P with 24-bit operands): the oracle's and the product's encoders
    write byte-identical containers at both edges and the library accepts
    them; below the range both encoders refuse to write one and the library
    rejects a header that claims it."""
    w = synth.weights(small_spec(24, 384, seed=30 + P))
    alpha, _ = oracle.alpha_search(w, 2.0)
    ref = oracle.container_build(w, alpha, P, 1024, 64)
    blob = eq.eqe_encode(w, alpha, prob_bits=P, chunk_syms=1024, lanes=64)
    assert np.array_equal(blob, ref)
    rc, L = _init(blob)
    assert rc == eq.EQ_OK and L.prob_bits == P
    rc_dec, q = oracle.container_decode(ref)
    assert rc_dec == oracle.OK and np.array_equal(q, oracle.quantize(w, oracle.container_scales(ref)))


def test_probability_precision_below_range_rejected():
    w = synth.weights(small_spec(8, 256, seed=37))
    with pytest.raises(ValueError):
        oracle.container_build(w, 300.0, 7, 1024, 64)
    with pytest.raises(eq.EqError):
        eq.eqe_encode(w, 300.0, prob_bits=7, chunk_syms=1024, lanes=64)
    ref = oracle.container_build(w, 300.0, 8, 1024, 64)
    bad = _patch(ref, 36, 7, np.uint32)
    with pytest.raises(ValueError):
        oracle.container_info(bad)
    assert _init(bad)[0] == eq.EQ_EFORMAT


def test_layer_init_version2():
    """A version-2 container validates and reports its tile shape and
    alphabet; damaged headers and sections are rejected on the host."""
    w = synth.weights(small_spec(70, 1000, seed=23))
    alpha, _ = oracle.alpha_search(w, 2.0)
    b2 = eq.eqe_encode2(w, alpha, tile_rows=64, tile_cols=256)
    info = oracle.container2_info(b2)
    rc, L = _init(b2)
    assert rc == eq.EQ_OK and L.version == 2
    assert (L.rows, L.cols, L.lanes, L.tile_cols, L.n_chunks, L.prob_bits, L.n_syms) == \
        (70, 1000, 64, 256, info.n_chunks, 12, info.n_syms)
    assert (L.n_quads, L.n_pairs, L.n_singles) == (info.n_quads, info.n_pairs, info.n_singles)
    assert eq.lib().eq_gemv_workspace_bytes(ctypes.byref(L), 8) >= 8 * 4 * 70 * 4
    bad = {
        "tile_cols": _patch(b2, 84, 250, np.uint32),
        "res_bits": _patch(b2, 36, 9, np.uint32),
        "parts": _patch(b2, 144, info.n_quads + 1, np.uint32),
        "chunks": _patch(b2, 28, info.n_chunks - 1, np.uint32),
        "freq": _patch(b2, info.off_freq, 7, np.uint16),
        "phrase_order": _patch(b2, info.off_phr, 0xFFFFFFF0, np.uint32),
        "pair_byte": _patch(b2, info.off_phr + 4 * info.n_quads + 3, 1, np.uint8),
        "nan_code": _patch(b2, info.off_phr + 4 * (info.n_syms - 1), 0x7F, np.uint8),
        "state_low": _patch(b2, info.off_chunk_state + 4, 3, np.uint32),
        "offsets": _patch(b2, info.off_chunk_off + 4, 0xFFFFFFF, np.uint32),
    }
    for name, b in bad.items():
        assert _init(b)[0] == eq.EQ_EFORMAT, name


def test_layer_init_version2_row_order():
    """A version-2 container with a row order: the layer points at its order
    section; a repeated or out-of-range row, an unknown flag, or an order
    offset without the flag is rejected on the host."""
    w = synth.weights(small_spec(70, 1000, seed=24))
    alpha, _ = oracle.alpha_search(w, 2.0)
    b2 = eq.eqe_encode2(w, alpha, tile_rows=64, tile_cols=256, row_order=True)
    info = oracle.container2_info(b2)
    rc, L = _init(b2)
    assert rc == eq.EQ_OK and L.version == 2
    assert L.row_order == _fake_ptr() + info.off_order
    order = oracle.container2_row_order(b2)
    bad = {
        "repeated": _patch(b2, info.off_order + 4, int(order[0]), np.uint32),
        "range": _patch(b2, info.off_order + 8, 70, np.uint32),
        "flag": _patch(b2, 44, 3, np.uint32),
        "offset_without_flag": _patch(b2, 44, 0, np.uint32),
        "section": _patch(b2, 160, info.file_bytes - 16, np.uint64),
    }
    for name, b in bad.items():
        assert _init(b)[0] == eq.EQ_EFORMAT, name
    plain = eq.eqe_encode2(w, alpha, tile_rows=64, tile_cols=256)
    rc, L = _init(plain)
    assert rc == eq.EQ_OK and not L.row_order
