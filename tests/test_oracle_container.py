"""Oracle container (Alg. 1 end to end, Alg. 2, entropy decoding) and linear layer.

Pins: decoded codes equal the quantiser's codes (lossless, Sec. 2.2), the
header's entropy equals the codes' empirical entropy, payload bits/param is
bounded below by that entropy (source coding), corrupted containers are
rejected, and the fp64 GEMV matches numpy's matmul of the dequantised weights.
"""
import numpy as np
import pytest

import oracle
import synth


def test_c1_container_round_trip(c1_container):
    spec, w, alpha, blob = c1_container
    info = oracle.container_info(blob)
    assert (info.rows, info.cols) == (spec.rows, spec.cols)
    assert info.n_chunks == spec.rows * spec.cols // spec.chunk_syms
    rc, q = oracle.container_decode(blob)
    assert rc == oracle.OK
    scale = oracle.container_scales(blob)
    assert (scale == oracle.row_scales(w, alpha)).all()
    assert (q == oracle.quantize(w, scale)).all()
    assert info.entropy_bits == pytest.approx(oracle.entropy_codes(q), abs=1e-6)
    assert abs(info.entropy_bits - spec.target_bits) <= 0.05


def test_payload_bounded_by_entropy(c1_container):
    """Source coding: the stored bits (words and final states) cannot go below
    n * H; the information actually used (words plus log2(x / 2^16) per final
    state) sits within 1 % of n * H."""
    spec, w, alpha, blob = c1_container
    info = oracle.container_info(blob)
    n = spec.rows * spec.cols
    st = blob[info.off_chunk_state:info.off_chunk_state + 4 * info.n_chunks * info.lanes]
    st = st.view(np.uint32).astype(np.float64)
    stored = 16 * info.total_words + 32 * st.size
    assert stored >= n * info.entropy_bits
    used = 16 * info.total_words + np.log2(st / 65536.0).sum()
    assert abs(used / n - info.entropy_bits) <= 0.01 * info.entropy_bits


@pytest.mark.parametrize("M,N,C,lanes", [(5, 77, 128, 64), (3, 64, 64, 64), (7, 300, 256, 128),
                                         (1, 1, 64, 64), (33, 1000, 1024, 256)])
def test_ragged_shapes_round_trip(M, N, C, lanes):
    from synth.configs import small_spec
    w = synth.weights(small_spec(M, N, seed=M * N))
    blob = oracle.container_build(w, 300.0, 12, C, lanes)
    rc, q = oracle.container_decode(blob)
    assert rc == oracle.OK
    assert (q == oracle.quantize(w, oracle.row_scales(w, 300.0))).all()


def test_single_symbol_matrix():
    w = np.zeros((4, 256), dtype=np.uint16)
    blob = oracle.container_build(w, 1.0, 12, 512, 64)
    info = oracle.container_info(blob)
    assert info.n_syms == 1 and info.total_words == 0
    rc, q = oracle.container_decode(blob)
    assert rc == oracle.OK and (q == 0).all()


def test_corrupted_container_rejected(c1_container):
    spec, w, alpha, blob = c1_container
    info = oracle.container_info(blob)
    _, q_ref = oracle.container_decode_chunk(blob, 7)
    r = np.random.default_rng(12)
    w0 = int(blob[info.off_chunk_off + 28:info.off_chunk_off + 32].view(np.uint32)[0])
    w1 = int(blob[info.off_chunk_off + 32:info.off_chunk_off + 36].view(np.uint32)[0])
    for _ in range(20):
        bad = blob.copy()
        byte = info.off_words + 2 * int(r.integers(w0, w1)) + int(r.integers(2))
        bad[byte] ^= np.uint8(1 << int(r.integers(8)))
        rc, q = oracle.container_decode_chunk(bad, 7)
        assert rc == oracle.ECORRUPT or not (q == q_ref).all()
    bad = blob.copy()
    bad[:4] = np.frombuffer(b"XQC1", dtype=np.uint8)
    with pytest.raises(ValueError):
        oracle.container_info(bad)
    with pytest.raises(ValueError):
        oracle.container_info(blob[:200])


def test_gemv_matches_numpy(c1_container):
    spec, w, alpha, blob = c1_container
    rc, q = oracle.container_decode(blob)
    w_hat = oracle.dequant(q, oracle.container_scales(blob))
    x = synth.activations(spec, 3)
    bias = synth.bias(spec)
    y = oracle.gemv(w_hat, x, bias)
    ref = synth.bf16_to_f32(x).astype(np.float64) @ synth.bf16_to_f32(w_hat).astype(np.float64).T
    ref += synth.bf16_to_f32(bias).astype(np.float64)
    assert np.allclose(y, ref, rtol=1e-12, atol=1e-12)
