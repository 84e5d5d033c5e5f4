"""Host-side rules of the benchmark: the version-2 tile shape of every
matrix it times (the full-size GPU tests use the same shapes)."""
import bench
from synth.configs import config_matrices


def test_v2_tile_shapes():
    """Tile width from the chunk size (state bytes per code), tile height
    halved when the matrix has fewer than 2048 tiles of the taller height."""
    want = {
        (1, "w"): (64, 32),            # 256 tiles of 128 x 32
        (2, "attn"): (64, 128),        # 1024 tiles of 128 x 128
        (3, "gate"): (128, 128), (3, "up"): (128, 128), (3, "down"): (128, 128),
        (4, "down"): (256, 256), (4, "up"): (256, 256),
    }
    for (cfg, name), shape in want.items():
        spec = {s.name: s for s in config_matrices(cfg)}[name]
        assert bench.v2_tiles(spec) == shape, (cfg, name)
    for spec in config_matrices(5, layers=[0]):
        short = spec.name.split(".")[-1]
        assert bench.v2_tiles(spec) == ((128, 256) if short in "qkvo" else (256, 256)), short
    # an explicit height keeps the width
    spec = config_matrices(4)[0]
    assert bench.v2_tiles(spec, 128) == (128, 256)
    assert bench.v2_tiles(config_matrices(2)[0], 128) == (128, 128)


def test_v2_tiles_hold_whole_chunks_of_state_bytes():
    """Every shape's width divides the chunk size, so the state bytes per
    code (one 4-byte state per row segment of TC codes) equal those of the
    chunk-sized tile the configuration names."""
    for cfg in (1, 2, 3, 4):
        for spec in config_matrices(cfg):
            tr, tc = bench.v2_tiles(spec)
            assert tr in (64, 128, 256) and tc % 4 == 0
            assert spec.chunk_syms % tc == 0
