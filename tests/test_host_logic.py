"""Host-side logic that needs no GPU."""
from test_gpu_parity import EXACT, RAGGED, _mirror_tile


def test_exact_shapes_cover_every_tile():
    fwd = {_mirror_tile(s.m, s.n) for s in EXACT}
    dx = {_mirror_tile(s.m, s.k) for s in EXACT}
    assert fwd == dx == {"256x256", "128x256", "128x128"}, (fwd, dx)


def test_ragged_shapes_have_tails():
    assert any(s.m % 64 for s in RAGGED) and any(s.k % 64 for s in RAGGED)
    assert any(s.n % 64 for s in RAGGED) and {1, 64} <= {s.r for s in RAGGED}
