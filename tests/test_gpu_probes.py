"""The microbenchmarks of include/ml2_probe.h run on the GPU and report
plausible work and times (measurement helpers; their numbers are the
benchmark's, not a test's)."""
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
from paper_2411_10764_amd import ml2  # noqa: E402


@pytest.mark.parametrize("depth,G,S,waves,F", [
    (6, 8, 2, 8, 128), (8, 4, 2, 8, 128), (8, 2, 2, 8, 128), (8, 8, 2, 8, 64), (8, 8, 2, 4, 128),
    (8, 4, 1, 8, 64), (8, 8, 1, 8, 64), (6, 4, 2, 4, 64), (10, 2, 1, 8, 64), (10, 4, 1, 6, 64),
    (10, 1, 2, 8, 64), (10, 4, 2, 6, 64), (8, 8, 2, 6, 128)])
def test_visit_probe(depth, G, S, waves, F):
    ms, visits = ml2.ml2_probe_visit(depth, G, S, waves, F, 4, 8)
    assert visits == 8 * waves * (64 // S) * 4 * (G * S) * depth
    assert ms > 0.0


@pytest.mark.parametrize("mode", range(6))
def test_lds_probe(mode):
    ms, nbytes = ml2.ml2_probe_lds(mode, 8, 4)
    assert nbytes == 4 * 256 * 8 * 8 * (4 << (mode % 3))
    assert ms > 0.0


def test_valu_probe():
    ms, ops = ml2.ml2_probe_valu(8, 4)
    assert ops == 4 * 256 * 8 * 16 * 8
    assert ms > 0.0
