"""The microbenchmarks of include/ml2_probe.h run on the GPU and report
plausible work and times (measurement helpers; their numbers are the
benchmark's, not a test's)."""
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
from paper_2411_10764_amd import ml2  # noqa: E402


@pytest.mark.parametrize("depth", [6, 8])
def test_visit_probe(depth):
    ms, visits = ml2.ml2_probe_visit(depth, 4, 8)
    G = 8 if depth == 6 else 4
    assert visits == 8 * 8 * 32 * 4 * (2 * G) * depth
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
