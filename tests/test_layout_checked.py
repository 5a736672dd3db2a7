"""The checked host build of the tree packing.

`paper_2411_10764_amd/csrc/pack.cpp` (the host code that writes the device
layout the walk kernels read) is compiled on its own with -DML2_CHECKED,
which checks every byte it writes against its record or chunk slot and
every encoded field against its bits, under the address and
undefined-behaviour sanitizers.  `tests/layout_check_driver.cpp` packs
random trees (perfect records of depth 1 to 12, ragged slots with default
directions, chains of depth 32, the largest trees a slot holds, 1 to 256
features) and walks every packed tree with the kernels' index arithmetic,
checking each address, feature index, header field and leaf hand-over, and
that each walk ends on the unpacked tree's leaf, bit for bit.  Its corrupt
mode damages packed bytes and must see every case rejected.
"""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(ROOT, "paper_2411_10764_amd", "csrc")


@pytest.fixture(scope="module")
def driver(tmp_path_factory):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not available")
    exe = str(tmp_path_factory.mktemp("layout") / "layout_check_driver")
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=all", "-DML2_CHECKED", "-Wall", "-Werror", "-I", CSRC,
           os.path.join(HERE, "layout_check_driver.cpp"), os.path.join(CSRC, "pack.cpp"),
           "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stdout + r.stderr
    return exe


def _run(exe, *args):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    return subprocess.run([exe, *args], capture_output=True, text=True, timeout=300, env=env)


def test_packed_layout_walks_in_bounds(driver):
    r = _run(driver)
    assert r.returncode == 0, r.stdout + r.stderr
    lines = r.stdout.strip().splitlines()
    assert len(lines) == 10 and all(line.startswith("ok ") for line in lines), r.stdout
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, r.stderr


def test_damaged_layout_is_rejected(driver):
    r = _run(driver, "corrupt")
    assert r.returncode == 0, r.stdout + r.stderr
    assert "corruption detected in every case" in r.stdout
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, r.stderr
