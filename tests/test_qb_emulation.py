"""Host emulation of the receiver's bucketed query: the kernels' own source
(k_qb_count, k_qb_scan, k_qb_scatter, k_qb_test, k_qb_fill and the record
reader they use, cut out of bloom.hip) compiled by g++ for the CPU against a
small stand-in for the HIP device runtime (tests/emu: every thread of a
block is a std::thread, __syncthreads a block barrier, the wave intrinsics
exchanges through a per-wave buffer), with AddressSanitizer and UBSan.  The
driver launches the kernels in the launcher's order, block by block, with
every buffer a heap allocation of exactly the size the host plans, and
compares the positives bitmap with a direct query.  A load or store outside
a buffer, a barrier some threads never reach (reported after 30 s), or a
wrong bitmap fails the test.  Host code only: no GPU."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2102_03112_amd", "csrc")
EMU = os.path.join(ROOT, "tests", "emu")


def _section(lines, start, end):
    a = next(i for i, l in enumerate(lines) if l.startswith(start))
    b = next(i for i, l in enumerate(lines) if i > a and l.startswith(end))
    # from the rule line above the section's title to the line before the next
    return "".join(lines[a - 1:b - 1])


@pytest.fixture(scope="module")
def emulator(tmp_path_factory):
    gxx = shutil.which("g++")
    if not gxx:
        pytest.skip("g++ not found")
    d = tmp_path_factory.mktemp("qb_emu")
    lines = open(os.path.join(CSRC, "bloom.hip")).readlines()
    (d / "ext_query.inc").write_text(_section(lines, "// Full-range query", "// Probe pass: the positives"))
    (d / "ext_qb.inc").write_text(_section(lines, "// Bucketed query", "// The received value of a positive"))
    exe = d / "qb_emu"
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
           f"-I{d}", f"-I{EMU}", f"-I{CSRC}", "-o", str(exe), os.path.join(EMU, "qb_emu.cpp"),
           os.path.join(EMU, "emu_rt.cpp"), "-lpthread"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    return str(exe)


CASES = [
    # d, items, m (bits), k, layout: one slice, chunk and region
    (36_864, 369, 5_312, 10, 0),
    (36_864, 369, 5_312, 10, 1),
    # three slices (the last one partial), two regions (the last one
    # partial), 17 chunks
    (530_001, 120_000, 1_050_016, 2, 0),
    # more slices (4) than round 0 has chunks (2): the count table is as
    # wide as the slices
    (40_000, 30_000, 3 * (1 << 19) + 1024, 3, 0),
]


@pytest.mark.parametrize("d,n,m,k,layout", CASES)
def test_bucketed_query_on_the_host(emulator, d, n, m, k, layout):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0")
    r = subprocess.run([emulator, str(d), str(n), str(m), str(k), str(layout)], capture_output=True, text=True,
                       timeout=600, env=env)
    assert r.returncode == 0, (r.stdout + r.stderr)[-3000:]
    assert r.stdout.startswith("OK"), r.stdout
