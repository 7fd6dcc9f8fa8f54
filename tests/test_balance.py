"""Chunking of the residue classes for the backward's resident waves
(balance_chunks in csrc/mfpsn_internal.h), on the CPU: the host function is
compiled with g++ and driven over the workload shapes.

Checked: chunks are multiples of k within the offset cap and cover the
class; the items and the run bound follow from them; the chosen cut never
has a longer estimated wave range than the whole classes; the audio-spike
shape (250/d steps per class, 3 waves per SIMD, 384 waves per channel group)
is cut into 16-step chunks at d = 1 and 2 and keeps whole classes at d = 3;
shapes with many short classes per wave keep them whole.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2501_14490_amd", "csrc")

pytestmark = pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")

DRIVER = r"""
#include <cstdio>
#include <cstdlib>
#include "mfpsn_internal.h"
using namespace mfpsn;
int main(int argc, char** argv)
{
    // T d k tiles ncls cap waves
    Geom g{};
    g.T = atoi(argv[1]); g.d = atoi(argv[2]); g.k = atoi(argv[3]);
    g.tiles = atoi(argv[4]); g.ncls = atoi(argv[5]); g.cap = atoi(argv[6]);
    const long waves = atol(argv[7]);
    const long L = (g.T + g.d - 1) / g.d;
    g.chunk = (int)((L + g.k - 1) / g.k * g.k);
    if (g.chunk > g.cap) g.chunk = g.cap;
    g.nchunks = (int)((L + g.chunk - 1) / g.chunk);
    g.items = (long)g.tiles * g.ncls * g.nchunks;
    g.run_max = 1;
    balance_chunks(g, waves);
    printf("%d %d %lld %d\n", g.chunk, g.nchunks, (long long)g.items, g.run_max);
    return 0;
}
"""


@pytest.fixture(scope="module")
def driver(tmp_path_factory):
    tmp = tmp_path_factory.mktemp("balance")
    src = tmp / "drv.cpp"
    src.write_text(DRIVER)
    exe = tmp / "drv"
    subprocess.run(["g++", "-std=c++20", "-O1", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", f"-I{CSRC}",
                    str(src), "-o", str(exe)], check=True, capture_output=True)

    def run(T, d, k, tiles, ncls, cap, waves):
        out = subprocess.run([str(exe), *map(str, (T, d, k, tiles, ncls, cap, waves))], check=True,
                             capture_output=True, text=True).stdout.split()
        return tuple(int(v) for v in out)
    return run


def estimate(L, n, items, waves, k):
    return -(-items // waves) * (L / n) + (k - 1 if n > 1 else 0)


CASES = [
    # T, d, k, tiles, ncls, cap, waves per group
    (250, 1, 16, 256, 1, 1 << 20, 384),   # audio spike, d = 1
    (250, 2, 16, 256, 2, 1 << 20, 384),
    (250, 3, 16, 256, 3, 1 << 20, 384),
    (250, 4, 16, 256, 4, 1 << 20, 384),
    (30, 1, 8, 512, 1, 1 << 20, 64),      # event vision
    (30, 3, 8, 512, 3, 1 << 20, 64),
    (32, 1, 8, 32, 1, 1 << 20, 16),       # sequential image
    (4096, 1, 32, 16, 1, 512, 128),       # long fixed point, chunks capped
    (4096, 3, 32, 16, 3, 1024, 128),
    (1000, 7, 5, 3, 7, 1 << 20, 1000),    # more waves than work
    (1, 1, 4, 10, 1, 1 << 20, 64),
]


@pytest.mark.parametrize("T,d,k,tiles,ncls,cap,waves", CASES)
def test_balance_invariants(driver, T, d, k, tiles, ncls, cap, waves):
    chunk, n, items, run_max = driver(T, d, k, tiles, ncls, cap, waves)
    L = -(-T // d)
    assert chunk % k == 0 and k <= chunk <= max(cap, k)
    assert n == -(-L // chunk) and n * chunk >= L
    assert items == tiles * ncls * n
    assert run_max >= 1 and (run_max == 1 or run_max * chunk <= cap)
    whole = min(-(-L // k) * k, cap)
    nw = -(-L // whole)
    assert estimate(L, n, items, waves, k) <= estimate(L, nw, tiles * ncls * nw, waves, k) + 1e-9


def test_audio_spike_cuts(driver):
    assert driver(250, 1, 16, 256, 1, 1 << 20, 384)[0] == 16
    assert driver(250, 2, 16, 256, 2, 1 << 20, 384)[0] == 16
    assert driver(250, 3, 16, 256, 3, 1 << 20, 384)[:2] == (96, 1)


def test_many_short_classes_stay_whole(driver):
    assert driver(30, 1, 8, 512, 1, 1 << 20, 64)[:2] == (32, 1)
    assert driver(30, 3, 8, 512, 3, 1 << 20, 64)[:2] == (16, 1)
    assert driver(32, 1, 8, 32, 1, 1 << 20, 16)[:2] == (32, 1)
