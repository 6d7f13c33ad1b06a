"""Host check of the division constants the contraction kernels use for output-pixel
decoding: n / d == (mulhi(n, m) + n) >> l for every n < 2^31 (Granlund and Montgomery's
division by invariant integers).  Compiles the library's argument header with g++."""
import os
import shutil
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2307_04339_amd", "csrc")

SRC = r"""
#include <cstdio>
#include <cstdint>
#include <random>
#include "kargs.h"
using namespace miriam;
int main() {
    std::mt19937_64 rng(1);
    long bad = 0;
    auto check = [&](uint32_t d) {
        const FastDiv f = make_fastdiv(d);
        const uint32_t edge[] = {0u, 1u, d - 1, d, d + 1, 0x7ffffffeu, 0x7fffffffu};
        for (uint32_t n : edge)
            if (n <= 0x7fffffffu && fastdiv_host(n, f) != n / d) ++bad;
        for (int i = 0; i < 64; ++i) {
            const uint32_t n = (uint32_t)(rng() & 0x7fffffffu);
            if (fastdiv_host(n, f) != n / d) ++bad;
            const uint32_t m = (uint32_t)(rng() % 4096u) * d;  // multiples and their neighbours
            if (m <= 0x7fffffffu && fastdiv_host(m, f) != m / d) ++bad;
            if (m >= 1 && m - 1 <= 0x7fffffffu && fastdiv_host(m - 1, f) != (m - 1) / d) ++bad;
        }
    };
    for (uint32_t d = 1; d <= 20000; ++d) check(d);
    for (int i = 0; i < 20000; ++i) check((uint32_t)(rng() % 0x7fffffffu) + 1u);
    for (uint32_t k = 0; k < 31; ++k) { check(1u << k); check((1u << k) + 1u); if (k) check((1u << k) - 1u); }
    std::printf("bad %ld\n", bad);
    return bad != 0;
}
"""


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_fastdiv_constants_exact():
    with tempfile.TemporaryDirectory() as d:
        src = os.path.join(d, "fd.cpp")
        exe = os.path.join(d, "fd")
        with open(src, "w") as f:
            f.write(SRC)
        subprocess.run(["g++", "-O2", "-std=c++17", "-I", CSRC, src, "-o", exe], check=True)
        r = subprocess.run([exe], capture_output=True, text=True)
        assert r.returncode == 0, r.stdout + r.stderr
