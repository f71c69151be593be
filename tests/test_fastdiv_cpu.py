"""The kernels divide work-item indices by launch constants with the host's
multiply-shift dividers (FastDiv in ws_kernels.h).  This compiles that header
with g++ and checks the quotient against plain division for every divisor
class the launches use and dividends up to the 2^31 bound."""
import os
import subprocess
import tempfile

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_25041_amd", "csrc")

PROGRAM = r"""
#include "ws_kernels.h"
#include <cstdio>
#include <cstdint>
#include <random>
#include <vector>
static uint32_t fd(uint32_t n, ws::FastDiv f) { return (uint32_t)(((uint64_t)n * f.mul) >> f.shift); }
int main() {
    std::mt19937_64 rng(12345);
    std::vector<uint32_t> ds;
    for (uint32_t d = 1; d <= 4096; ++d) ds.push_back(d);
    for (int k = 1; k < 31; ++k) { ds.push_back((1u << k) - 1); ds.push_back(1u << k); ds.push_back((1u << k) + 1); }
    for (int i = 0; i < 2000; ++i) ds.push_back(1 + (uint32_t)(rng() % 0x7FFFFFFEu));
    long bad = 0, checks = 0;
    for (uint32_t d : ds) {
        if (d == 0 || d >= 0x80000000u) continue;
        const ws::FastDiv f = ws::fastdiv_make(d);
        std::vector<uint32_t> ns = {0u, 1u, d - 1, d, d + 1, 2 * d - 1 < 0x80000000u ? 2 * d - 1 : 0u,
                                    0x7FFFFFFFu, 0x7FFFFFFEu, 0x40000000u};
        for (uint64_t m = 1; m * d < 0x80000000ull && ns.size() < 200; m = m * 3 + 1) {
            ns.push_back((uint32_t)(m * d - 1)); ns.push_back((uint32_t)(m * d));
        }
        for (int i = 0; i < 300; ++i) ns.push_back((uint32_t)(rng() % 0x80000000ull));
        for (uint32_t n : ns) {
            if (n >= 0x80000000u) continue;
            ++checks;
            if (fd(n, f) != n / d) { if (bad < 5) printf("d=%u n=%u got %u want %u\n", d, n, fd(n, f), n / d); ++bad; }
        }
    }
    printf("checks %ld bad %ld\n", checks, bad);
    return bad != 0;
}
"""


def test_fastdiv_matches_division():
    with tempfile.TemporaryDirectory() as tmp:
        src = os.path.join(tmp, "fd.cpp")
        exe = os.path.join(tmp, "fd")
        open(src, "w").write(PROGRAM)
        subprocess.run(["g++", "-O2", "-std=c++17", "-I", CSRC, src, "-o", exe], check=True)
        res = subprocess.run([exe], capture_output=True, text=True)
        assert res.returncode == 0, res.stdout + res.stderr
        assert "bad 0" in res.stdout
