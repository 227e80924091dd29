"""CPU check of the grid decode's division by launch constants: the
multiplier and shift that vx_fastdiv_make (csrc/vx_args.h) derives must give
x / d exactly as (mulhi32(x, m) + x) >> s -- the kernels' fdiv -- for every
0 <= x < 2^31.  Checked in C++ (g++, the header itself) on every divisor up to
70,000 with x at and around its multiples, plus random divisors and
dividends up to 2^31 - 1."""
import os
import subprocess

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

SRC = r"""
#include <stdio.h>
#include <stdlib.h>
#include "vx_args.h"
static unsigned apply(unsigned x, VxFastDiv f)
{
    return (unsigned)((((unsigned long long)x * f.m) >> 32) + x) >> f.s;
}
static unsigned long long rng = 88172645463325252ull;
static unsigned next(void) { rng ^= rng << 13; rng ^= rng >> 7; rng ^= rng << 17; return (unsigned)rng; }
int main(void)
{
    const unsigned top = 0x7fffffffu;
    long long checked = 0;
    for (unsigned d = 1; d <= 70000; ++d) {
        VxFastDiv f = vx_fastdiv_make(d);
        unsigned xs[] = {0, 1, d - 1, d, d + 1, 2 * d - 1, 2 * d, top, top - 1, top - d, top / d * d, top / d * d - 1};
        for (unsigned i = 0; i < sizeof xs / sizeof xs[0]; ++i) {
            unsigned x = xs[i] > top ? top : xs[i];
            if (apply(x, f) != x / d) { printf("FAIL d=%u x=%u\n", d, x); return 1; }
            ++checked;
        }
        for (int r = 0; r < 64; ++r) {
            unsigned q = next() % (top / d + 1), e = next() % 3;
            unsigned long long x = (unsigned long long)q * d + e;
            if (x > top) x = top;
            if (apply((unsigned)x, f) != (unsigned)x / d) { printf("FAIL d=%u x=%llu\n", d, x); return 1; }
            x = x ? x - 1 : 0;
            if (apply((unsigned)x, f) != (unsigned)x / d) { printf("FAIL d=%u x=%llu\n", d, x); return 1; }
            checked += 2;
        }
    }
    for (int r = 0; r < 2000000; ++r) {
        unsigned d = next() % top + 1, x = next() & top;
        VxFastDiv f = vx_fastdiv_make(d);
        if (apply(x, f) != x / d) { printf("FAIL d=%u x=%u\n", d, x); return 1; }
        unsigned y = x / d * d;
        if (apply(y, f) != y / d || (y && apply(y - 1, f) != (y - 1) / d)) { printf("FAIL d=%u y=%u\n", d, y); return 1; }
        checked += 3;
    }
    printf("OK %lld\n", checked);
    return 0;
}
"""


def test_fastdiv_multipliers_are_exact(tmp_path):
    c = tmp_path / "fd.cpp"
    c.write_text(SRC)
    exe = tmp_path / "fd"
    subprocess.run(["g++", "-O2", "-x", "c++", "-I", os.path.join(ROOT, "paper_2409_01075_amd", "csrc"),
                    "-o", str(exe), str(c)], check=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert out.returncode == 0 and out.stdout.startswith("OK"), out.stdout
