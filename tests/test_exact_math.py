"""Host check of the library's exact ceil(x * a / d) helper (fp64 estimate
plus exact correction) against 128-bit integer division, on random and edge
operands across its documented range, on both of its paths (products below
2^53 and above) and around the boundary between them. CPU only."""
import os
import subprocess

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

DRIVER = r'''
#include <stdio.h>
#include <stdlib.h>
#include "exact_math.h"
typedef unsigned __int128 u128;
static uint64_t rnd(uint64_t *s) { *s ^= *s << 13; *s ^= *s >> 7; *s ^= *s << 17; return *s; }
static int check(uint64_t x, uint64_t a, uint64_t d) {
    u128 n = (u128)x * a;
    uint64_t want = (uint64_t)((n + d - 1) / d);
    uint64_t got = heddle::ceil_muldiv(x, a, d);
    if (got != want) { printf("MISMATCH x=%llu a=%llu d=%llu got=%llu want=%llu\n",
        (unsigned long long)x, (unsigned long long)a, (unsigned long long)d,
        (unsigned long long)got, (unsigned long long)want); return 1; }
    return 0;
}
int main(void) {
    uint64_t s = 88172645463325252ull; int bad = 0; long n = 0;
    const uint64_t XM = (1ull << 51) - 1, AM = (1ull << 28) - 1, DM = (1ull << 50) - 1;
    uint64_t xs[] = {0, 1, 2, 3, 999, 1000, (1ull<<24)+1, (1ull<<32)-1, 1ull<<40, XM, XM-1, 123456789012345ull};
    uint64_t as[] = {1, 2, 1000, 2000, 131068000ull, AM};
    uint64_t ds[] = {1, 2, 3, 7, 1000, 25000, 400000, (1ull<<32)+1, 1ull<<49, DM, DM-2, 65535ull*17179869183ull};
    for (int i = 0; i < 12; i++) for (int j = 0; j < 6; j++) for (int k = 0; k < 12; k++) {
        u128 q = ((u128)xs[i] * as[j] + ds[k] - 1) / ds[k];
        if (q >= ((u128)1 << 62)) continue;            /* outside the documented result range */
        bad += check(xs[i], as[j], ds[k]); n++;
    }
    for (long t = 0; t < 3000000; t++) {
        uint64_t x = rnd(&s) & XM, a = (rnd(&s) & AM) | 1, d = (rnd(&s) >> (rnd(&s) % 63)) & DM;
        if (d == 0) d = 1 + (rnd(&s) & 0xFFFF);
        if (t % 3 == 0) x >>= rnd(&s) % 50;
        u128 q = ((u128)x * a + d - 1) / d;
        if (q >= ((u128)1 << 62)) continue;
        bad += check(x, a, d); n++;
        if (bad > 5) break;
    }
    /* products below 2^53 (the one-division path) and around that boundary */
    for (long t = 0; t < 2000000 && bad <= 5; t++) {
        uint64_t a = (rnd(&s) & AM) | 1, d = (rnd(&s) >> (rnd(&s) % 63)) & DM;
        if (d == 0) d = 1 + (rnd(&s) & 0xFFFF);
        uint64_t lim = ((1ull << 53) - d) / a;                 /* x * a + d - 1 < 2^53 */
        uint64_t x = lim ? rnd(&s) % (lim + 1) : 0;
        if (t % 4 == 0) x = lim;
        if (t % 4 == 1 && x > 0) x = rnd(&s) % (x >> (rnd(&s) % 40) | 1);
        if (x > XM) continue;
        bad += check(x, a, d); n++;
    }
    for (uint64_t dd = 1; dd < 40 && bad <= 5; dd++) {
        const uint64_t d = dd * 977 + (dd & 1);
        for (int64_t off = -3; off <= 3; off++) {
            const uint64_t target = (1ull << 53) + off;          /* n = x * a + d - 1 near 2^53 */
            if (target < d - 1) continue;
            bad += check(target - (d - 1), 1, d); n++;
        }
    }
    printf("checked %ld bad %d\n", n, bad);
    return bad != 0;
}
'''


def test_ceil_muldiv_exact(tmp_path):
    src = tmp_path / "drv.cpp"
    src.write_text(DRIVER)
    exe = tmp_path / "drv"
    inc = os.path.join(ROOT, "paper_2609_34244_amd", "csrc")
    r = subprocess.run(["g++", "-O2", "-std=c++17", "-I", inc, "-o", str(exe), str(src)], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([str(exe)], capture_output=True, text=True)
    assert r.returncode == 0, r.stdout
    assert "bad 0" in r.stdout
