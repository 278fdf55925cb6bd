"""The division the weight fake quantisation uses instead of one divide per element, checked on the CPU.

u = w / S_q (Eq. 7, 8) is formed from y = fl32(1 / S_q), one correctly rounded division per scale, by
q0 = fl(w y) and two corrections q <- fl(q - fl(q S_q - w) y), each residual one FMA (Markstein's
method). The library takes that path when 2^-40 <= S_q <= 2^40 and |w| <= 2^80. This test runs the
same five operations in C (gcc, libm's correctly rounded fmaf, no contraction) and checks:
  * every dividend of the binades whose quotient lies in [2^-5, 2^5), for divisors across the range
    (all-ones and all-zero significands included), against IEEE division bit for bit;
  * random dividends up to 2^80 against IEEE division bit for bit;
  * quotients below 2^-4 (dividends down to the smallest subnormal): below the smallest E2M1 midpoint
    0.25 and with the sign of the dividend, zeros keeping their sign.
"""
import os
import subprocess

import pytest

SRC = r"""
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>
static float f_of(uint32_t b) { float f; memcpy(&f, &b, 4); return f; }
static uint32_t b_of(float f) { uint32_t b; memcpy(&b, &f, 4); return b; }
static float quot(float a, float b, float y) {
    float q0 = a * y;
    float r0 = fmaf(q0, b, -a);
    float q1 = fmaf(-r0, y, q0);
    float r1 = fmaf(q1, b, -a);
    return fmaf(-r1, y, q1);
}
static uint64_t st = 88172645463325252ULL;
static uint64_t rnd(void) { st ^= st << 13; st ^= st >> 7; st ^= st << 17; return st; }
int main(void) {
    uint64_t bad = 0, n = 0, small = 0;
    for (int t = 0; t < 24; t++) {
        int e = -40 + (int)(rnd() % 81);
        uint32_t man = (uint32_t)rnd() & 0x7FFFFF;
        if (t == 0) man = 0x7FFFFF;
        if (t == 1) man = 0;
        if (t == 2) e = -40;
        if (t == 3) e = 39, man = 0x7FFFFF;
        float b = f_of(((uint32_t)(e + 127) << 23) | man), y = 1.0f / b;
        for (int ea = e - 5; ea <= e + 5; ea++)
            for (uint32_t m = 0; m < (1u << 23); m += 7) {
                float a = f_of(((uint32_t)(ea + 127) << 23) | m);
                n += 2;
                if (b_of(quot(a, b, y)) != b_of(a / b)) bad++;
                if (b_of(quot(-a, b, y)) != b_of(-a / b)) bad++;
            }
        for (int k = 0; k < 200000; k++) {
            uint32_t r = (uint32_t)rnd();
            float a = f_of((r & 0x80000000u) | (r & 0x7FFFFFFFu) % 0x67800001u);  /* |a| <= 2^80 */
            n++;
            float u = quot(a, b, y), ref = a / b;
            if (fabsf(ref) >= 0x1p-4f) { if (b_of(u) != b_of(ref)) bad++; }
            else {
                small++;
                if (!(fabsf(u) < 0.25f) || signbit(u) != signbit(a)) bad++;
            }
        }
        for (uint32_t m = 0; m < 4096; m++) {  /* the smallest dividends: subnormals and zeros */
            float a = f_of(m), u = quot(a, b, y), un = quot(-a, b, y);
            n += 2;
            if (!(fabsf(u) < 0.25f) || signbit(u) || !(fabsf(un) < 0.25f) || !signbit(un)) bad++;
        }
    }
    printf("%llu %llu %llu\n", (unsigned long long)n, (unsigned long long)bad, (unsigned long long)small);
    return 0;
}
"""


def test_markstein_quotient_matches_ieee_division(tmp_path):
    src = tmp_path / "quot.c"
    src.write_text(SRC)
    exe = tmp_path / "quot"
    r = subprocess.run(["gcc", "-O2", "-fno-fast-math", "-ffp-contract=off", str(src), "-o", str(exe), "-lm"],
                       capture_output=True, text=True)
    if r.returncode != 0:
        pytest.fail(r.stderr)
    out = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300, env=dict(os.environ))
    n, bad, small = map(int, out.stdout.split())
    assert n > 100_000_000 and small > 1000
    assert bad == 0
