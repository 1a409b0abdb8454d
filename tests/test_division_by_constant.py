"""The step kernel computes the dequantization steps A/127 and A/255 as the product
with the rounded reciprocal corrected once by its fma residual (zero, infinite and
NaN A take the plain product).  This test checks, for every one of the 2^32 fp32
bit patterns, that the sequence equals the correctly rounded quotient bit for bit
(NaN results compared as NaN), on the host's IEEE fma.  The sequence is restated
here in C; the test shares no code with the HIP library."""
import os
import subprocess
import tempfile

SRC = r"""
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>
static float bits_to_float(uint32_t u) { float f; memcpy(&f, &u, 4); return f; }
static uint32_t float_to_bits(float f) { uint32_t u; memcpy(&u, &f, 4); return u; }
static float divide(float a, float d, float c) {
    float q = a * c;
    if (a == 0.0f || !isfinite(a)) return q;
    float r = fmaf(-q, d, a);
    return fmaf(r, c, q);
}
int main(void) {
    const float ds[2] = {127.0f, 255.0f};
    const float cs[2] = {0x1.020408p-7f, 0x1.010102p-8f};
    long bad = 0;
    for (int i = 0; i < 2; ++i) {
        if (cs[i] != 1.0f / ds[i]) { printf("constant %d is not RN(1/d)\n", i); return 2; }
#pragma omp parallel for reduction(+:bad) schedule(static, 1 << 20)
        for (int64_t u = 0; u <= 0xFFFFFFFFll; ++u) {
            float a = bits_to_float((uint32_t)u);
            float want = a / ds[i], got = divide(a, ds[i], cs[i]);
            if (float_to_bits(want) != float_to_bits(got) && !(isnan(want) && isnan(got))) ++bad;
        }
    }
    printf("mismatches %ld\n", bad);
    return bad != 0;
}
"""


def test_constant_division_is_correctly_rounded_for_all_inputs():
    with tempfile.TemporaryDirectory() as d:
        c = os.path.join(d, "div.c")
        exe = os.path.join(d, "div")
        open(c, "w").write(SRC)
        subprocess.run(["gcc", "-O2", "-ffp-contract=off", "-fopenmp", "-o", exe, c, "-lm"],
                       check=True)
        r = subprocess.run([exe], capture_output=True, text=True, timeout=600)
        assert r.returncode == 0, r.stdout + r.stderr
        assert "mismatches 0" in r.stdout
