"""The step kernel encodes a normalized moment with the dynamic code map by one
table read and one integer comparison: the fp32 pattern's exponent and top 7
mantissa bits pick a bucket whose entry holds the nearest code at the bucket's
lower end and the low 16 bits of the last pattern that keeps it; patterns above
that take the next code.  That is exact only if no bucket holds two decision
points of the map.  This test restates the procedure in C (it shares no code
with the HIP library or the oracle) and compares it with brute-force
nearest-code search over every code on every bucket's first and last value,
every code value and every midpoint between codes with their fp32 neighbours,
NaN, negatives and every 64th fp32 value in [0, 1 + 2^-23]; and with a local
search (binary search, then the two neighbours of the found code) on every fp32
value in [0, 1 + 2^-23], the domain of normalized moments."""
import os
import subprocess
import tempfile

SRC = r"""
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>
static float f_of(uint32_t u) { float f; memcpy(&f, &u, 4); return f; }
static uint32_t u_of(float f) { uint32_t u; memcpy(&u, &f, 4); return u; }
static const double P10[8] = {1.0, 1e-1, 1e-2, 1e-3, 1e-4, 1e-5, 1e-6, 1e-7};
static void build_map(int bits, float* t) {
    t[0] = 0.0f;
    for (int c = 1; c < (1 << bits); ++c) {
        int p = 31 - __builtin_clz((unsigned)c);
        int z = bits - 1 - p, f = c - (1 << p);
        t[c] = (float)((0.1 + 0.9 * ((double)(f + 1) / (double)(1 << p))) * P10[z]);
    }
    t[1 << bits] = INFINITY;
}
static int brute(const float* t, int n, float a) {
    int best = 0; float bd = fabsf(a - t[0]);
    for (int c = 1; c < n; ++c) { float d = fabsf(a - t[c]); if (d < bd) { bd = d; best = c; } }
    return best;
}
static int base_of(int bits) { return (127 - (bits == 7 ? 21 : 25)) << 7; }
static int top_of(int bits) { return (127 << 7) - base_of(bits); }
static uint32_t ENT[2][4096];
/* entry: code at the bucket's first pattern << 16 | last low half keeping it
   (the first low half where brute force moves on, minus one; 0xFFFF if none) */
/* nearest code by binary search for the largest t[c] <= a, then the better
   of c - 1, c, c + 1 by fp32 distance (ties to the smaller) */
static int local(const float* t, int n, float a) {
    if (!(a >= 0)) return 0;
    int lo = 0, hi = n - 1;
    while (lo < hi) { int mid = (lo + hi + 1) / 2; if (t[mid] <= a) lo = mid; else hi = mid - 1; }
    int best = lo > 0 ? lo - 1 : lo; float bd = fabsf(a - t[best]);
    for (int c = best + 1; c <= lo + 1 && c < n; ++c) {
        float d = fabsf(a - t[c]); if (d < bd) { bd = d; best = c; }
    }
    return best;
}
static void build_entries(int which, int bits, const float* t) {
    int n = 1 << bits;
    for (int i = 0; i <= top_of(bits); ++i) {
        uint32_t p0 = (uint32_t)(base_of(bits) + i) << 16;
        int c = brute(t, n, f_of(p0));
        uint32_t last = 0xFFFF;
        if (brute(t, n, f_of(p0 | 0xFFFF)) != c) {  /* first low half that moves on */
            uint32_t a = 1, b = 0xFFFF;
            while (a < b) { uint32_t m = (a + b) / 2; if (brute(t, n, f_of(p0 | m)) != c) b = m; else a = m + 1; }
            last = a - 1;
        }
        ENT[which][i] = ((uint32_t)c << 16) | last;
    }
    ENT[which][top_of(bits) + 1] = 0xFFFF;
}
static int bucket(int which, int bits, const float* t, float a) {
    (void)t;
    uint32_t u = u_of(a);
    int i = (int)(u >> 16) - base_of(bits);
    i = i < 0 ? 0 : (i > top_of(bits) + 1 ? top_of(bits) + 1 : i);
    uint32_t e = ENT[which][i];
    return (int)(e >> 16) + ((u & 0xFFFF) > (e & 0xFFFF));
}
static long bad = 0, checked = 0;
static const uint32_t ONE_PLUS = 0x3F800001u; /* 1 + 2^-23: the largest normalized value */
static void check(int which, int bits, const float* t, float a) {
    if (a == a && a > 0 && u_of(a) > ONE_PLUS) return; /* outside the domain */
    int want = brute(t, 1 << bits, a), got = bucket(which, bits, t, a);
    if (want != got) {
        if (bad < 10) printf("map %d a=%a: bucket %d brute %d\n", bits, a, got, want);
        ++bad;
    }
    ++checked;
}
int main(void) {
    static float tm[129], tv[257];
    build_map(7, tm); build_map(8, tv);
    build_entries(0, 7, tm); build_entries(1, 8, tv);
    for (int w = 0; w < 2; ++w) {
        int bits = w ? 8 : 7; const float* t = w ? tv : tm; int n = 1 << bits;
        for (int i = 0; i <= top_of(bits) + 1; ++i) {
            uint32_t u = (uint32_t)(base_of(bits) + i) << 16;
            check(w, bits, t, f_of(u)); check(w, bits, t, f_of(u - 1)); check(w, bits, t, f_of(u + 1));
        }
        for (int c = 0; c < n; ++c)
            for (int d = -2; d <= 2; ++d) {
                if (c == 0 && d < 0) continue;
                check(w, bits, t, f_of(u_of(t[c]) + d));
                if (c + 1 < n) {
                    float m = (float)(((double)t[c] + t[c + 1]) / 2);
                    check(w, bits, t, f_of(u_of(m) + d));
                }
            }
        check(w, bits, t, NAN); check(w, bits, t, -NAN); check(w, bits, t, -0.0f);
        check(w, bits, t, -1e-3f); check(w, bits, t, 1.0f + 0x1p-23f);
        long lb = 0, lc = 0;
        #pragma omp parallel for reduction(+:lb, lc) schedule(dynamic, 1 << 16)
        for (int64_t u = 0; u <= (int64_t)ONE_PLUS; u += 64) {
            float a = f_of((uint32_t)u);
            lb += bucket(w, bits, t, a) != brute(t, n, a);
            ++lc;
        }
        #pragma omp parallel for reduction(+:lb, lc) schedule(dynamic, 1 << 20)
        for (int64_t u = 0; u <= (int64_t)ONE_PLUS; ++u) {
            float a = f_of((uint32_t)u);
            lb += bucket(w, bits, t, a) != local(t, n, a);
            ++lc;
        }
        bad += lb; checked += lc;
    }
    printf("checked %ld mismatches %ld\n", checked, bad);
    return bad != 0;
}
"""


def test_bucket_encoder_equals_brute_force_nearest():
    with tempfile.TemporaryDirectory() as d:
        c = os.path.join(d, "enc.c")
        exe = os.path.join(d, "enc")
        open(c, "w").write(SRC)
        subprocess.run(["gcc", "-O2", "-ffp-contract=off", "-fopenmp", "-o", exe, c, "-lm"],
                       check=True)
        r = subprocess.run([exe], capture_output=True, text=True, timeout=900)
        assert r.returncode == 0, r.stdout + r.stderr
        assert "mismatches 0" in r.stdout
