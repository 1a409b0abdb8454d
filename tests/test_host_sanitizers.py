"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer, without a GPU.

The oracle and the synthetic-input generator (gcc) are driven through every entry
point on ragged sizes, both gradient dtypes, both code maps, one and four threads,
the non-finite skip and the zero block.  The HIP library is rebuilt with the
sanitizers on its host half only and driven through its host-only entry points and
its argument checks (tests/sanitize_abi_driver.cpp).  Any out-of-bounds access,
leak or undefined operation fails the run."""
import glob
import os
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

DRIVER = r"""
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>
#include "lazytrain_oracle.h"
void lts_fill(void* out, int dtype, int64_t offset, int64_t n, uint64_t seed, uint64_t stream,
              uint64_t tensor, int dist, double scale, double outlier_p, int outlier_mode,
              double outlier_value, int64_t zero_block, uint64_t zero_stream, int64_t zero_mod,
              int n_threads);
int lts_block_is_zero(uint64_t seed, uint64_t zero_stream, uint64_t tensor, int64_t block,
                      int64_t zero_mod);
enum { K = 5 };
static const int64_t N[K] = {1, 7, 8193, 2049, 70001};

int main(void) {
    for (int gdt = 0; gdt < 2; ++gdt)
    for (int map = 0; map < 2; ++map)
    for (int threads = 1; threads <= 4; threads += 3)
    for (int64_t B = 64; B <= 4096; B *= 8) {
        float* w[K]; void* g[K]; int8_t* mq[K]; uint8_t* vq[K]; float* ma[K]; float* va[K];
        for (int k = 0; k < K; ++k) {
            int64_t nb = (N[k] + B - 1) / B;
            w[k] = malloc(N[k] * 4); g[k] = malloc(N[k] * (gdt ? 2 : 4));
            mq[k] = calloc(N[k], 1); vq[k] = calloc(N[k], 1);
            ma[k] = calloc(nb, 4); va[k] = calloc(nb, 4);
            lts_fill(w[k], 0, 0, N[k], 3, 0, k, 0, 0.02, 0, 0, 0, 0, 101, 0, threads);
            lts_fill(g[k], gdt, 0, N[k], 3, 2, k, 1, 1e-3, 0.01, 1, 100.0, 256, 101, 8, threads);
        }
        double sk[K], S; int32_t st;
        if (lto_grad_sqnorm((const void* const*)g, N, K, gdt, sk, &S, &st, threads)) return 1;
        double naive = lto_grad_sqnorm_naive((const void* const*)g, N, K, gdt);
        if (fabs(naive - S) > 1e-9 * S) { printf("sum mismatch\n"); return 1; }
        float norm, coef;
        lto_clip_coef(S, 1.0f, &norm, &coef);
        for (int t = 1; t <= 2; ++t)
            if (lto_hybrid8bit_adamw_step(w, (const void* const*)g, gdt, mq, ma, vq, va, N, K, B,
                                          map, 1e-4, 0.9, 0.999, 1e-8, 0.01, t, &coef, &st,
                                          threads)) return 1;
        int32_t skip = LTO_STATUS_NONFINITE;
        lto_hybrid8bit_adamw_step(w, (const void* const*)g, gdt, mq, ma, vq, va, N, K, B, map,
                                  1e-4, 0.9, 0.999, 1e-8, 0.01, 3, NULL, &skip, threads);
        float* m32 = calloc(N[K - 1], 4); float* v32 = calloc(N[K - 1], 4);
        lto_adamw_fp32_step(w[K - 1], g[K - 1], gdt, m32, v32, N[K - 1], 1e-4, 0.9, 0.999, 1e-8,
                            0.01, 1, coef);
        uint16_t* b16 = malloc(N[K - 1] * 2);
        lto_round_bf16(w[K - 1], N[K - 1], b16);
        for (int k = 0; k < K; ++k) {
            free(w[k]); free(g[k]); free(mq[k]); free(vq[k]); free(ma[k]); free(va[k]);
        }
        free(m32); free(v32); free(b16);
    }
    /* block quantizers on edge blocks: zero, tiny, infinite, NaN */
    float x[5] = {0, 0, 0, 0, 0}, back[5];
    int8_t q[5]; uint8_t u[5]; float A;
    lto_quantize_signed(x, 5, q, &A); lto_dequantize_signed(q, 5, A, back);
    lto_quantize_dynamic_signed(x, 5, q, &A); lto_dequantize_dynamic_signed(q, 5, A, back);
    x[2] = INFINITY; x[3] = NAN; x[4] = 1e-39f;
    lto_quantize_unsigned(x, 5, u, &A); lto_dequantize_unsigned(u, 5, A, back);
    lto_quantize_dynamic_unsigned(x, 5, u, &A); lto_dequantize_dynamic_unsigned(u, 5, A, back);
    float tm[128], tv[256];
    lto_dynamic_map(1, tm); lto_dynamic_map(0, tv);
    lto_scalars sc;
    lto_step_scalars(1e-4, 0.9, 0.999, 1e-8, 0.01, 7, &sc);
    printf("sanitized run ok\n");
    return 0;
}
"""


def test_oracle_and_generator_under_asan_and_ubsan():
    with tempfile.TemporaryDirectory() as d:
        c = os.path.join(d, "drv.c")
        exe = os.path.join(d, "drv")
        open(c, "w").write(DRIVER)
        cmd = ["gcc", "-O1", "-g", "-fno-omit-frame-pointer", "-ffp-contract=off",
               "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fopenmp",
               "-I", os.path.join(ROOT, "oracle"), "-o", exe, c,
               os.path.join(ROOT, "oracle", "lazytrain_oracle.c"),
               os.path.join(ROOT, "synth", "ltsynth.c"), "-lm"]
        subprocess.run(cmd, check=True)
        env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
                   UBSAN_OPTIONS="print_stacktrace=1")
        r = subprocess.run([exe], capture_output=True, text=True, timeout=600, env=env)
        assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
        assert "sanitized run ok" in r.stdout


def _clang_rt_dir():
    dirs = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux"))
    return dirs[-1] if dirs else None


@pytest.mark.skipif(_clang_rt_dir() is None, reason="no clang sanitizer runtime")
def test_library_host_code_under_asan_and_ubsan():
    from paper_2608_11919_amd import build as lib_build
    rt = _clang_rt_dir()
    with tempfile.TemporaryDirectory() as d:
        so = os.path.join(d, "liblazytrain_asan.so")
        flags = [f for f in lib_build.HIPCC_FLAGS if f != "-O3"]
        cmd = [lib_build.hipcc()] + flags + [
            "-O1", "-g", "-Xarch_host", "-fsanitize=address", "-Xarch_host",
            "-fsanitize=undefined", "-Xarch_host", "-shared-libsan",
            "-I", os.path.join(ROOT, "include"), "-o", so] + lib_build.SOURCES
        subprocess.run(cmd, check=True, capture_output=True)
        exe = os.path.join(d, "drv")
        clang = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "llvm", "bin", "clang++")
        subprocess.run([clang, "-g", "-std=c++17", "-fsanitize=address,undefined",
                        "-shared-libsan", "-I", os.path.join(ROOT, "include"), "-o", exe,
                        os.path.join(ROOT, "tests", "sanitize_abi_driver.cpp"), so,
                        f"-Wl,-rpath,{d}", f"-Wl,-rpath,{rt}"], check=True)
        env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1", UBSAN_OPTIONS="print_stacktrace=1")
        r = subprocess.run([exe], capture_output=True, text=True, timeout=300, env=env)
        assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-3000:]
        assert "0 failures" in r.stdout
