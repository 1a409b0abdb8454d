/*
 * ltsynth.c -- seeded, counter-based synthetic inputs (weights and gradients)
 * for the optimizer step.  This module holds none of the optimizer's
 * arithmetic: it only draws numbers.  Both the CPU oracle's tests and the GPU
 * path receive the same bytes from it.
 *
 * Every value is a pure function of (seed, stream, tensor, element index), so
 * any slice of a tensor can be regenerated on its own and the thread count
 * never changes a bit.
 *
 * Generator: SplitMix64 (Steele, Lea and Flood, "Fast splittable
 * pseudorandom number generators", OOPSLA 2014), used as a counter-based
 * generator: output i of the sequence seeded with s is mix(s + (i+1)*golden).
 * A uniform takes 24 bits of one output plus one half, scaled into (0, 1).
 * Normal pairs use the Box-Muller transform in fp32 on two uniforms drawn from
 * output p of the sequence (bits 40..63 and 8..31).  Student-t with 3 degrees
 * of freedom is Z / sqrt(W / 3) with W = Z'^2 - 2 ln U a chi-square with 3
 * degrees of freedom (Z, Z' one Box-Muller pair, U an independent uniform).
 * Values are computed in fp32 (the normal tails end near 5.9 sigma), and bf16
 * outputs round that fp32 to bf16 (RNE).
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

#define GOLDEN 0x9E3779B97F4A7C15ull
#define TWO_PI_F 6.2831853071795865f

enum { LTS_F32 = 0, LTS_BF16 = 1 };
enum { LTS_NORMAL = 0, LTS_STUDENT_T3 = 1 };
enum { LTS_OUTLIER_NONE = 0, LTS_OUTLIER_SCALE = 1, LTS_OUTLIER_SET = 2 };

static inline uint64_t mix64(uint64_t z)
{
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

static inline uint64_t sm64_at(uint64_t state, uint64_t i)
{
    return mix64(state + (i + 1) * GOLDEN);
}

uint64_t lts_stream_key(uint64_t seed, uint64_t stream, uint64_t tensor)
{
    uint64_t k = sm64_at(seed, 0);
    k = sm64_at(k ^ stream, 0);
    return sm64_at(k ^ tensor, 0);
}

/* Uniform in (0, 1) from 24 bits of v starting at bit `shift`. */
static inline float u24(uint64_t v, int shift)
{
    return ((float)((v >> shift) & 0xFFFFFFu) + 0.5f) * 0x1.0p-24f;
}

static inline double u01(uint64_t key, uint64_t ctr)
{
    return ((double)(sm64_at(key, ctr) >> 11) + 0.5) * 0x1.0p-53;
}

static inline void normal_pair(uint64_t key, uint64_t pair, float* z0, float* z1)
{
    uint64_t h = sm64_at(key, pair);
    float r = sqrtf(-2.0f * logf(u24(h, 40)));
    float th = TWO_PI_F * u24(h, 8);
    *z0 = r * cosf(th);
    *z1 = r * sinf(th);
}

static inline uint16_t f32_to_bf16_rne(float f)
{
    uint32_t u;
    memcpy(&u, &f, 4);
    if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu)) /* NaN stays NaN */
        return (uint16_t)((u >> 16) | 0x40);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

/* Block-level zero mask: block b of the tensor is all zero when
 * sm64_at(key(seed, zero_stream, tensor), b) mod zero_mod == 0. */
int lts_block_is_zero(uint64_t seed, uint64_t zero_stream, uint64_t tensor, int64_t block,
                      int64_t zero_mod)
{
    return zero_mod > 0 &&
           sm64_at(lts_stream_key(seed, zero_stream, tensor), (uint64_t)block) % (uint64_t)zero_mod == 0;
}

/*
 * Fill elements [offset, offset + n) of one tensor.
 *   dist: LTS_NORMAL (value = scale * Z) or LTS_STUDENT_T3 (scale * t3).
 *   outliers: element i is an outlier when U(key(seed, stream + 1000, tensor), i)
 *     < outlier_p; LTS_OUTLIER_SCALE multiplies it by outlier_value,
 *     LTS_OUTLIER_SET replaces it by +-outlier_value (sign from the next counter).
 *   zero blocks: when zero_block > 0, blocks of zero_block elements selected by
 *     lts_block_is_zero(seed, zero_stream, tensor, b, zero_mod) are all zero.
 */
void lts_fill(void* out, int dtype, int64_t offset, int64_t n, uint64_t seed, uint64_t stream,
              uint64_t tensor, int dist, double scale, double outlier_p, int outlier_mode,
              double outlier_value, int64_t zero_block, uint64_t zero_stream, int64_t zero_mod,
              int n_threads)
{
    const uint64_t key = lts_stream_key(seed, stream, tensor);
    const uint64_t okey = lts_stream_key(seed, stream + 1000, tensor);
    const uint64_t zkey = lts_stream_key(seed, zero_stream, tensor);
    const uint64_t ckey = lts_stream_key(seed, stream + 2000, tensor);

#pragma omp parallel for schedule(static, 65536) num_threads(n_threads > 1 ? n_threads : 1)
    for (int64_t j = 0; j < n; ++j) {
        const uint64_t i = (uint64_t)(offset + j);
        double x;
        if (dist == LTS_STUDENT_T3) {
            float z, z1;
            normal_pair(key, i, &z, &z1);
            float chi3 = z1 * z1 - 2.0f * logf(u24(sm64_at(ckey, i), 40));
            x = (double)(z / sqrtf(chi3 / 3.0f));
        } else {
            float z0, z1;
            normal_pair(key, i >> 1, &z0, &z1);
            x = (double)((i & 1) ? z1 : z0);
        }
        x *= scale;
        if (outlier_mode != LTS_OUTLIER_NONE && u01(okey, 2 * i) < outlier_p) {
            if (outlier_mode == LTS_OUTLIER_SCALE)
                x *= outlier_value;
            else
                x = (sm64_at(okey, 2 * i + 1) & 1) ? -outlier_value : outlier_value;
        }
        if (zero_block > 0 && zero_mod > 0 &&
            sm64_at(zkey, i / (uint64_t)zero_block) % (uint64_t)zero_mod == 0)
            x = 0.0;
        float f = (float)x;
        if (dtype == LTS_BF16)
            ((uint16_t*)out)[j] = f32_to_bf16_rne(f);
        else
            ((float*)out)[j] = f;
    }
}
