/*
 * lazytrain_oracle.c -- TEST INFRASTRUCTURE: the CPU definition of the
 * Hybrid 8-bit operator's optimizer step (paper Sec. 3.5, Hybrid 8-bit
 * operator paragraph; App. C training-configuration and variant tables).
 *
 * Written for reading, not for speed: plain loops, one element at a time, in
 * the order the definition states.  Build with -ffp-contract=off and without
 * -ffast-math so that every written operation is one IEEE rounding.
 * See lazytrain_oracle.h for the contract of each function.
 */
#include "lazytrain_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

/* ---------------------------------------------------------------- inputs */

static float bf16_bits_to_float(uint16_t h)
{
    uint32_t u = (uint32_t)h << 16; /* bf16 is the top half of an fp32 */
    float f;
    memcpy(&f, &u, sizeof f);
    return f;
}

static float grad_value(const void* g, int gdt, int64_t i)
{
    if (gdt == LTO_BF16)
        return bf16_bits_to_float(((const uint16_t*)g)[i]);
    return ((const float*)g)[i];
}

/* ------------------------------------------------- sum of squares (a1-a2) */

/* Sum of squares of chunk c of one tensor (n elements), fixed order.  Part of
 * the per-tensor norm of Sec. 3.5's clipping path; the chunk and lane order is
 * this implementation's reading, since the paper fixes no order. */
static double chunk_sum_of_squares(const void* g, int gdt, int64_t n, int64_t c)
{
    const int64_t base = c * LTO_CHUNK;
    double lane_sum[LTO_LANES];

    /* Lane sums: lane l visits its four 8-element granules in order. */
    for (int lane = 0; lane < LTO_LANES; ++lane) {
        double a = 0.0;
        for (int r = 0; r < 4; ++r) {
            for (int e = 0; e < 8; ++e) {
                int64_t idx = base + 8 * ((int64_t)lane + (int64_t)LTO_LANES * r) + e;
                if (idx < n) { /* positions past the end count as zero */
                    double x = (double)grad_value(g, gdt, idx);
                    a = a + x * x; /* the square is exact in fp64 */
                }
            }
        }
        lane_sum[lane] = a;
    }

    /* Halving tree inside each group of 64 lanes. */
    double W[4];
    for (int w = 0; w < 4; ++w) {
        double t[64];
        for (int i = 0; i < 64; ++i)
            t[i] = lane_sum[64 * w + i];
        for (int o = 32; o >= 1; o /= 2)
            for (int i = 0; i < o; ++i)
                t[i] = t[i] + t[i + o];
        W[w] = t[0];
    }
    return (W[0] + W[2]) + (W[1] + W[3]);
}

/* The per-tensor norm of Sec. 3.5, as its square: chunk partials combined in a
 * fixed order. */
static double tensor_sum_of_squares(const void* g, int gdt, int64_t n, int n_threads)
{
    const int64_t n_chunks = (n + LTO_CHUNK - 1) / LTO_CHUNK;
    double* P = (double*)malloc((size_t)(n_chunks > 0 ? n_chunks : 1) * sizeof(double));

#pragma omp parallel for schedule(static) num_threads(n_threads > 1 ? n_threads : 1)
    for (int64_t c = 0; c < n_chunks; ++c)
        P[c] = chunk_sum_of_squares(g, gdt, n, c);

    /* Chunk partials round-robin into 256 accumulators, ascending chunk. */
    double b[LTO_LANES];
    for (int t = 0; t < LTO_LANES; ++t)
        b[t] = 0.0;
    for (int64_t c = 0; c < n_chunks; ++c)
        b[c % LTO_LANES] = b[c % LTO_LANES] + P[c];
    for (int o = LTO_LANES / 2; o >= 1; o /= 2)
        for (int t = 0; t < o; ++t)
            b[t] = b[t] + b[t + o];

    free(P);
    return b[0];
}

/* Sec. 3.5: one global norm aggregated from the per-tensor norms; App. C
 * safety-checks row: non-finite gradients are detected (here, as the status). */
int lto_grad_sqnorm(const void* const* grads, const int64_t* numels, int n_tensors, int gdt,
                    double* sq_per_tensor, double* sq_total, int32_t* status, int n_threads)
{
    if (n_tensors < 0 || (n_tensors > 0 && (!grads || !numels)) || !sq_total || !status ||
        (gdt != LTO_F32 && gdt != LTO_BF16))
        return LTO_ERR_INVALID_ARG;

    double S = 0.0;
    for (int k = 0; k < n_tensors; ++k) {
        double Sk = tensor_sum_of_squares(grads[k], gdt, numels[k], n_threads);
        if (sq_per_tensor)
            sq_per_tensor[k] = Sk;
        S = S + Sk; /* list order */
    }
    *sq_total = S;
    *status = isfinite(S) ? LTO_STATUS_OK : LTO_STATUS_NONFINITE;
    return LTO_OK;
}

/* Not from the paper: the plain definition of the sum of squares, used as a pin. */
double lto_grad_sqnorm_naive(const void* const* grads, const int64_t* numels, int n_tensors,
                             int gdt)
{
    double s = 0.0;
    for (int k = 0; k < n_tensors; ++k)
        for (int64_t i = 0; i < numels[k]; ++i) {
            double x = (double)grad_value(grads[k], gdt, i);
            s = s + x * x;
        }
    return s;
}

/* ----------------------------------------------------- clip coefficient (a3) */

/* Sec. 3.5: one scale applied to all gradients; App. C: max grad norm.  The
 * formula is the usual clip-by-global-norm rule with a 1e-6 guard. */
void lto_clip_coef(double sq_total, float max_norm, float* total_norm, float* coef)
{
    float norm = (float)sqrt(sq_total);
    float c = max_norm / (norm + 1e-6f);
    *total_norm = norm;
    *coef = fminf(1.0f, c);
}

/* --------------------------------------------------- block quantizer (a8-a9) */

static float clampf(float x, float lo, float hi)
{
    return fminf(fmaxf(x, lo), hi);
}

/* Sec. 3.5: block-wise 8-bit states with a scale per block.  The linear absmax
 * code is a reading (the paper names no code map); this is the first moment's. */
void lto_quantize_signed(const float* x, int64_t n, int8_t* q, float* absmax)
{
    float A = 0.0f;
    for (int64_t i = 0; i < n; ++i)
        A = fmaxf(A, fabsf(x[i]));
    float inv = 127.0f / A;
    int ok = isfinite(A) && isfinite(inv);
    for (int64_t i = 0; i < n; ++i)
        q[i] = ok ? (int8_t)clampf(rintf(x[i] * inv), -127.0f, 127.0f) : (int8_t)0;
    *absmax = ok ? A : 0.0f;
}

/* As above, for the second moment (non-negative): 255 levels. */
void lto_quantize_unsigned(const float* x, int64_t n, uint8_t* q, float* absmax)
{
    float A = 0.0f;
    for (int64_t i = 0; i < n; ++i)
        A = fmaxf(A, x[i]);
    float inv = 255.0f / A;
    int ok = isfinite(A) && isfinite(inv);
    for (int64_t i = 0; i < n; ++i)
        q[i] = ok ? (uint8_t)clampf(rintf(x[i] * inv), 0.0f, 255.0f) : (uint8_t)0;
    *absmax = ok ? A : 0.0f;
}

/* The inverse maps of the two linear codes (Sec. 3.5: dequantization). */
void lto_dequantize_signed(const int8_t* q, int64_t n, float absmax, float* x)
{
    float step = absmax / 127.0f;
    for (int64_t i = 0; i < n; ++i)
        x[i] = (float)q[i] * step;
}

void lto_dequantize_unsigned(const uint8_t* q, int64_t n, float absmax, float* x)
{
    float step = absmax / 255.0f;
    for (int64_t i = 0; i < n; ++i)
        x[i] = (float)q[i] * step;
}

/* ------------------------------------------------- dynamic code map (f2) */

/* Powers of ten of the map's decades, as correctly rounded double literals. */
static const double pow10_neg[8] = {1.0, 1e-1, 1e-2, 1e-3, 1e-4, 1e-5, 1e-6, 1e-7};

/* The dynamic tree code map (a second reading of Sec. 3.5's 8-bit states,
 * after Dettmers et al.'s block-wise 8-bit optimizers): magnitudes by decade. */
void lto_dynamic_map(int is_signed, float* table)
{
    const int bits = is_signed ? 7 : 8; /* magnitude bits of a code */
    const int n = 1 << bits;
    table[0] = 0.0f;
    for (int c = 1; c < n; ++c) {
        int p = 0; /* position of the leading one: p fraction bits follow it */
        while ((c >> (p + 1)) != 0)
            ++p;
        const int zeros = bits - 1 - p; /* leading zero bits: the decade */
        const int f = c - (1 << p);      /* the fraction bits */
        const double frac = 0.1 + 0.9 * ((double)(f + 1) / (double)(1 << p));
        table[c] = (float)(frac * pow10_neg[zeros]);
    }
}

/* The code whose magnitude is nearest to a: the smallest c with the least
 * fabsf(a - table[c]) (a NaN a gives 0). */
static int nearest_code(const float* table, int n, float a)
{
    int best = 0;
    float bd = fabsf(a - table[0]);
    for (int c = 1; c < n; ++c) {
        const float d = fabsf(a - table[c]);
        if (d < bd) {
            bd = d;
            best = c;
        }
    }
    return best;
}

void lto_quantize_dynamic_signed(const float* x, int64_t n, int8_t* q, float* absmax)
{
    float T[128];
    lto_dynamic_map(1, T);
    float A = 0.0f;
    for (int64_t i = 0; i < n; ++i)
        A = fmaxf(A, fabsf(x[i]));
    const float inv = 1.0f / A;
    const int ok = isfinite(A) && isfinite(inv);
    for (int64_t i = 0; i < n; ++i) {
        int c = ok ? nearest_code(T, 128, fabsf(x[i]) * inv) : 0;
        if (ok && x[i] < 0.0f)
            c |= 0x80; /* sign-magnitude byte: the sign of x, also on magnitude 0 */
        q[i] = (int8_t)(uint8_t)c;
    }
    *absmax = ok ? A : 0.0f;
}

void lto_quantize_dynamic_unsigned(const float* x, int64_t n, uint8_t* q, float* absmax)
{
    float U[256];
    lto_dynamic_map(0, U);
    float A = 0.0f;
    for (int64_t i = 0; i < n; ++i)
        A = fmaxf(A, x[i]);
    const float inv = 1.0f / A;
    const int ok = isfinite(A) && isfinite(inv);
    for (int64_t i = 0; i < n; ++i)
        q[i] = ok ? (uint8_t)nearest_code(U, 256, x[i] * inv) : (uint8_t)0;
    *absmax = ok ? A : 0.0f;
}

void lto_dequantize_dynamic_signed(const int8_t* q, int64_t n, float absmax, float* x)
{
    float T[128];
    lto_dynamic_map(1, T);
    for (int64_t i = 0; i < n; ++i) {
        const uint8_t b = (uint8_t)q[i];
        const float mag = T[b & 0x7F];
        x[i] = ((b & 0x80) ? -mag : mag) * absmax;
    }
}

void lto_dequantize_dynamic_unsigned(const uint8_t* q, int64_t n, float absmax, float* x)
{
    float U[256];
    lto_dynamic_map(0, U);
    for (int64_t i = 0; i < n; ++i)
        x[i] = U[q[i]] * absmax;
}

/* --------------------------------------------------------- AdamW step (a4-a10) */

/* App. C optimizer-hyperparameters row (beta1, beta2, eps, learning rate,
 * weight decay): the per-step scalars of Adam with bias correction and
 * decoupled weight decay (AdamW), each rounded once to fp32. */
void lto_step_scalars(double lr, double beta1, double beta2, double eps, double weight_decay,
                      int64_t step, lto_scalars* out)
{
    double t = (double)step;
    double bias1 = 1.0 - pow(beta1, t);
    double bias2 = 1.0 - pow(beta2, t);
    out->beta1 = (float)beta1;
    out->beta2 = (float)beta2;
    out->eps = (float)eps;
    out->c1 = (float)(1.0 - beta1);
    out->c2 = (float)(1.0 - beta2);
    out->decay = (float)(1.0 - lr * weight_decay);
    out->step_size = (float)(lr / bias1);
    out->rbc2 = (float)(1.0 / sqrt(bias2));
}

typedef struct {
    lto_scalars h;
    float coef;
} adamw_scalars;

/* AdamW on one element with fp32 moments m0, v0; returns m1, v1 and the new
 * weight.  Decoupled weight decay, bias corrections of the 1-based step. */
static void adamw_element(const adamw_scalars* s, float m0, float v0, float grad, float w,
                          float* m1, float* v1, float* w1)
{
    const lto_scalars* h = &s->h;
    float g = grad * s->coef;
    float m = fmaf(h->beta1, m0, h->c1 * g);
    float v = fmaf(h->beta2, v0, h->c2 * (g * g));
    float d = fmaf(sqrtf(v), h->rbc2, h->eps);
    *w1 = fmaf(-h->step_size, m / d, w * h->decay);
    *m1 = m;
    *v1 = v;
}

/* One quantization block: elements [off, off + len) of a tensor; *am, *av are
 * this block's stored scales.  Sec. 3.5: dequantize the 8-bit states, update
 * them and the fp32 master weights, requantize with new block scales. */
static void step_block(const adamw_scalars* s, int code_map, float* w, const void* g, int gdt,
                       int64_t off, int64_t len, int8_t* qm, float* am, uint8_t* qv, float* av,
                       float* m1, float* v1)
{
    float* m0 = m1; /* reuse the scratch: dequantize in place, then update */
    float* v0 = v1;
    const int dyn = code_map == LTO_MAP_DYNAMIC;
    (dyn ? lto_dequantize_dynamic_signed : lto_dequantize_signed)(qm + off, len, *am, m0);
    (dyn ? lto_dequantize_dynamic_unsigned : lto_dequantize_unsigned)(qv + off, len, *av, v0);
    for (int64_t i = 0; i < len; ++i) {
        float mn, vn, wn;
        adamw_element(s, m0[i], v0[i], grad_value(g, gdt, off + i), w[off + i], &mn, &vn, &wn);
        w[off + i] = wn;
        m1[i] = mn; /* the update uses the unquantized m1, v1; codes are storage */
        v1[i] = vn;
    }
    (dyn ? lto_quantize_dynamic_signed : lto_quantize_signed)(m1, len, qm + off, am);
    (dyn ? lto_quantize_dynamic_unsigned : lto_quantize_unsigned)(v1, len, qv + off, av);
}

/* Sec. 3.5's Hybrid 8-bit operator, optimizer side: the clipped AdamW step over
 * 8-bit block-wise states; App. C: a non-finite step is skipped. */
int lto_hybrid8bit_adamw_step(float* const* params, const void* const* grads, int gdt,
                              int8_t* const* m_codes, float* const* m_absmax,
                              uint8_t* const* v_codes, float* const* v_absmax,
                              const int64_t* numels, int n_tensors, int64_t block_size,
                              int code_map, double lr, double beta1, double beta2, double eps,
                              double weight_decay, int64_t step, const float* coef,
                              const int32_t* status, int n_threads)
{
    if (n_tensors < 0 || block_size < 1 || step < 1 || (gdt != LTO_F32 && gdt != LTO_BF16) ||
        (code_map != LTO_MAP_LINEAR && code_map != LTO_MAP_DYNAMIC))
        return LTO_ERR_INVALID_ARG;
    if (n_tensors > 0 && (!params || !grads || !m_codes || !m_absmax || !v_codes || !v_absmax ||
                          !numels))
        return LTO_ERR_INVALID_ARG;
    if (status && *status == LTO_STATUS_NONFINITE)
        return LTO_OK; /* skipped step: nothing is written */

    adamw_scalars s;
    s.coef = coef ? *coef : 1.0f;
    lto_step_scalars(lr, beta1, beta2, eps, weight_decay, step, &s.h);

    for (int k = 0; k < n_tensors; ++k) {
        const int64_t n = numels[k];
        const int64_t n_blocks = (n + block_size - 1) / block_size;
#pragma omp parallel num_threads(n_threads > 1 ? n_threads : 1)
        {
            float* m1 = (float*)malloc((size_t)block_size * sizeof(float));
            float* v1 = (float*)malloc((size_t)block_size * sizeof(float));
#pragma omp for schedule(static)
            for (int64_t b = 0; b < n_blocks; ++b) {
                int64_t off = b * block_size;
                int64_t len = (n - off < block_size) ? n - off : block_size;
                step_block(&s, code_map, params[k], grads[k], gdt, off, len, m_codes[k],
                           &m_absmax[k][b], v_codes[k], &v_absmax[k][b], m1, v1);
            }
            free(m1);
            free(v1);
        }
    }
    return LTO_OK;
}

/* Sec. 3.5: the parameters outside the 8-bit slice keep full-precision Adam
 * states (DeepSpeed CPUAdam in the paper's run); same operation order. */
void lto_adamw_fp32_step(float* w, const void* grad, int gdt, float* m, float* v, int64_t n,
                         double lr, double beta1, double beta2, double eps, double weight_decay,
                         int64_t step, float coef)
{
    adamw_scalars s;
    s.coef = coef;
    lto_step_scalars(lr, beta1, beta2, eps, weight_decay, step, &s.h);
    for (int64_t i = 0; i < n; ++i)
        adamw_element(&s, m[i], v[i], grad_value(grad, gdt, i), w[i], &m[i], &v[i], &w[i]);
}

/* Sec. 3.1 and 3.4: parameters travel to the GPU for each layer; this is the
 * bf16 copy of the updated weights that such a transfer carries. */
void lto_round_bf16(const float* x, int64_t n, uint16_t* y)
{
    for (int64_t i = 0; i < n; ++i) {
        uint32_t u;
        memcpy(&u, &x[i], 4);
        uint32_t hi = u >> 16, lo = u & 0xFFFFu;
        if (isnan(x[i])) {
            y[i] = (uint16_t)(hi | 0x0040u);  /* quiet, sign kept */
            continue;
        }
        /* above the midpoint, or on it with an odd kept part: round up (the
         * carry may run into the exponent, up to infinity) */
        if (lo > 0x8000u || (lo == 0x8000u && (hi & 1u)))
            hi += 1;
        y[i] = (uint16_t)hi;
    }
}
