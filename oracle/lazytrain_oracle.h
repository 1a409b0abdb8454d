/*
 * lazytrain_oracle.h -- TEST INFRASTRUCTURE, not part of the product.
 *
 * A plain, slow, obviously correct CPU definition of the optimizer-side hot
 * path of LazyTrain's Hybrid 8-bit operator: the global gradient L2 norm and
 * clip coefficient, then block-wise 8-bit AdamW over fp32 master weights
 * (paper Sec. 3.5 "Objective and Execution", the Hybrid 8-bit operator
 * paragraph; hyperparameters and the non-finite rule from the App. C
 * training-configuration table; block size from the App. C variant table).
 *
 * Only the test suite, the package smoke check and the benchmark's CPU
 * baseline leg may load this library.  It shares no code, header or constant
 * with the HIP library; both are written from the same definition.
 *
 * Precision: the paper keeps fp32 master weights, so the AdamW update is
 * fp32 with an explicit operation order (every fmaf is one rounding, every
 * other operation is a separately rounded IEEE operation, no contraction).
 * The gradient norm is accumulated in fp64, which the paper's FP32
 * aggregation does not require but which makes the per-tensor fallback for
 * unsupported or non-finite cases unnecessary.
 *
 * All pointers are host pointers.  Functions never allocate on behalf of the
 * caller beyond transient scratch and never keep pointers after returning.
 * n_threads <= 1 runs single-threaded; any thread count gives bitwise the same
 * results because every partial has a fixed index.
 *
 * Parity unpinned, in part: two choices here are readings that the paper does
 * not fix, the fixed reduction order of the sum of squares and the 8-bit code
 * maps.  Their values are pinned (the sum within the order's rounding bound and
 * exactly on exactly representable inputs; the codes by round-trip, rounding
 * and map-structure properties), but their exact bits are this definition's.
 *
 * Step labels in the section titles of the source: a1-a2 the sum of squares
 * and its fixed-order finish, a3 the clip coefficient, a4-a10 the step
 * (dequantize, clip, moments, weight update, block absmax, requantize, skip),
 * a8-a9 the block quantizer on its own, f1 fp32-state AdamW, f2 the dynamic
 * code map, f3 the bf16 weight copy.
 */
#ifndef LAZYTRAIN_ORACLE_H
#define LAZYTRAIN_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { LTO_F32 = 0, LTO_BF16 = 1 };
enum { LTO_STATUS_OK = 0, LTO_STATUS_NONFINITE = 1 };
enum { LTO_OK = 0, LTO_ERR_INVALID_ARG = 1 };
enum { LTO_MAP_LINEAR = 0, LTO_MAP_DYNAMIC = 1 };

/* Chunk length and lane layout of the fixed sum-of-squares order. */
#define LTO_CHUNK 8192
#define LTO_LANES 256

/*
 * Global sum of squares of a list of gradient tensors (Sec. 3.5: per-tensor
 * norms, then one global aggregate).  grads[k] points to numels[k] elements of
 * dtype gdt (LTO_F32 or LTO_BF16).  Writes S_k to sq_per_tensor[k] (may be
 * NULL), S to *sq_total and LTO_STATUS_NONFINITE to *status when S is not
 * finite (else LTO_STATUS_OK).  Reduction order: each tensor splits into
 * 8192-element chunks; a chunk is summed by 256 lanes (lane l owns elements
 * 8*(l + 256*r) + e, r = 0..3, e = 0..7, in that order), a 64-lane halving
 * tree per group of 64 lanes, then (W0 + W2) + (W1 + W3); a tensor's chunk
 * partials go round-robin into 256 accumulators in ascending chunk order,
 * which a halving tree combines; S sums the S_k in list order.
 */
int lto_grad_sqnorm(const void* const* grads, const int64_t* numels, int n_tensors, int gdt,
                    double* sq_per_tensor, double* sq_total, int32_t* status, int n_threads);

/* Brute force: fp64 sum of (double)x*(double)x in plain index order. */
double lto_grad_sqnorm_naive(const void* const* grads, const int64_t* numels, int n_tensors,
                             int gdt);

/*
 * Clip coefficient (Sec. 3.5 scale step; max grad norm from App. C):
 * norm = fp32(sqrt(S)), coef = fminf(1, max_norm / (norm + 1e-6f)), all fp32
 * after the rounding of the fp64 square root.  max_norm = +inf gives 1.
 */
void lto_clip_coef(double sq_total, float max_norm, float* total_norm, float* coef);

/*
 * The fp32 scalars of one AdamW step (App. C optimizer-hyperparameters row;
 * Adam with bias correction and decoupled weight decay).  Hyperparameters arrive as doubles (as a
 * Python or C caller holds them); each scalar is computed in fp64 and rounded
 * once to fp32: decay = 1 - lr*wd, step_size = lr / (1 - beta1^t),
 * rbc2 = 1 / sqrt(1 - beta2^t), c1 = 1 - beta1, c2 = 1 - beta2, and beta1,
 * beta2, eps themselves.  beta^t uses the C library pow().
 */
typedef struct {
    float beta1, beta2, eps, c1, c2, decay, step_size, rbc2;
} lto_scalars;
void lto_step_scalars(double lr, double beta1, double beta2, double eps, double weight_decay,
                      int64_t step, lto_scalars* out);

/*
 * One Hybrid 8-bit AdamW step over a list of tensors (Sec. 3.5, the Hybrid
 * 8-bit operator; App. C hyperparameters and safety checks).  For tensor k:
 * params[k] fp32[n], grads[k] gdt[n] (read only), m_codes[k] int8[n],
 * v_codes[k] uint8[n], m_absmax[k] / v_absmax[k] fp32[ceil(n / block_size)].
 * coef may be NULL (no clipping, 1.0f).  status may be NULL (never skip);
 * when *status == LTO_STATUS_NONFINITE nothing is written.  step is the
 * 1-based index t of the step being applied.  Returns LTO_OK or
 * LTO_ERR_INVALID_ARG (block_size < 1, step < 1, n_tensors < 0, a NULL list).
 * Per element (fp32, scalars from lto_step_scalars):
 * m0 = q_m*(A_m/127), v0 = q_v*(A_v/255),
 * g = grad*coef, m1 = fmaf(b1, m0, c1*g), v1 = fmaf(b2, v0, c2*(g*g)),
 * d = fmaf(sqrtf(v1), rbc2, eps), w1 = fmaf(-step_size, m1/d, w*decay);
 * per block the new absmax A'_m = max|m1|, A'_v = max v1 and the codes
 * rint(m1*127/A'_m), rint(v1*255/A'_v) (clamped); a block whose absmax or
 * reciprocal is not finite stores zero codes and absmax 0.  code_map
 * LTO_MAP_LINEAR is that map; LTO_MAP_DYNAMIC decodes and encodes with the
 * dynamic map below instead (the same absmax and zero-block rule).
 */
int lto_hybrid8bit_adamw_step(float* const* params, const void* const* grads, int gdt,
                              int8_t* const* m_codes, float* const* m_absmax,
                              uint8_t* const* v_codes, float* const* v_absmax,
                              const int64_t* numels, int n_tensors, int64_t block_size,
                              int code_map, double lr, double beta1, double beta2, double eps,
                              double weight_decay, int64_t step, const float* coef,
                              const int32_t* status, int n_threads);

/* Block quantizers used by the step (Sec. 3.5 block-wise scales; the linear map
 * is a reading), exported for the quantizer tests.
 * Signed (first moment): A = max|x|, q = clamp(rint(x * (127/A)), -127, 127).
 * Unsigned (second moment, x >= 0): A = max x, q = clamp(rint(x * (255/A)), 0, 255).
 * A block whose A or reciprocal is not finite gets q = 0 and A = 0. */
void lto_quantize_signed(const float* x, int64_t n, int8_t* q, float* absmax);
void lto_quantize_unsigned(const float* x, int64_t n, uint8_t* q, float* absmax);
void lto_dequantize_signed(const int8_t* q, int64_t n, float absmax, float* x);
void lto_dequantize_unsigned(const uint8_t* q, int64_t n, float absmax, float* x);

/*
 * Dynamic (non-linear) code map.  The paper names block-wise 8-bit AdamW
 * states without giving a code map (Sec. 3.5); besides the linear absmax map,
 * the common reading is the dynamic tree quantization of Dettmers et al.
 * (8-bit optimizers via block-wise quantization, 2022), restated here.  A code's
 * magnitude bits read: leading zero bits give the decade 10^-zeros, the first
 * one bit is an indicator, and the p bits after it are a linear fraction f:
 *   magnitude = fp32((0.1 + 0.9 * ((f + 1) / 2^p)) * 10^-zeros), in fp64 in
 *   that order (10^-zeros a double literal), 0 for the all-zero code.
 * Signed (first moment): a sign bit and 7 magnitude bits (sign-magnitude byte,
 * the sign bit set for x < 0, so a negative value below half the smallest
 * magnitude is stored as -0; magnitudes 1e-6 .. 1).  Unsigned (second moment): 8
 * magnitude bits (1e-7 .. 1).  Magnitudes rise with the code and the top code
 * is exactly 1, so a block's absmax element is stored exactly.
 * lto_dynamic_map writes the 128 (signed) or 256 (unsigned) magnitudes.
 * Quantize: A = max |x| (max x), inv = 1/A in fp32; code = the nearest
 * magnitude to |x| * inv by fp32 distance (ties to the smaller code, NaN to 0),
 * with the sign bit for x < 0; a block whose A or inv is not finite stores zero
 * codes and absmax 0.  Dequantize: +-magnitude * A (-0 * A for the code 0x80).
 */
void lto_dynamic_map(int is_signed, float* table);
void lto_quantize_dynamic_signed(const float* x, int64_t n, int8_t* q, float* absmax);
void lto_quantize_dynamic_unsigned(const float* x, int64_t n, uint8_t* q, float* absmax);
void lto_dequantize_dynamic_signed(const int8_t* q, int64_t n, float absmax, float* x);
void lto_dequantize_dynamic_unsigned(const uint8_t* q, int64_t n, float absmax, float* x);

/* fp32-state AdamW (Sec. 3.5: the parameters outside the 8-bit slice) with the
 * same operation order as the 8-bit step (states
 * m, v stay fp32 and are updated in place).  Used to check that the 8-bit
 * step reduces to plain AdamW when its states are exactly representable. */
void lto_adamw_fp32_step(float* w, const void* grad, int gdt, float* m, float* v, int64_t n,
                         double lr, double beta1, double beta2, double eps, double weight_decay,
                         int64_t step, float coef);

/* bf16 copy of fp32 values, as the step's optional low-precision weight copy
 * (the parameters the layer-streaming executor moves to the GPU for the next
 * forward pass: Sec. 3.1, and the parameter H2D traffic of Sec. 3.4).  Round to nearest, ties to even, on the 16 dropped bits of the
 * fp32 pattern (an overflow rounds to infinity, subnormals round like any other
 * value); a NaN gives a quiet NaN of the same sign. */
void lto_round_bf16(const float* x, int64_t n, uint16_t* y);

#ifdef __cplusplus
}
#endif
#endif
