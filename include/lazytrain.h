/*
 * lazytrain.h -- C ABI of the MI355X (gfx950) Hybrid 8-bit optimizer step.
 *
 * The operation is the optimizer-side component of LazyTrain's Hybrid 8-bit
 * operator (paper Sec. 3.5, Hybrid 8-bit operator paragraph): fast gradient
 * clipping (per-tensor norms, one global norm, one scale) coupled with AdamW
 * whose first and second moments are stored as block-wise absmax 8-bit codes
 * over fp32 master weights.  Hyperparameter roles follow the App. C
 * training-configuration table (beta1, beta2, eps, learning rate, weight
 * decay, max grad norm; non-finite gradients skip the step).
 *
 * Steps, as named in this header and in the sources:
 *   a1  sum of squares of the gradients: one fp64 partial per 8192-element chunk;
 *   a2  the fixed-order finish: per-tensor sums S_k, the total S, the status;
 *   a3  the norm and the clip coefficient;
 *   a4  dequantizing the stored 8-bit moments;   a5  the clipped gradient;
 *   a6  the moment update;   a7  the AdamW weight update;
 *   a8  the new block absmax of each moment;   a9  requantizing and storing;
 *   a10 skipping a step whose gradients are not finite;
 *   a11 the same step over host-resident state streamed layer by layer;
 *   f1  fp32-state AdamW for tensors outside the 8-bit slice, and the slice;
 *   f2  the dynamic (non-linear) 8-bit code map;
 *   f3  the bf16 copy of the updated weights;
 *   f4  the gradient norm accumulated as gradients arrive.
 *
 * Conventions for every entry point:
 *  - Tensor data, workspace and scalar outputs are DEVICE pointers on the
 *    current HIP device, owned by the caller.  The library never frees them
 *    and keeps no reference after the work it enqueued has run.
 *  - Lists (arrays of pointers and numels) are HOST arrays of length
 *    n_tensors, read during the call only.  n_tensors may be 0 (the lists may
 *    then be NULL) and a numel may be 0: an empty tensor contributes nothing
 *    (its sum of squares is 0, its step writes nothing) and its pointers are
 *    neither checked nor dereferenced.  The streamed step needs at least one
 *    tensor per layer; those may be empty too.
 *  - All work is enqueued on `stream` (a hipStream_t; NULL is the default
 *    stream) in call order.  No call waits for the device; lt_read_status is
 *    the one entry point that synchronizes (a stream).
 *  - The return value reports argument and launch problems synchronously.
 *    Data problems (a non-finite gradient) are reported on the device through
 *    a status word.  lt_last_error() gives a message for the calling thread.
 *  - Every tensor is dense and contiguous.  Base pointers of weights,
 *    gradients and codes must be 16-byte aligned, absmax arrays 4-byte
 *    aligned, the workspace 256-byte aligned.
 *  - The workspace holds the tensor-list descriptors the call builds (and,
 *    for the norm, its partial sums).  Calls that overlap on the device must
 *    use different workspaces.  The library remembers what it last wrote into
 *    each workspace (by address) and copies descriptors in only when they
 *    differ, from a library-owned pinned staging buffer (the ring of buffers
 *    grows rather than wait for a copy still in flight).  Between calls the
 *    caller therefore must not write into a workspace; before freeing it or
 *    using its memory for anything else, call lt_workspace_release.  A kernel
 *    whose workspace no longer holds the descriptors it was launched for
 *    (checked through a per-copy tag in the workspace's first word) returns
 *    without reading or writing any tensor; lt_grad_sqnorm and
 *    lt_grad_sqnorm_finish then report LT_STATUS_BAD_WORKSPACE.
 *  - HIP graph capture: a list call whose descriptors are already in its
 *    workspace enqueues kernels only, and may be captured (also on another
 *    stream than the one the descriptors were copied on).  It must come after
 *    one uncaptured call with the same workspace and tensor list whose work has
 *    completed; a captured call that would have to copy descriptors returns
 *    LT_ERR_INVALID_ARG.  lt_clip_coef copies nothing and may always be
 *    captured.  The streamed step (host copies) is not capturable.
 *  - Results are bitwise reproducible: they do not depend on the grid size,
 *    the device occupancy or the stream.
 */
#ifndef LAZYTRAIN_H
#define LAZYTRAIN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum lt_err {
    LT_OK = 0,
    LT_ERR_INVALID_ARG = 1, /* NULL pointer, negative size, unsupported block size or dtype, bad hyperparameter */
    LT_ERR_ALIGNMENT = 2,   /* a base pointer is not aligned as stated above */
    LT_ERR_HIP = 3,         /* a HIP runtime call failed (device query, copy, launch, sync) */
    LT_ERR_WORKSPACE = 4    /* workspace NULL, misaligned or smaller than the size query returns */
} lt_err;

/* The status word written on the device by the norm (and lt_clip_coef).  The
 * steps skip, writing nothing, unless it holds LT_STATUS_OK. */
typedef enum lt_status {
    LT_STATUS_OK = 0,
    LT_STATUS_NONFINITE = 1,    /* the global sum of squares is NaN or infinite */
    LT_STATUS_BAD_WORKSPACE = 2 /* the workspace did not hold the call's descriptors (see above) */
} lt_status;

typedef enum lt_dtype {
    LT_DTYPE_F32 = 0,
    LT_DTYPE_BF16 = 1
} lt_dtype;

/* Code map of the 8-bit moments (see lt_hybrid8bit_adamw_step). */
typedef enum lt_code_map {
    LT_MAP_LINEAR = 0, /* linear absmax codes: m = q * A / 127 (int8), v = q * A / 255 (uint8) */
    LT_MAP_DYNAMIC = 1 /* this library's decade-tree codes: sign-magnitude m, unsigned v, 1e-7 .. 1 */
} lt_code_map;

/* Device-resident step count, for callers that enqueue steps ahead of the GPU
 * without reading each step's status first (App. C: a step with a non-finite
 * gradient is skipped and does not count; training stops after three skips in a
 * row).  A step state is caller-owned device memory of lt_step_state_bytes: this
 * header, then table_len entries; entry i holds the parts of the bias corrections
 * of step t = i + 1 that do not depend on the learning rate.  A step entry point
 * given a step state applies step t = applied + 1 with
 * step_size = fp32(lr / one_minus_beta1_t) (fp64 division on the device) and that
 * entry's rbc2: bitwise the scalars the host computes for that t.
 * lt_step_state_advance, enqueued after a step's kernels, counts the step. */
typedef struct lt_step_state {
    int64_t applied;      /* steps applied so far */
    int64_t table_len;    /* entries after this header */
    int32_t skips;        /* consecutive steps skipped */
    int32_t max_skips;    /* stop after this many skips in a row; 0: never */
    int32_t stopped;      /* 1: max_skips skips in a row; 2: the table ran out.  Every
                             later step then skips (writes nothing). */
    int32_t reserved[9];
} lt_step_state;          /* 64 bytes */

typedef struct lt_step_table_entry {
    double one_minus_beta1_t; /* 1 - beta1^t in fp64 (the C library's pow) */
    float rbc2;               /* fp32(1 / sqrt(1 - beta2^t)), computed in fp64 */
    float reserved;
} lt_step_table_entry;        /* 16 bytes */

/* Bytes of a step state with table_len entries; 0 if table_len < 1. */
size_t lt_step_state_bytes(int64_t table_len);

/* Host only: table entries of t = t_first .. t_first + count - 1 into out[count]. */
lt_err lt_step_table(double beta1, double beta2, int64_t t_first, int64_t count,
                     lt_step_table_entry* out);

/*
 * Writes a step state into device memory `state` (bytes >= lt_step_state_bytes(
 * table_len), 16-byte aligned), on `stream`: the table of t = 1 .. table_len for
 * beta1, beta2 (0 <= beta < 1), and the header with `applied` (>= 0), `skips`,
 * `max_skips` (>= 0) and stopped = 0.  from_state: NULL, or another device step
 * state whose applied, skips, max_skips and stopped the new one takes instead, on
 * the device in stream order (to grow a table without reading the count back).
 */
lt_err lt_step_state_init(void* state, size_t bytes, int64_t table_len, double beta1,
                          double beta2, int64_t applied, int32_t skips, int32_t max_skips,
                          const void* from_state, void* stream);

/* Counts one step on the device, after its step kernels on `stream`: with
 * *status == LT_STATUS_OK, applied += 1 and skips = 0 (or stopped = 2 if the table
 * did not reach the step); otherwise skips += 1, and stopped = 1 once skips reaches
 * a nonzero max_skips.  A stopped state is left as it is. */
lt_err lt_step_state_advance(void* state, const int32_t* status, void* stream);

/* Bytes of device workspace lt_grad_sqnorm needs for this list (descriptors,
 * one fp64 partial per 8192-element chunk, one fp64 per tensor); never 0 for a
 * valid list.  Returns 0 if n_tensors < 0, numels is NULL for n_tensors > 0 or
 * a numel is < 0. */
size_t lt_grad_sqnorm_workspace_bytes(const int64_t* numels, int n_tensors);

/*
 * Steps a1-a2: global sum of squares of a list of gradient tensors
 * (Sec. 3.5: per-tensor norms, then one global aggregate).
 *   grads[k]       device, numels[k] elements of grad_dtype (LT_DTYPE_F32 or
 *                  LT_DTYPE_BF16), read only.
 *   sq_per_tensor  device double[n_tensors] or NULL: S_k, the sum of squares
 *                  of tensor k.
 *   sq_total       device double: S = S_0 + S_1 + ... in list order (0 for
 *                  an empty list).
 *   status         device int32: LT_STATUS_NONFINITE if S is NaN or
 *                  infinite, else LT_STATUS_OK (LT_STATUS_BAD_WORKSPACE, with
 *                  S = NaN, if the workspace lost its descriptors; see above).
 * Accumulation is fp64 in a fixed order: each tensor is cut into 8192-element
 * chunks; in a chunk, lane l of 256 adds the squares of elements
 * 8*(l + 256*r) + e (r = 0..3, e = 0..7) in that order, a 64-lane halving
 * tree follows, then (W0 + W2) + (W1 + W3) over the four 64-lane groups; a
 * tensor's chunk sums go round-robin into 256 accumulators in ascending chunk
 * order, combined by a halving tree.  Results are therefore bitwise fixed.
 */
lt_err lt_grad_sqnorm(const void* const* grads, const int64_t* numels, int n_tensors,
                      int grad_dtype, void* workspace, size_t workspace_bytes,
                      double* sq_per_tensor, double* sq_total, int32_t* status, void* stream);

/*
 * For callers that cannot allocate device memory: code under HIP graph capture,
 * serving loops and harnesses that forbid hipMalloc.  Steps a1-a2 exactly as
 * lt_grad_sqnorm (same arguments without the workspace, same results bit for
 * bit), with the descriptors and partial sums held in a 16 MiB array of the
 * library's own in device memory (one per device, for the process's lifetime),
 * written by kernels from kernel arguments: the call allocates nothing, stages
 * nothing on the host and copies nothing from it.  Lists whose descriptors and
 * partials need more than 16 MiB (about 2 million 8192-element chunks, some
 * 1.7e10 elements) return LT_ERR_INVALID_ARG before any device work.  All calls
 * on one device share that array: calls that overlap on the device (on different
 * streams, or from different host threads) race and give undefined results; calls
 * in one stream's order do not.  Nothing in the array needs to start at zero.
 */
lt_err lt_grad_sqnorm_noalloc(const void* const* grads, const int64_t* numels, int n_tensors,
                              int grad_dtype, double* sq_per_tensor, double* sq_total,
                              int32_t* status, void* stream);

/*
 * Step a3: clip coefficient, device-resident (Sec. 3.5 scale step; App. C max
 * grad norm).  total_norm = fp32(sqrt(*sq_total)): the fp64 square root, correctly
 * rounded, then rounded to fp32 (ties to even);
 * coef = fminf(1, max_norm / (total_norm + 1e-6f)) in fp32.  max_norm must be
 * > 0; +INFINITY gives coef = 1 exactly.  total_norm may be NULL.
 *   status  device int32 or NULL.  When given, it is set to LT_STATUS_OK or
 *           LT_STATUS_NONFINITE from *sq_total, unless it already holds another
 *           value (a library error such as LT_STATUS_BAD_WORKSPACE), which it
 *           keeps; so a sum of squares obtained elsewhere (for example reduced
 *           across devices) yields the status the steps read.
 */
lt_err lt_clip_coef(const double* sq_total, float max_norm, float* total_norm, float* coef,
                    int32_t* status, void* stream);

/* Number of 8192-element chunks of a tensor list: the number of fp64 partials
 * the sum of squares keeps for it.  0 if an argument is invalid. */
int64_t lt_grad_chunk_count(const int64_t* numels, int n_tensors);

/* Bytes of device workspace lt_grad_sqnorm_partials needs (descriptors). */
size_t lt_grad_sqnorm_partials_workspace_bytes(int n_tensors);

/*
 * Step a1 on part of a model, as its gradients arrive (f4: norm accumulation
 * during backward, so that a layer-streaming executor, which offloads
 * gradients layer by layer, never streams them back in for the norm;
 * Sec. 3.1 and the gradient D2H traffic of Sec. 3.4).  Writes the fp64 chunk
 * partials of grads[0..n_tensors) in the fixed order of lt_grad_sqnorm.
 *   partials  device double[lt_grad_chunk_count(numels, n_tensors)]: the slice
 *             of the model-wide partials array that starts at these tensors'
 *             first chunk (the chunk count of the model's earlier tensors).
 *             Not touched (and may be NULL) when the count is 0.
 * The parts of a model may arrive in any order, on any streams; once all are
 * written, lt_grad_sqnorm_finish gives bitwise the result of lt_grad_sqnorm
 * over the whole list.
 */
lt_err lt_grad_sqnorm_partials(const void* const* grads, const int64_t* numels, int n_tensors,
                               int grad_dtype, double* partials, void* workspace,
                               size_t workspace_bytes, void* stream);

/* Bytes of device workspace lt_grad_sqnorm_finish needs for n_tensors. */
size_t lt_grad_sqnorm_finish_workspace_bytes(int n_tensors);

/*
 * Step a2 from the model-wide partials (f4): S_k, S and the non-finite status
 * exactly as lt_grad_sqnorm computes them (same accumulators, same trees).
 *   numels    host int64[n_tensors]: the whole model's tensor sizes.
 *   partials  device double[lt_grad_chunk_count(numels, n_tensors)], every
 *             entry written by lt_grad_sqnorm_partials (may be NULL when the
 *             count is 0).
 *   sq_per_tensor (may be NULL), sq_total, status: as in lt_grad_sqnorm.
 */
lt_err lt_grad_sqnorm_finish(const int64_t* numels, int n_tensors, const double* partials,
                             void* workspace, size_t workspace_bytes, double* sq_per_tensor,
                             double* sq_total, int32_t* status, void* stream);

/* Bytes of device workspace lt_hybrid8bit_adamw_step needs for n_tensors
 * tensors (the uploaded descriptor table).  0 if n_tensors < 0. */
size_t lt_step_workspace_bytes(int n_tensors);

/*
 * Steps a4-a10: one fused Hybrid 8-bit AdamW step over a list of tensors
 * (Sec. 3.5: block-wise 8-bit AdamW states, block-wise scale handling, the
 * clip scale; App. C: AdamW hyperparameters and the non-finite skip).
 * For tensor k with n = numels[k] and nb = ceil(n / block_size):
 *   params[k]   device float[n], read and written (fp32 master weights);
 *   grads[k]    device grad_dtype[n], read only;
 *   m_codes[k]  device int8[n]  and m_absmax[k] device float[nb]: first moment,
 *               value = code * absmax / 127;
 *   v_codes[k]  device uint8[n] and v_absmax[k] device float[nb]: second
 *               moment, value = code * absmax / 255.
 * Blocks are contiguous runs of block_size elements of one tensor (the last
 * may be partial).  block_size is a multiple of 64 in [64, 65536] (the paper's
 * run uses 4096, App. C variant table).  Powers of two up to 8192 take the
 * fast kernel; other sizes a kernel that owns one block per workgroup, with
 * the same results.
 * Per element, in fp32 with one rounding per operation (fma rounds once,
 * division and sqrt are correctly rounded):
 *   m0 = q_m * (A_m / 127), v0 = q_v * (A_v / 255), g = grad * coef,
 *   m1 = fma(b1, m0, c1 * g), v1 = fma(b2, v0, c2 * (g * g)),
 *   w1 = fma(-step_size, m1 / fma(sqrt(v1), rbc2, eps), w * decay),
 * with b1 = fp32(beta1), b2 = fp32(beta2), c1 = fp32(1 - beta1),
 * c2 = fp32(1 - beta2), decay = fp32(1 - lr * weight_decay),
 * step_size = fp32(lr / (1 - beta1^step)), rbc2 = fp32(1 / sqrt(1 - beta2^step)),
 * eps = fp32(eps), each computed on the host in fp64 from the double
 * arguments.  Per block: A'_m = max |m1|, A'_v = max v1; codes
 * rint(m1 * (127 / A'_m)) clamped to [-127, 127] and rint(v1 * (255 / A'_v))
 * clamped to [0, 255] (round half to even); a block whose new absmax or its
 * reciprocal is not finite stores zero codes and absmax 0.  These are the
 * codes of code_map = LT_MAP_LINEAR.
 *   code_map LT_MAP_DYNAMIC: both moments use non-linear decade-tree codes
 *            instead (the paper names block-wise 8-bit AdamW states without a
 *            code map).  This map is this library's own, after the dynamic tree
 *            quantization of Dettmers et al.'s block-wise 8-bit optimizers, and
 *            differs from that construction: each code sits at the upper end
 *            of its linear sub-interval (not its midpoint), so the top code is
 *            exactly 1 with no separate code for it; m codes are sign-magnitude
 *            bytes with a -0; v spans 8 decades.  Codes are therefore not
 *            interchangeable with that map's.  A code's magnitude bits are
 *            leading zeros z (decade 10^-z), an indicator one and p fraction
 *            bits f: magnitude
 *            fp32((0.1 + 0.9 * ((f + 1) / 2^p)) * 10^-z), computed in fp64 in
 *            that order, 0 for the zero code.  m codes are sign-magnitude
 *            bytes (sign bit 0x80 set for m1 < 0, 7 magnitude bits, 1e-6 .. 1),
 *            v codes 8 magnitude bits (1e-7 .. 1).  Decode: m0 = +-magnitude *
 *            A_m (0x80 gives -0), v0 = magnitude * A_v.  Encode: inv = 1 / A'
 *            (fp32), the code whose magnitude is nearest |m1| * inv (v1 * inv)
 *            by fp32 distance, ties to the smaller code, NaN to magnitude 0; the
 *            same absmax and zero-block rule.  A second moment down to 5e-8 of its
 *            block's absmax keeps a nonzero code (2e-3 with the linear map).
 *   step     1-based index t of the step being applied (>= 1), unless step_state
 *            is given.
 *   step_state  NULL, or a device step state (lt_step_state): the step index and
 *            its bias corrections come from it on the device (t = applied + 1;
 *            `step` is then ignored), and a stopped state makes the step write
 *            nothing.  The caller enqueues lt_step_state_advance after the step.
 *   lr, weight_decay >= 0; 0 <= beta1, beta2 < 1; eps > 0, also after its
 *            rounding to fp32 (with eps = 0 a zero gradient on a zero second
 *            moment divides 0 by 0); all finite.  Otherwise LT_ERR_INVALID_ARG.
 *   coef     device float or NULL (no clipping, 1.0f).
 *   status   device int32 or NULL (never skip).  When it holds anything but
 *            LT_STATUS_OK the kernel writes nothing: weights, codes and
 *            absmax stay bitwise unchanged.
 *   params_bf16  NULL, or a host list of device uint16[n] arrays (entries may
 *            be NULL: no copy of that tensor), 16-byte aligned: a bf16 copy of
 *            the weights for the next forward pass of a layer-streaming
 *            executor, which moves parameters to the GPU for every layer
 *            (Sec. 3.1; parameter H2D traffic in Sec. 3.4).  After the call it
 *            holds bf16(w1), rounded to nearest even (a NaN becomes a quiet
 *            NaN), written by the step kernel from registers
 *            (+2 B/param); after a skipped step, bf16 of the unchanged weights.
 * No array the call writes may share a byte with another array of the call
 * (gradients may alias one another): otherwise LT_ERR_INVALID_ARG.
 */
lt_err lt_hybrid8bit_adamw_step(float* const* params, const void* const* grads, int grad_dtype,
                                int8_t* const* m_codes, float* const* m_absmax,
                                uint8_t* const* v_codes, float* const* v_absmax,
                                uint16_t* const* params_bf16, const int64_t* numels,
                                int n_tensors, int block_size, int code_map, double lr,
                                double beta1, double beta2, double eps, double weight_decay,
                                int64_t step, const float* coef, const int32_t* status,
                                const void* step_state, void* workspace, size_t workspace_bytes,
                                void* stream);

/* Bytes of device workspace lt_streamed_hybrid8bit_adamw_step needs: the
 * descriptors of every layer, one fp64 partial per 8192-element chunk of the
 * whole model, and ring_slots slots each large enough for the largest layer's
 * weights, gradients, codes and scales (and its bf16 weight copy when
 * bf16_copy is nonzero: the call passes a params_bf16 list).  With keep_grads
 * nonzero the slots hold no gradients and every gradient gets a region of its
 * own instead (the call passes keep_grads).  0 if an argument is invalid. */
size_t lt_streamed_workspace_bytes(const int64_t* numels, int n_tensors, const int* layer_first,
                                   int n_layers, int grad_dtype, int block_size, int ring_slots,
                                   int bf16_copy, int keep_grads);

/*
 * Step a11: one clipped Hybrid 8-bit AdamW step over a model whose fp32
 * weights, gradients and 8-bit states stay in HOST memory and pass through HBM
 * layer by layer (Sec. 3.5: parameters and optimizer states are kept in CPU
 * memory while the GPU is a transient compute cache; Sec. 3.4: the CPU-GPU
 * link is the shared transfer resource).  Same per-element arithmetic, block
 * layout and skip rule as lt_hybrid8bit_adamw_step, and the same fixed-order
 * sum of squares over the whole model, so every result is bitwise that of the
 * resident path on the same data.
 *   params .. v_absmax  HOST pointers, one entry per tensor, layouts as in
 *                       lt_hybrid8bit_adamw_step.
 *   params_bf16         NULL or a HOST list of host uint16[n] arrays (entries
 *                       may be NULL) receiving the bf16 weight copy as in
 *                       lt_hybrid8bit_adamw_step (+2 B/param copied out); the
 *                       workspace must then be sized with bf16_copy = 1.  Pinned memory (hipHostMalloc)
 *                       lets copies overlap compute; pageable memory works but
 *                       serializes the copies.  Read and written asynchronously:
 *                       the caller must not touch them until compute_stream has
 *                       completed the call's work.
 *   layer_first         host int[n_layers + 1]: layer i is tensors
 *                       [layer_first[i], layer_first[i + 1]); 0 = first, n_tensors
 *                       = last, strictly rising.  Layers are streamed in order.
 *   max_norm            > 0; +INFINITY disables clipping (coef = 1).
 *   norm_ready          nonzero: *sq_total and *status already hold S and its
 *                       status (from lt_grad_sqnorm_finish over gradients summed
 *                       as they arrived); pass 1 and the finish are skipped and
 *                       the gradients are copied in once.
 *   keep_grads          nonzero: every gradient keeps its own region of the
 *                       workspace (sized with keep_grads = 1: 2 or 4 B/param more,
 *                       and the slots then hold no gradient), so a gradient copied
 *                       in by pass 1 stays in HBM for pass 2 and crosses the link
 *                       once.  Results are bitwise those without it.  With
 *                       norm_ready, pass 2 copies the gradients into those regions.
 *   ring_slots          device slots in the ring, 2..16 (3 lets one layer copy in
 *                       while one computes and one copies out).
 *   sq_total, total_norm (may be NULL), coef, status: device outputs as in
 *                       lt_grad_sqnorm and lt_clip_coef (sq_total and status are
 *                       inputs when norm_ready is set).  A NONFINITE status
 *                       skips the update: weights, codes and scales are copied
 *                       back unchanged.
 *   layer_events        NULL, or a host array of 8 * n_layers hipEvent_t created by
 *                       the caller (entries may be NULL), which the call records
 *                       around layer i's work: [8i] and [8i+1] on h2d_stream before
 *                       and after its pass-1 gradient copies (not recorded with
 *                       norm_ready), [8i+2] and [8i+3] before and after its pass-2
 *                       copies in, [8i+6] and [8i+7] on compute_stream before and
 *                       after its step kernels, [8i+4] and [8i+5] on d2h_stream
 *                       before and after its copies out.  Each "before" is recorded
 *                       once the stream may start that work, so timing events give
 *                       each phase's own duration; an executor can also wait on
 *                       them.
 *   compute_stream, h2d_stream, d2h_stream: the copies in, the kernels and the
 *                       copies out are ordered by events; the call's work ends on
 *                       compute_stream (synchronize it before reading results).
 *                       The three may be the same stream.  Streamed calls on one
 *                       device are serialized by the library.
 * Host arrays of different tensors should not overlap: the call does not check it
 * (a caller may stream one host buffer for several layers to measure transfer
 * rates), and the results of tensors that share bytes are then undefined.
 * Pass 1 copies each layer's gradients in (2 or 4 B/param) and sums them; pass 2
 * copies weights, gradients, codes and scales in (8 or 10 B/param + 8 B/block;
 * 6 B/param + 8 B/block with keep_grads) and weights, codes and scales out
 * (6 B/param + 8 B/block).
 */
lt_err lt_streamed_hybrid8bit_adamw_step(float* const* params, const void* const* grads,
                                         int grad_dtype, int8_t* const* m_codes,
                                         float* const* m_absmax, uint8_t* const* v_codes,
                                         float* const* v_absmax, uint16_t* const* params_bf16,
                                         const int64_t* numels, int n_tensors,
                                         const int* layer_first, int n_layers,
                                         int block_size, int code_map, double lr, double beta1,
                                         double beta2,
                                         double eps, double weight_decay, int64_t step,
                                         float max_norm, int norm_ready, int keep_grads,
                                         int ring_slots, void* workspace,
                                         size_t workspace_bytes, double* sq_total,
                                         float* total_norm, float* coef, int32_t* status,
                                         void* const* layer_events, void* compute_stream,
                                         void* h2d_stream, void* d2h_stream);

/* Bytes of device workspace lt_adamw_fp32_step needs for n_tensors tensors. */
size_t lt_adamw_fp32_workspace_bytes(int n_tensors);

/*
 * fp32-state AdamW over a list of tensors: the part of the Hybrid 8-bit
 * operator that keeps full-precision optimizer states (Sec. 3.5: DeepSpeed
 * CPUAdam handles most parameters, a 2% slice uses 8-bit states; App. C
 * variant table).  exp_avg[k], exp_avg_sq[k] are device float[numels[k]], read
 * and written.  Per element, the same fp32 operations as
 * lt_hybrid8bit_adamw_step with m0, v0 taken from and m1, v1 stored to these
 * arrays.  coef, status, step_state and params_bf16 (NULL or a list of device bf16
 * copies, entries may be NULL) as there.  Pointers 16-byte aligned; workspace
 * 256-byte aligned.  As there, written arrays may not overlap any other array of
 * the call (LT_ERR_INVALID_ARG).
 */
lt_err lt_adamw_fp32_step(float* const* params, const void* const* grads, int grad_dtype,
                          float* const* exp_avg, float* const* exp_avg_sq,
                          uint16_t* const* params_bf16, const int64_t* numels, int n_tensors, double lr, double beta1, double beta2, double eps,
                          double weight_decay, int64_t step, const float* coef,
                          const int32_t* status, const void* step_state, void* workspace,
                          size_t workspace_bytes, void* stream);

/*
 * Chooses the tensors that take 8-bit states when only a fraction of the
 * parameters should (Sec. 3.5: a 2% parameter slice; the paper does not say
 * which).  Greedy by decreasing size, ties in list order: a tensor is taken
 * when the running total stays <= fraction * total parameters.  Host only.
 *   is_8bit       host uint8[n_tensors]: 1 for a chosen tensor, else 0.
 *   n_8bit_params host int64 or NULL: parameters chosen.
 */
lt_err lt_select_8bit_slice(const int64_t* numels, int n_tensors, double fraction,
                            uint8_t* is_8bit, int64_t* n_8bit_params);

/* Copies the device status word to *out and synchronizes `stream` (the only
 * entry point that blocks the host).  An asynchronous device fault from
 * earlier work on the stream surfaces here as LT_ERR_HIP. */
lt_err lt_read_status(const int32_t* status, void* stream, int32_t* out);

/* Forgets what the library last wrote into `workspace` (a device pointer
 * passed as the workspace of earlier calls; NULL or an unknown pointer is a
 * no-op).  Call it before freeing a workspace, reusing its memory, or writing
 * into it; the next call with it copies its descriptors in again.  Host only:
 * it enqueues nothing and waits for nothing. */
lt_err lt_workspace_release(const void* workspace);

/* Caps the number of workgroups of the persistent kernels (0 = size the grid
 * from the device's compute units and occupancy).  Results do not depend on
 * it; tests use it to check that.  Process-wide. */
lt_err lt_set_max_workgroups(int max_workgroups);

/* Message of the last error returned on the calling thread ("" if none). */
const char* lt_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* LAZYTRAIN_H */
