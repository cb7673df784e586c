/*
 * gefen.h -- C ABI of the MI355X (gfx950) implementation of the Gefen optimizer
 * ("Gefen: Optimized Stochastic Optimizer", arXiv 2606.13894).
 *
 * Gefen keeps, per parameter tensor, (i) one uint8 code per weight into a learned
 * codebook and one absmax scale per block for the first moment, and (ii) one shared
 * second moment per block. Blocks are consecutive runs of `period` elements of the
 * flattened tensor, inferred once from the first gradient (Sec. 5.1, Alg. 2), or an
 * explicit table of block offsets. The codebook is fitted by an exact histogram DP
 * (Alg. 3, App. D). Each step (Alg. 1) dequantizes, updates and requantizes the
 * momentum, updates the shared second moment and applies the bias-corrected,
 * decoupled-weight-decay update.
 *
 * Conventions for every function below:
 *  - Return value: GEFEN_OK (0) or a negative gefen_status. On error,
 *    gefen_last_error() returns a message for the calling thread.
 *  - `stream` is a hipStream_t passed as void* (NULL = the default stream). Every
 *    device operation is enqueued on it; functions that must return host values
 *    synchronise that stream and say so.
 *  - Device pointers are HIP device (or managed) memory of the current device;
 *    "host" pointers are ordinary host memory. Nothing is retained after a call
 *    returns unless stated.
 *  - Parameters and gradients are owned by the caller, contiguous, row-major. A
 *    tensor is identified by its position in the arrays passed at init; later calls
 *    must pass the same number of tensors with the same numel and gradient dtype.
 *  - The state and every device buffer inside it are owned by the library: allocated
 *    by gefen_init, freed by gefen_destroy. gefen_step allocates nothing.
 *  - Calls on one state must be ordered (same stream, or externally synchronised).
 *
 * Environment variable (debugging only):
 *  GEFEN_DEBUG_SYNC  set: gefen_step synchronises its stream and reports kernel errors.
 */
#ifndef GEFEN_H
#define GEFEN_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    GEFEN_OK = 0,
    GEFEN_EINVAL = -1,      /* bad argument: null pointer, size mismatch, t < 1, beta
                               outside [0, 1), non-finite hyperparameter, eps < 0 */
    GEFEN_EDTYPE = -2,      /* unsupported dtype, or dtype differs from the one at init */
    GEFEN_EHIP = -3,        /* a HIP runtime call failed; the message names it */
    GEFEN_ENOMEM = -4,      /* device or host allocation failed */
    GEFEN_EDEGENERATE = -5  /* reserved, returned by no call: a fit that sees fewer
                               non-empty histogram bins than codebook entries is not an
                               error; it installs a valid fallback codebook and
                               gefen_get_fit_info reports status 1 (fits are
                               asynchronous, so no call could return it in time) */
} gefen_status;

typedef enum { GEFEN_F32 = 0, GEFEN_BF16 = 1 } gefen_dtype;

/* A device tensor: `ptr` is a device pointer to `numel` contiguous elements of `dtype`.
 * Parameters are always GEFEN_F32; gradients are GEFEN_F32 or GEFEN_BF16. */
typedef struct {
    void* ptr;
    int64_t numel;
    int32_t dtype;
    int32_t reserved;   /* must be 0 */
} gefen_tensor;

typedef struct gefen_state gefen_state;   /* opaque, library-owned */

/* ------------------------------------------------------------------------------
 * gefen_init -- Alg. 1 initialisation: block partitioning of every tensor from the
 * first gradient (Sec. 5.1, Alg. 2), codebook fit on that gradient (Alg. 3), and
 * zero state (codes 0, scales 0, second moments 0).
 *
 *  grads0          n_tensors device gradient tensors of the first step (F32/BF16).
 *  period_override host int64[n_tensors] or NULL. Entry > 0 fixes that tensor's
 *                  period (must divide numel); 0 infers it with Alg. 2.
 *  block_offsets   host int64[n_blocks + 1] or NULL. Explicit blocks over the
 *                  concatenation of all tensors in order: block b covers global
 *                  elements [block_offsets[b], block_offsets[b+1]). Must start at 0,
 *                  increase strictly, end at the total numel, and have a boundary at
 *                  every tensor boundary. Overrides inference and period_override.
 *  code_bits       bits per momentum code: 8 (k = 256 entries, 16k = 4096 histogram
 *                  bins, one code per byte) or 4 (k = 16, 256 bins, two codes per
 *                  byte; the paper's 4-bit variant, Sec. 7 ablation).
 *  eps_part        eps inside log(g^2 + eps) of the partition score (>= 0; the
 *                  paper leaves it open -- the optimizer eps, 1e-8, is the default).
 *  stream          stream for all work; synchronised once (the inferred periods
 *                  size the state).
 *  out             receives the new state.
 * Errors: EINVAL, EDTYPE, EHIP, ENOMEM. A degenerate codebook fit returns OK (the
 * fallback codebook is installed); query it with gefen_get_fit_info.
 * ---------------------------------------------------------------------------- */
int gefen_init(const gefen_tensor* grads0, int32_t n_tensors,
               const int64_t* period_override,
               const int64_t* block_offsets, int64_t n_blocks,
               int32_t code_bits, double eps_part, void* stream, gefen_state** out);

/* ------------------------------------------------------------------------------
 * gefen_step -- one optimizer step (Alg. 1, loop body), for every block B:
 *   m_i   = beta1 * (c_dec[q_i] * s_B) + (1 - beta1) * g_i
 *   s_B'  = max_i |m_i|;   q_i' = nearest entry of c_enc to m_i / s_B'
 *           (ties to the lower index; s_B' = 0 gives code 0)
 *   v_B'  = beta2 * v_B + (1 - beta2) * mean_{i in B} g_i^2
 *   theta = theta - lr * ( m_i / (1 - beta1^t) / (sqrt(v_B' / (1 - beta2^t)) + eps)
 *                          + weight_decay * theta )
 *  params  n_tensors device F32 tensors, updated in place.
 *  grads   n_tensors device gradients (dtype as at init), read only.
 *  t       step number, >= 1 (the first step after init is 1).
 *  lr, beta1, beta2, eps, weight_decay  hyperparameters as in AdamW. The scalars the
 *          kernels use (beta1, 1 - beta1, beta2, 1 - beta2, lr / (1 - beta1^t),
 *          1 / (1 - beta2^t), eps, 1 - lr * weight_decay) are formed in float64 and
 *          rounded once to fp32.
 * Asynchronous: enqueues kernels on `stream` only; no allocation. The state keeps
 * device tables of tensor addresses for the last four parameter/gradient buffer sets
 * it was given; a call with another set first enqueues a small host-to-device copy of
 * its table (the host waits only if that slot's previous copy is still pending).
 * The decode codebook is the current one; after gefen_fit_codebook the
 * next step encodes with the new codebook, and later steps decode with it too.
 * NaN or Inf in gradients propagate into parameters and state as in AdamW.
 * Errors: EINVAL, EDTYPE, EHIP (launch failure). Kernel faults surface at the next
 * synchronisation of `stream`.
 * ---------------------------------------------------------------------------- */
int gefen_step(gefen_state* st, const gefen_tensor* params, const gefen_tensor* grads,
               int32_t n_tensors, double lr, double beta1, double beta2, double eps,
               double weight_decay, int64_t t, void* stream);

/* ------------------------------------------------------------------------------
 * gefen_step_fit -- gefen_step, and the codebook refit (Alg. 3) on the same gradients:
 * the result of gefen_step followed by gefen_fit_codebook(grads), bit for bit. The step
 * kernels of explicit and irregular blocks take the histogram while they stream the
 * gradients (each element is binned once its block's max |g| is known), so those blocks
 * are not read a second time; the other tiles go through the histogram kernel. The
 * new codebook ENCODES at the next step (this step decodes and encodes with the current
 * one) and is used for both from the step after. The histogram stays readable as state
 * array 7 until the next fit. Arguments, asynchrony and errors as gefen_step.
 * ---------------------------------------------------------------------------- */
int gefen_step_fit(gefen_state* st, const gefen_tensor* params, const gefen_tensor* grads,
                   int32_t n_tensors, double lr, double beta1, double beta2, double eps,
                   double weight_decay, int64_t t, void* stream);

/* ------------------------------------------------------------------------------
 * gefen_fit_codebook -- refit the codebook (Alg. 3) on the gradients `grads`:
 * histogram of the block-absmax-normalised gradients (using the state's blocks),
 * then the exact DP on device. The new codebook is used to ENCODE at the next
 * gefen_step (whose decode still uses the previous codebook) and for both from the
 * step after. Asynchronous, no host synchronisation.
 * Errors: EINVAL, EDTYPE, EHIP. (Degenerate fits are reported by
 * gefen_get_fit_info, which synchronises.)
 * ---------------------------------------------------------------------------- */
int gefen_fit_codebook(gefen_state* st, const gefen_tensor* grads, int32_t n_tensors,
                       void* stream);

/* ------------------------------------------------------------------------------
 * Row-level entry points (each one step of the path on its own, on device).
 * ---------------------------------------------------------------------------- */

/* gefen_partition_scores -- Alg. 2 on one tensor: the divisors of numel in
 * increasing order, the score S(p) of each (partition-score equation; S(numel) = 0),
 * and the chosen period. divisors_out/scores_out are host arrays of `cap` entries;
 * *n_div receives the divisor count (EINVAL if it exceeds cap). Synchronises. */
int gefen_partition_scores(const gefen_tensor* grad, double eps_part, int64_t* divisors_out,
                           double* scores_out, int32_t cap, int32_t* n_div,
                           int64_t* period_out, void* stream);

/* gefen_histogram -- Alg. 3 histogram with the state's blocks: every block with
 * nonzero absmax a contributes each element x = g / a to bin
 * min(NB - 1, floor((x + 1) * NB / 2)), NB = 16 * k. hist_out is a device
 * uint64[NB]; it is overwritten. Asynchronous. */
int gefen_histogram(gefen_state* st, const gefen_tensor* grads, int32_t n_tensors,
                    uint64_t* hist_out, void* stream);

/* gefen_dp_codebook -- Alg. 3 / App. D exact DP over a histogram (device
 * uint64[nbins]) into k sorted entries with the first forced to -1 and the last to
 * +1. Outputs: codebook_out device double[k], cost_out device double[1],
 * status_out device int32[1] (0 ok, 1 degenerate: fewer non-empty bins than k, the
 * DP then uses max(b, 2) entries and pads with +1). Asynchronous; its workspace is
 * allocated and freed stream-ordered on `stream`.
 * Errors: EINVAL (NULL pointer, k outside [2, 256], nbins outside [1, 4096]), EHIP. */
int gefen_dp_codebook(const uint64_t* hist, int32_t nbins, int32_t k, double* codebook_out,
                      double* cost_out, int32_t* status_out, void* stream);

/* gefen_dp_codebook_static -- gefen_dp_codebook for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): the same DP, the same kernels and the same results, with its workspace in
 * one fixed array per GPU that the library holds until the process ends (11 MiB; enough
 * for the largest DP, 4096 bins and 256 entries). It calls no hipMalloc, hipFree or other
 * allocating routine. Arguments, outputs and errors as gefen_dp_codebook; a DP larger
 * than the fixed workspace is refused with EINVAL. The first call on a device looks up
 * that device's array (EHIP if the runtime cannot). Every call on one GPU shares that
 * GPU's array: calls that overlap on one GPU (different streams, or threads without
 * ordering) race and give undefined results; calls ordered on one stream do not. The
 * workspace needs no clearing: the DP writes every entry before reading it.
 * Asynchronous on `stream`. */
int gefen_dp_codebook_static(const uint64_t* hist, int32_t nbins, int32_t k,
                             double* codebook_out, double* cost_out, int32_t* status_out,
                             void* stream);

/* ------------------------------------------------------------------------------
 * Queries, state access and checkpointing.
 * ---------------------------------------------------------------------------- */

/* Periods per tensor (0 for tensors under explicit blocks). Host int64[n_tensors].
 * Errors: EINVAL (NULL). */
int gefen_get_periods(const gefen_state* st, int64_t* periods_out);

/* Layout of the state buffers (host int64 arrays of n_tensors + 1 entries each):
 * element e of tensor i has code index j = code_offsets[i] + e (code_offsets are
 * multiples of 32, so every tensor starts on a 16-byte boundary). With 8-bit codes,
 * code j is byte j of the codes buffer; with 4-bit codes it is the low (j even) or high
 * (j odd) nibble of byte j / 2. Tensor i's blocks are global block indices
 * [block_index[i], block_index[i+1]). total_code_bytes is the codes buffer's size.
 * Any output pointer may be NULL. Errors: EINVAL (NULL state). */
int gefen_get_layout(const gefen_state* st, int64_t* code_offsets, int64_t* block_index,
                     int64_t* total_code_bytes, int64_t* total_blocks, int32_t* k);

/* Copy state arrays to `dst` (host or device memory; stream-ordered). which:
 * 0 = codes (uint8[total_code_bytes]), 1 = scales (float[total_blocks]),
 * 2 = second moments (float[total_blocks]), 3 = decode codebook (float[k]),
 * 4 = encode codebook (float[k]), 5 = decode codebook in double (double[k]),
 * 6 = the Gefen-Muon bfloat16 momentum matrix (uint16[code index count], after
 * gefen_muon_init), 7 = the histogram of the last codebook fit (uint64[16 k]: init,
 * gefen_fit_codebook or gefen_step_fit); 5, 6 and 7 are read-only.
 * `bytes` must equal the array size. Synchronises `stream` when dst is host memory.
 * Errors: EINVAL (NULL, unknown `which`, 6 before gefen_muon_init, size mismatch), EHIP. */
int gefen_read_state(const gefen_state* st, int32_t which, void* dst, int64_t bytes,
                     void* stream);

/* Overwrite a state array from `src` (host or device), same `which` and sizes as
 * gefen_read_state, except 5, 6 and 7. Writing 3 or 4 installs a codebook (float[k]:
 * finite, first -1, last +1, never decreasing -- a degenerate fit repeats +1 at the
 * end; EINVAL otherwise) into that slot. */
int gefen_write_state(gefen_state* st, int32_t which, const void* src, int64_t bytes,
                      void* stream);

/* Result of the last codebook fit (init or gefen_fit_codebook): DP cost and
 * status (0 ok, 1 degenerate). Either output may be NULL. Synchronises `stream`.
 * Errors: EINVAL (NULL state), EHIP. */
int gefen_get_fit_info(const gefen_state* st, double* cost_out, int32_t* status_out,
                       void* stream);

/* Bytes of persistent device state (codes + scales + second moments + codebooks)
 * and of library workspace (tile tables, histogram and DP buffers). */
int gefen_state_bytes(const gefen_state* st, int64_t* persistent, int64_t* workspace);

/* Checkpoint: serialise the whole mutable state (codes, scales, second moments,
 * both codebook slots, slot indices) into `dst` (host or device) of exactly
 * gefen_checkpoint_bytes() bytes; gefen_import restores it into a state created
 * with the same tensors and blocks. Stream-ordered; synchronises for host memory.
 * gefen_import checks the header and the codebooks of the slots in use (decode and
 * encode; as gefen_write_state does) before it writes anything: on EINVAL the state
 * is unchanged. */
int gefen_checkpoint_bytes(const gefen_state* st, int64_t* bytes);
int gefen_export(const gefen_state* st, void* dst, int64_t bytes, void* stream);
int gefen_import(gefen_state* st, const void* src, int64_t bytes, void* stream);

/* ------------------------------------------------------------------------------
 * Measurement support. gefen_profile_begin arms per-launch timing for the next
 * `max_steps` calls of gefen_step: a pair of HIP events is recorded on the step's
 * stream around every step-kernel launch (one launch per kernel class: KIND 0 =
 * uniform blocks in registers, 1 = one streamed block per workgroup (or, with 8-bit
 * codes, a run of consecutive explicit blocks of 33-2042 elements in registers), 2 = one small
 * block per lane, 3 = blocks over 65536 elements split across workgroups (two
 * kernels, timed together), 4 = the leftover small tiles of all other classes in one
 * generic launch). gefen_profile_end synchronises those events and returns, for each
 * class (host arrays of `cap` entries): kind, vectors per lane (kind 0), workgroup
 * size, gradient dtype, number of timed launches, summed kernel time in milliseconds, elements per
 * launch and algorithmic HBM bytes per launch (per element: 8 for the parameter
 * read and write, 4 or 2 for the gradient, 2 (8-bit) or 1 (4-bit) for the code read
 * and write; per
 * block: 16 for scale and second moment read and write, plus 8 for an explicit block
 * offset read by the small-block kernel). It then disarms and frees the events.
 * Errors: EINVAL (NULL state or n_classes, max_steps < 1, cap below the class count),
 * EHIP (event creation or timing).
 * ---------------------------------------------------------------------------- */
int gefen_profile_begin(gefen_state* st, int32_t max_steps);
int gefen_profile_end(gefen_state* st, int32_t cap, int32_t* n_classes, int32_t* kind,
                      int32_t* vpl, int32_t* threads, int32_t* gdtype, int64_t* launches,
                      double* total_ms, int64_t* elems_per_launch, int64_t* bytes_per_launch);

/* ------------------------------------------------------------------------------
 * Gefen-Muon (appendix "Gefen-Muon"): Muon's momentum buffer held in Gefen's quantized
 * form (the state's codes, per-block scales and codebooks; its second moments are not
 * used), followed by Muon's Newton-Schulz orthogonalisation of each matrix.
 *
 * gefen_muon_init -- prepare a state made by gefen_init (same tensors, its inferred or
 * explicit blocks) for gefen_muon_step.
 *  rows    host int64[n_tensors]: tensor i is the rows[i] x (numel_i / rows[i]) matrix,
 *          row-major (a 1-D tensor is 1 x numel). rows[i] must divide numel_i.
 * Allocates the bfloat16 momentum matrix (2 bytes per parameter) and the Newton-Schulz
 * buffers of each of three lanes, sized for the lane's largest group of tensors that share
 * one wide shape (X and X^T twice, the two m x m products: about 8 bytes per element of
 * that group), and checks every matrix product of the steps against them on the host;
 * synchronises `stream`. Call once per state.
 * Errors: EINVAL (NULL, count mismatch, rows, second call, a matrix side above
 * 2^31 - 4096), ENOMEM, EHIP.
 * ---------------------------------------------------------------------------- */
int gefen_muon_init(gefen_state* st, const int64_t* rows, int32_t n_tensors, void* stream);

/* ------------------------------------------------------------------------------
 * gefen_muon_step -- one Gefen-Muon step. Per block B of the quantized buffer:
 *   m_i = mu * c_dec[q_i] * s_B + (1 - mu) * g_i;  s_B' = max_B |m_i|;
 *   q_i' = nearest entry of c_enc to m_i / s_B'   (ties to the lower index)
 * per tensor (a rows x cols matrix):
 *   U = nesterov ? (1 - mu) * G + mu * M : M, rounded to bfloat16
 *   X = bf16(U / max(bf16(||U||_F), bf16(ns_eps))), transposed if rows > cols
 *   ns_steps times: A = X X^T; B = ns_b A + ns_c A A; X = ns_a X + B X
 *       (bfloat16 matrices, float32 accumulation, each product rounded once, as Muon's
 *       PyTorch implementation; the library's own matrix-core kernels)
 *   theta = theta * (1 - lr * weight_decay) - lr * sqrt(max(1, rows / cols)) * X^(T)
 *  params, grads  as for gefen_step; momentum in [0, 1); ns_steps in [0, 100];
 *  ns_eps > 0. Muon's defaults: ns_steps 5, (ns_a, ns_b, ns_c) =
 *  (3.4445, -4.7750, 2.0315), ns_eps 1e-7, nesterov 1.
 * Asynchronous on `stream`; no allocation. The shape groups are split over three lanes
 * that run concurrently: one on `stream`, the others on streams the state owns, which
 * wait for the norms on `stream`; `stream` then waits for them, so all of the step's
 * work is ordered before later work on `stream`. Refits (gefen_fit_codebook) apply as for
 * gefen_step. The bfloat16 momentum matrix of the last step can be read as array 6 of
 * gefen_read_state (uint16 bit patterns at each element's code index).
 * Errors: EINVAL (arguments, gefen_muon_init not called), EDTYPE, EHIP.
 * ---------------------------------------------------------------------------- */
int gefen_muon_step(gefen_state* st, const gefen_tensor* params, const gefen_tensor* grads,
                    int32_t n_tensors, double lr, double momentum, double weight_decay,
                    int32_t nesterov, int32_t ns_steps, double ns_a, double ns_b, double ns_c,
                    double ns_eps, void* stream);

/* Measurement of Gefen-Muon steps (after gefen_muon_init and gefen_profile_begin):
 * sums over the profiled steps of the codec time (codec and norms) and of the
 * orthogonalisation wall time (normalise, Newton-Schulz and update of every shape
 * group, on all of the step's streams, from the end of the norms to the joins), in
 * milliseconds, from HIP events on the step's stream; then disarms like
 * gefen_profile_end. Errors: EINVAL (NULL), EHIP. */
int gefen_muon_profile_end(gefen_state* st, int32_t* steps, double* codec_ms, double* ortho_ms);

/* ------------------------------------------------------------------------------
 * gefen_newton_schulz -- Muon's orthogonalisation iterations (appendix "Gefen-Muon"),
 * the matrix-product part of gefen_muon_step on its own: `steps` times
 *   A = X X^T;  B = b A + c A A;  X = a X + B X
 * on each of `batch` wide bfloat16 matrices, every product rounded once to bfloat16 from
 * float32 accumulation (the same kernels as gefen_muon_step). No normalisation: x_in is
 * the first iteration's input.
 *  x_in   device uint16[batch * m * n]: bfloat16 bit patterns, matrix b row-major m x n
 *         at x_in + b * m * n, 1 <= m <= n <= 2^31 - 4096, batch in [1, 65535].
 *  x_out  device uint16[batch * m * n], same layout; may equal x_in.
 *  steps  in [0, 100] (0 copies x_in to x_out); a, b, c finite.
 * Asynchronous on `stream`; its workspace (about 8 bytes per element of the batch) is
 * allocated and freed stream-ordered on `stream`.
 * Errors: EINVAL (NULL, sizes, steps, coefficients), ENOMEM, EHIP.
 * ---------------------------------------------------------------------------- */
int gefen_newton_schulz(const uint16_t* x_in, uint16_t* x_out, int32_t batch, int64_t m,
                        int64_t n, int32_t steps, double a, double b, double c, void* stream);

/* ------------------------------------------------------------------------------
 * gefen_stream_mix -- measurement support: the practical HBM ceiling for the step's
 * access mix. One pass over n elements that reads and writes `theta` (float32), reads
 * `grad` (GEFEN_F32 or GEFEN_BF16) and reads and writes `codes` (one byte per element),
 * with none of the optimizer's arithmetic (two lanes of each theta vector gain the
 * gradient, every code byte flips its low bit). It uses the tile shape that moves this
 * mix fastest: one-shot tiles of 1024 elements, 256 threads, one 16-byte parameter
 * vector per thread, non-temporal accesses.
 * Bytes moved: n * (8 + 4 or 2 + 2), the step's per-element algorithmic bytes.
 *  theta, grad, codes  caller-owned device arrays of n elements; modified in place
 *                      (theta and codes). theta 16-byte aligned, grad 16 (F32) or 8
 *                      (BF16) byte aligned, codes 4-byte aligned.
 * Asynchronous on `stream`. n = 0 is a no-op.
 * Errors: EINVAL (n < 0, NULL array, misaligned pointer), EDTYPE, EHIP.
 * ---------------------------------------------------------------------------- */
int gefen_stream_mix(float* theta, const void* grad, int32_t grad_dtype, uint8_t* codes,
                     int64_t n, void* stream);

/* Free the state and every device buffer it owns. NULL is a no-op. */
void gefen_destroy(gefen_state* st);

/* Message of the last failing call on this thread ("" if none). */
const char* gefen_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* GEFEN_H */
