/*
 * onebit.h -- C ABI of the 1-bit Adam hot path on AMD Instinct MI355X (gfx950).
 *
 * Method: Tang et al., "1-bit Adam: Communication Efficient Large-Scale
 * Training with Adam's Convergence Speed" (arXiv 2102.02888).  Warm-up runs
 * original Adam (eq. (alg:v), Section 3.3); the compression stage freezes the
 * variance and runs error-compensated 1-bit compressed momentum SGD
 * (Algorithm 1, Section 4.3) whose averaging is the three-phase "compressed
 * allreduce" of Section 6 / Figure "allreduce" (all-to-all of chunks, average
 * on each chunk owner, all-gather).  On one GPU the n data-parallel workers
 * are rows of HBM buffers and the exchange is addressing: chunk j of every
 * worker row is read in place by the kernel that plays chunk owner j.
 *
 * ---------------------------------------------------------------------------
 * Conventions shared by every entry point
 * ---------------------------------------------------------------------------
 * Layout.  A plan describes K tensors of numel d_k and n workers.  Tensor k
 *   starts at element off_k (off_0 = 0, off_{k+1} = off_k + 64*ceil(d_k/64));
 *   D = padded total, W = D/64 words.  Each tensor is cut into n chunks of
 *   c_k = 64*ceil(d_k/(64 n)) elements; chunk j of tensor k is segment
 *   q = k*n + j, covering [off_k + min(j c_k, d_k), off_k + min((j+1) c_k, d_k)).
 *   Trailing segments may be short or empty.  Chunk owner ("server") j owns
 *   segments (k, j) for all k.  Padding elements are never written.
 * Compressed message (Section 4.3): one sign bit per element plus one fp32
 *   scale per segment, scale = ||z||_2 / sqrt(len) so the decoded vector
 *   +-scale has the l2 magnitude of z.  Bit (e mod 64) of uint64 word (e/64)
 *   belongs to flat element e; bit 1 <=> z >= 0 (+0 and -0 give 1, NaN 0);
 *   bits of padding elements are 0.  An empty segment has scale 0.
 * Arithmetic.  fp32 state; each fp32 operation rounded once (no FMA
 *   contraction); reductions (gradient average, sum of squares, server sum of
 *   decoded messages) in fp64, rounded once to fp32.  sqrt and division are
 *   correctly rounded.
 * Error state (compensated form).  An error buffer (a worker row of
 *   worker_err, or server_err) does not hold the error delta itself: it holds
 *   z, the compensated value that was last compressed, and the scale array
 *   written by that same call holds s.  The error is
 *       delta = (z >= 0) ? z - s : z + s          (i.e. z - C[z])
 *   and is formed inside the next call from the pair, which saves a second
 *   pass over the buffer.  All-zero buffers and scales mean delta = 0.  To
 *   load an explicit delta, write it into the error buffer and zero the
 *   matching scales; onebit_error_materialize() produces explicit delta.
 * Pointers.  Every buffer pointer is a device pointer on the plan's device;
 *   element buffers (sized by D or W) may be NULL only when the plan has no
 *   elements (D = 0), where calls touch nothing but the segment scales.
 *   fp32 buffers must be 16-byte aligned and leading dimensions (in elements)
 *   multiples of 4; uint64 bit buffers 8-byte aligned.  The caller owns every
 *   buffer; calls never allocate, never synchronize the host and never read
 *   device data back.  Buffers written by a call must not alias any other
 *   buffer of that call except where "in/out" says so.
 * Streams.  Every call is asynchronous on `stream` (0 = the null stream).  A
 *   plan may be used from several streams if each has its own workspace.
 * Graphs.  Every call that takes a stream issues only kernel launches on it
 *   (no memset, copy, allocation or host synchronisation), so such a call or
 *   a sequence of them may be captured into a HIP graph and replayed; the
 *   graph keeps the pointers and scalar arguments given at capture.  Plan
 *   creation and destruction allocate and copy, and are not captured.
 * Errors.  Every function returns ONEBIT_OK (0) or a negative status; on an
 *   error nothing is launched and no buffer is written.  onebit_status_str()
 *   names a status and onebit_last_error() describes the last failure of the
 *   calling thread.
 */
#ifndef ONEBIT_H
#define ONEBIT_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ONEBIT_OK 0
#define ONEBIT_EINVAL (-1) /* null pointer, bad size, n, range or leading dim */
#define ONEBIT_EALIGN (-2) /* misaligned pointer or leading dimension        */
#define ONEBIT_EHIP (-3)   /* HIP runtime or launch error                    */
#define ONEBIT_ENOMEM (-4) /* device allocation failed (plan creation only)  */

/* Gradient element types.  16-bit gradients are widened to fp32 exactly on
 * load, so every later operation is the fp32 arithmetic described above. */
#define ONEBIT_GRAD_F32 0
#define ONEBIT_GRAD_BF16 1
#define ONEBIT_GRAD_F16 2

typedef struct onebit_plan_s *onebit_plan;
typedef struct ihipStream_t *onebit_stream; /* a hipStream_t */

typedef struct {
    int64_t d;               /* real elements, sum of d_k                  */
    int64_t padded_len;      /* D                                           */
    int64_t words;           /* W = D / 64                                  */
    int64_t num_tensors;     /* K                                           */
    int64_t num_segments;    /* S = K * n                                   */
    int64_t num_tiles;       /* work tiles (<= 1024 elements, one segment)  */
    int32_t n_workers;       /* n                                           */
    int32_t tile_elems;      /* elements per full tile                      */
    size_t workspace_bytes;  /* workspace needed by the calls below: per-tile
                                partial sums, and the chunk owners' lookup
                                tables (2 KB per segment and group of 8
                                workers) when those of all S segments fit
                                in 32 MiB                                   */
} onebit_plan_sizes;

/* Creates a plan for K = num_tensors tensors (tensor_numel[k] >= 0, host
 * array) and n = n_workers >= 1 workers on the current HIP device.  The plan
 * owns small device tables (tiles, segments); *out receives the handle.
 * Errors: EINVAL (null, K < 1, n < 1, a numel below 0 or above 2^40,
 * D >= 2^40, 2^25 or more tiles, more than 2^31 - 1 segments), ENOMEM,
 * EHIP. */
int onebit_plan_create(const int64_t *tensor_numel, int32_t num_tensors,
                       int32_t n_workers, onebit_plan *out);

/* Frees the plan's device tables.  The caller must ensure no call using the
 * plan is still running on any stream. */
int onebit_plan_destroy(onebit_plan plan);

/* Copies the plan's sizes into *info (host struct). */
int onebit_plan_get_info(onebit_plan plan, onebit_plan_sizes *info);

/* Host copies of the layout: tensor_offset[K], seg_begin[S], seg_end[S]
 * (element indices into the padded buffer).  Any output may be NULL. */
int onebit_plan_get_layout(onebit_plan plan, int64_t *tensor_offset,
                           int64_t *seg_begin, int64_t *seg_end);

/* Where the chunk owners' calls on this plan take their lookup tables from
 * (the signed sums of the scales of each group of 8 workers, Algorithm 1's
 * server average): built once per call in the workspace (possible when the
 * plan reserved the space, see workspace_bytes) or built for every tile.
 * ONEBIT_SERVER_TABLES_AUTO (the default) uses the workspace when the call's
 * segments average 4 or more tiles and its tiles times its groups of 8
 * workers reach 32768; ON uses it whenever the space is there; OFF never.
 * Results are bit-identical either way; the switch exists to compare the two
 * paths.  Not to be changed while a call on the plan is in flight.
 * Errors: EINVAL (null plan, another mode). */
#define ONEBIT_SERVER_TABLES_OFF 0
#define ONEBIT_SERVER_TABLES_AUTO 1
#define ONEBIT_SERVER_TABLES_ON 2
int onebit_plan_set_server_tables(onebit_plan plan, int32_t mode);

/* The sizes a caller allocates by, as separate host outputs (any may be
 * NULL): D, W, S, the chunk length c_k of every tensor (chunk_len[K], see
 * Layout above) and the workspace size in bytes for the calls below. */
int onebit_plan_info(onebit_plan plan, int64_t *padded_len, int64_t *words,
                     int64_t *num_segments, int64_t *chunk_len,
                     size_t *workspace_bytes);

/* Warm-up step: original Adam on the data-parallel average gradient
 * (eq. (alg:v), Section 3.3; Algorithm 1's warm-up stage):
 *   g = (1/n_grads) sum_i grads[i]      (fp64 sum in row order, one rounding)
 *   m = beta1 m + (1-beta1) g ;  v = beta2 v + (1-beta2) g*g
 *   x = x - lr * m_hat / (sqrt(v_hat) + eps)
 * with m_hat = m, v_hat = v when bias_correction == 0 (the paper's choice)
 * and m_hat = m/(1-beta1^step), v_hat = v/(1-beta2^step) otherwise (step is
 * 1-based; the factors are computed in fp64 on the host and rounded to fp32).
 * x, m, v: in/out [D].  grads: n_grads rows of grad_ld >= D elements of type
 * grad_dtype (ONEBIT_GRAD_F32, _BF16 or _F16; 16-byte aligned for fp32, 8-byte
 * for 16-bit types; n_grads = 1 when the caller already holds the averaged
 * gradient).  The v left after
 * the last warm-up step is the frozen variance of the compression stage.
 * Errors: EINVAL (null, n_grads < 1, grad_ld < D, step < 1, unknown
 * grad_dtype), EALIGN, EHIP. */
int onebit_warmup_adam_step(onebit_plan plan, float *x, float *m, float *v,
                            const void *grads, int32_t grad_dtype, int64_t grad_ld,
                            int32_t n_grads,
                            float lr, float beta1, float beta2, float eps,
                            int32_t bias_correction, int64_t step,
                            onebit_stream stream);

/* Worker side of a compression step for n_local simulated workers
 * (Algorithm 1, local momentum, compression and error update):
 *   m_i   = beta1 m + (1-beta1) grads[i]    (m: the shared momentum m_{t-1})
 *   z_i   = m_i + delta_i                   (delta_i from the error state)
 *   bits, scale per segment = C[z_i]        ;  delta_i <- z_i - C[z_i]
 * The shared momentum comes from one of two places.  m != NULL: an fp32
 * buffer [D] (the warm-up's m before the first compression step).  m == NULL:
 * the previous step's gathered server message, m = bit ? scale : -scale with
 * its sign words m_bits [W] and segment scales m_scales [S] -- Algorithm 1
 * sets every worker's momentum to that decoded message, so it never has to be
 * stored as fp32 ("packed momentum"; 1/8 byte per element instead of 4).
 * grads: n_local rows of grad_ld >= D elements of type grad_dtype.  worker_err: in/out,
 * n_local rows of err_ld >= D (compensated form, see above).  worker_bits:
 * out, n_local rows of bits_ld >= W words.  worker_scales: in/out, n_local
 * rows of scales_ld >= S floats (in: the previous call's scales, which with
 * worker_err form the error state; out: this step's scales).  workspace:
 * >= workspace_bytes of device memory, contents undefined between calls.
 * Errors: EINVAL (null, n_local < 1 or > n, a leading dim too small, m and
 * m_bits/m_scales both NULL), EALIGN, EHIP. */
int onebit_worker_compress(onebit_plan plan, const float *m, const uint64_t *m_bits,
                           const float *m_scales, const void *grads, int32_t grad_dtype,
                           int64_t grad_ld, int32_t n_local,
                           float *worker_err, int64_t err_ld,
                           uint64_t *worker_bits, int64_t bits_ld,
                           float *worker_scales, int64_t scales_ld,
                           float beta1, void *workspace, onebit_stream stream);

/* Chunk-owner side for chunks [server_begin, server_end) (Algorithm 1's
 * server average and recompression; Figure "allreduce" average step):
 *   avg   = (1/n) sum_{i<n} decode(bits_i, scale_i)   (fp64, one rounding)
 *   z_bar = avg + delta_bar ;  bits, scale = C[z_bar] ;  delta_bar <- z_bar - C[z_bar]
 * Incoming messages of all n workers: the bit word of worker row i for
 * global word w is worker_bits[i*bits_ld + (w - bits_word_base)] and its
 * scale for segment q is worker_scales[i*scales_ld + (q - scales_seg_base)].
 * The simulated all-to-all is bits_ld = W, bits_word_base = 0, scales_ld = S,
 * scales_seg_base = 0 (the worker_compress outputs as they are).  A real
 * received buffer of one chunk j (rows of chunk j's words, one scale per row)
 * uses bits_word_base = first word of chunk j and scales_seg_base = q.
 * server_err: in/out [D] (compensated form; only the owned segments are
 * touched).  server_bits: out [W], server_scales: in/out [S]; only the owned
 * segments' words and scales are written (the rest stand for what the
 * all-gather brings from the other chunk owners).
 * Errors: EINVAL (null, empty or out-of-range chunk range, a base or leading
 * dim that does not cover the owned segments), EALIGN, EHIP. */
int onebit_server_reduce_compress(onebit_plan plan, int32_t server_begin,
                                  int32_t server_end,
                                  const uint64_t *worker_bits, int64_t bits_ld,
                                  int64_t bits_word_base,
                                  const float *worker_scales, int64_t scales_ld,
                                  int64_t scales_seg_base,
                                  float *server_err, uint64_t *server_bits,
                                  float *server_scales, void *workspace,
                                  onebit_stream stream);

/* Every worker after the all-gather (Algorithm 1, final step): decode the
 * averaged momentum and take the frozen-variance preconditioned step
 *   m_bar = bit ? scale : -scale ;  x = x - lr * m_bar / sqrt(v_frozen + eps)
 *   m = m_bar (when m_out is not NULL)
 * over every real element.  server_bits [W], server_scales [S]: in.  x: in/out
 * [D]; m_out: out [D] or NULL; v_frozen: in [D].
 * Errors: EINVAL, EALIGN, EHIP. */
int onebit_decompress_update(onebit_plan plan, const uint64_t *server_bits,
                             const float *server_scales, float *x, float *m_out,
                             const float *v_frozen, float lr, float eps,
                             onebit_stream stream);

/* One whole compression-stage step with all n workers and all n chunk owners
 * simulated on this GPU: onebit_worker_compress (n_local = n, bits rows of W,
 * scales rows of S, in worker_bits / worker_scales), then
 * onebit_server_reduce_compress over chunks [0, n) reading those rows in
 * place, then onebit_decompress_update with m_out = m.
 * m != NULL: fp32 momentum, read by the worker pass and overwritten with the
 * decoded server message.  m == NULL: packed momentum -- the worker pass
 * decodes m from server_bits / server_scales as the previous step left them,
 * and no fp32 momentum is written (valid from the second compression step on;
 * onebit_decode() materialises it on demand).
 * x: in/out [D]; v_frozen: in [D]; grads: n rows of grad_ld;
 * worker_err: in/out n rows of err_ld; server_err: in/out [D];
 * worker_bits [n][W], worker_scales [n][S] (in/out), server_bits [W],
 * server_scales [S] (in/out).
 * Errors: those of the three calls. */
int onebit_step(onebit_plan plan, float *x, float *m, const float *v_frozen,
                const void *grads, int32_t grad_dtype, int64_t grad_ld, float *worker_err,
                int64_t err_ld, float *server_err, uint64_t *worker_bits,
                float *worker_scales, uint64_t *server_bits, float *server_scales,
                float lr, float beta1, float eps, void *workspace,
                onebit_stream stream);

/* onebit_step for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc): the
 * same launches and results, with no workspace argument.  The per-tile
 * partial sums go to the library's own static device array of
 * ONEBIT_NOALLOC_SCRATCH_BYTES (96 MiB), which every GPU the library runs on
 * holds until the process ends; its address is looked up on the first call
 * on each device.  The call allocates and frees nothing.  Every call on one
 * GPU shares that GPU's array: calls that overlap on one GPU (other streams,
 * other threads, other plans) race and must be serialised by the caller.
 * Nothing in the array needs clearing between calls (each step writes every
 * partial and table entry it reads).  Errors: those of onebit_step; EINVAL
 * when the plan's workspace_bytes (about 8 (n + 1) bytes per tile of 1024
 * elements, plus 2 KB per segment and group of 8 workers when the plan keeps
 * the chunk owners' tables) exceeds ONEBIT_NOALLOC_SCRATCH_BYTES -- a
 * BERT-Large-shaped buffer of 334M parameters with n = 32 needs 86 MB and
 * fits; EHIP if the array's address cannot be found. */
#define ONEBIT_NOALLOC_SCRATCH_BYTES ((size_t)96 << 20)
int onebit_step_noalloc(onebit_plan plan, float *x, float *m, const float *v_frozen,
                        const void *grads, int32_t grad_dtype, int64_t grad_ld,
                        float *worker_err, int64_t err_ld, float *server_err,
                        uint64_t *worker_bits, float *worker_scales, uint64_t *server_bits,
                        float *server_scales, float lr, float beta1, float eps,
                        onebit_stream stream);

/* onebit_step with timing marks, to profile the fused step phase by phase:
 * the same launches, and in addition hipEventRecord(events[k], stream)
 * before the worker pass (k = 0), before the chunk owners' pass (k = 1),
 * before the update (k = 2) and after it (k = 3).  events: a host array of
 * four hipEvent_t (void *) created by the caller, with timing enabled to read
 * elapsed times; a NULL entry skips that mark.  The marks add no host
 * synchronisation; a call with events is not meant for graph capture.
 * Errors: those of onebit_step (all checked before the first launch or
 * mark), EINVAL if events is NULL, EHIP if a record fails. */
int onebit_step_events(onebit_plan plan, float *x, float *m, const float *v_frozen,
                       const void *grads, int32_t grad_dtype, int64_t grad_ld,
                       float *worker_err, int64_t err_ld, float *server_err,
                       uint64_t *worker_bits, float *worker_scales, uint64_t *server_bits,
                       float *server_scales, float lr, float beta1, float eps,
                       void *workspace, void *const *events, onebit_stream stream);

/* Comparison variants of Section 7.2 (not part of 1-bit Adam itself). */

/* "1-bit Adam (32-bits)": the compression stage with the identity compressor
 * -- variance frozen, momenta averaged uncompressed:
 *   m_i = beta1 m + (1-beta1) grads[i];  m = (1/n) sum_i m_i (fp64, one rounding)
 *   x = x - lr * m / sqrt(v_frozen + eps)
 * x, m: in/out [D]; v_frozen: in [D]; grads: n_grads rows of grad_ld >= D
 * elements of grad_dtype.  Errors: EINVAL, EALIGN, EHIP. */
int onebit_uncompressed_step(onebit_plan plan, float *x, float *m, const float *v_frozen,
                             const void *grads, int32_t grad_dtype, int64_t grad_ld,
                             int32_t n_grads, float lr, float beta1, float eps,
                             onebit_stream stream);

/* Adam step (eq. (alg:v)) whose gradient is a decoded message,
 * g = bit ? scale : -scale: the update of "Adam(1-bit Naive)", which
 * error-compensates and compresses the gradient (onebit_worker_compress with
 * beta1 = 0 and a zero momentum, then onebit_server_reduce_compress) and
 * updates both m and v from the result, without freezing v.  Bias correction
 * as in onebit_warmup_adam_step.  x, m, v: in/out [D]; bits [W], scales [S]:
 * in.  Errors: EINVAL, EALIGN, EHIP. */
int onebit_adam_message_step(onebit_plan plan, float *x, float *m, float *v,
                             const uint64_t *bits, const float *scales, float lr, float beta1,
                             float beta2, float eps, int32_t bias_correction, int64_t step,
                             onebit_stream stream);

/* Variance-stability indicator (Section 7.1, warm-up auto-tuning): the l1
 * norm ||v||_1 = sum_e |v[e]| over every real element, summed in fp64 in a
 * fixed order (per-tile partials, then one ordered pass), written to *out.
 * The warm-up can be stopped at the first step t (not before the learning-rate
 * warm-up ends) with ||v_t||_1 / ||v_{t-Delta}||_1 >= 0.96, Delta = 1/(1-beta2);
 * keeping the history of norms and taking that decision is host logic.
 * v: in [D]; workspace: as for the step calls (its server partial area is
 * used); out: device pointer to one double (8-byte aligned).
 * Errors: EINVAL, EALIGN, EHIP. */
int onebit_l1_norm(onebit_plan plan, const float *v, void *workspace, double *out,
                   onebit_stream stream);

/* Decoded message: out[e] = bit(e) ? scales[q] : -scales[q] over every real
 * element e of segment q (padding of out is not written).  With the server
 * bits and scales this is the momentum m_t of Algorithm 1's final step.
 * bits [W], scales [S]: in; out: out [D].  Errors: EINVAL, EALIGN, EHIP. */
int onebit_decode(onebit_plan plan, const uint64_t *bits, const float *scales, float *out,
                  onebit_stream stream);

/* Explicit errors from the compensated form: for `rows` rows,
 *   delta_out[r*out_ld + e] = z - C[z] with z = err_state[r*err_ld + e] and
 *   the scale of e's segment from scales[r*scales_ld + q]
 * over every real element (padding of delta_out is not written).  For the
 * server error use rows = 1.  delta_out may equal err_state (same ld) to
 * convert in place; the scales must then be zeroed by the caller to keep the
 * pair consistent.
 * Errors: EINVAL, EALIGN, EHIP. */
int onebit_error_materialize(onebit_plan plan, const float *err_state,
                             int64_t err_ld, const float *scales,
                             int64_t scales_ld, int32_t rows, float *delta_out,
                             int64_t out_ld, onebit_stream stream);

/* Name of a status code (static string). */
const char *onebit_status_str(int32_t status);

/* Description of the calling thread's last failure (static per thread). */
const char *onebit_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* ONEBIT_H */
