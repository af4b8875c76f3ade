/*
 * onebit_oracle.c -- TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT.
 *
 * A plain, slow, single-threaded CPU statement of what the 1-bit Adam hot
 * path computes (Tang et al., "1-bit Adam: Communication Efficient
 * Large-Scale Training with Adam's Convergence Speed", arXiv 2102.02888).
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg
 * may call it.  It shares no code, header, table or helper with the GPU
 * library, and the GPU library never calls it.
 *
 * Arithmetic model (the precision the GPU path also uses, so that both sides
 * take every sign decision in the same precision):
 *   - state (x, m, v, worker errors, server error) is IEEE binary32;
 *   - every written fp32 operation is rounded once, round-to-nearest-even,
 *     never contracted into an FMA (build with -ffp-contract=off, no
 *     fast-math);
 *   - reductions (the warm-up gradient average, the squared norm behind a
 *     scale, the server's sum of decoded worker messages) accumulate in
 *     binary64 in plain index order and are rounded to binary32 once.
 *
 * Layout convention (a reading of the chunked exchange of Section 6 and of
 * the per-chunk parameter-server equivalence in the appendix "Proof to the
 * updating form"; the paper leaves the cut of a tensor into n chunks open):
 *   - tensor k of numel d_k starts at off_k; off_0 = 0 and
 *     off_{k+1} = off_k + 64*ceil(d_k/64); D is the padded total;
 *   - chunk length c_k = 64*ceil(d_k/(64 n)); chunk j of tensor k is the
 *     segment q = k*n + j covering [off_k + min(j c_k, d_k),
 *     off_k + min((j+1) c_k, d_k)); trailing segments may be short or empty;
 *   - the sign bit of flat element e is bit (e mod 64) of 64-bit word
 *     (e div 64); bit = 1 means the element is >= 0 (so +0 and -0 give 1,
 *     NaN gives 0); bits of padding elements are 0;
 *   - an empty segment has scale 0.
 * Padding elements are never read or written.
 *
 * What pins each function (tests/test_oracle_pins.py, tests/test_freeze_cpu.py;
 * none is "parity unpinned"):
 *   orc_chunk_len, orc_layout  brute-force chunk membership, the BERT sizes
 *   orc_compress               numpy.packbits, numpy.linalg.norm, the
 *                              correctly rounded fp32 of the exact rational
 *                              root mean square, +-0/NaN/empty segments,
 *                              equal-magnitude inputs (exact, zero error)
 *   orc_decode(_range)         the hand-worked example's decoded momentum
 *   orc_warmup_range           torch.optim.Adam (with and without bias
 *                              correction), a constant-gradient closed form,
 *                              the variance's closed form
 *   orc_l1_norm_range          an exact (fractions) sum
 *   orc_worker_segment,        the hand-worked two-step example, the
 *   orc_server_segment,        error-feedback identity, the appendix's
 *   orc_update_segment,        telescoping form, identical workers, n = 1,
 *   orc_step                   chunk independence, the exact rational mean
 *                              of the decoded messages, a checkpoint resume
 *   orc_step_uncompressed_range  torch.optim.SGD momentum (change of variables)
 */
#include <math.h>
#include <stdint.h>
#include <stddef.h>

/* ------------------------------------------------------------------------ */
/* Layout                                                                    */
/* ------------------------------------------------------------------------ */

static int64_t round_up64(int64_t a) { return ((a + 63) / 64) * 64; }

/* Chunk length of a tensor of d elements cut into n chunks (64-aligned). */
int64_t orc_chunk_len(int64_t d, int32_t n)
{
    if (d <= 0) return 0;
    int64_t per = (d + (int64_t)n * 64 - 1) / ((int64_t)n * 64);
    return per * 64;
}

/* Fills tensor offsets [K] and segment bounds [K*n] (begin, end); returns D. */
int64_t orc_layout(const int64_t *numel, int32_t K, int32_t n,
                   int64_t *tensor_off, int64_t *seg_begin, int64_t *seg_end)
{
    int64_t off = 0;
    for (int32_t k = 0; k < K; ++k) {
        tensor_off[k] = off;
        int64_t d = numel[k];
        int64_t c = orc_chunk_len(d, n);
        for (int32_t j = 0; j < n; ++j) {
            int64_t b = (int64_t)j * c, e = (int64_t)(j + 1) * c;
            if (b > d) b = d;
            if (e > d) e = d;
            seg_begin[(int64_t)k * n + j] = off + b;
            seg_end[(int64_t)k * n + j] = off + e;
        }
        off += round_up64(d);
    }
    return off;
}

/* ------------------------------------------------------------------------ */
/* The compression operator C (Section 4.3): one sign bit per element plus  */
/* one scaling factor chosen so that the compressed vector has the same     */
/* l2 magnitude as its input: scale = ||z||_2 / ||sign(z)||_2               */
/*                                  = sqrt(sum z^2 / len).                  */
/* ------------------------------------------------------------------------ */

static int sign_bit(float z) { return z >= 0.0f; }

static void set_bit(uint64_t *bits, int64_t e, int b)
{
    uint64_t mask = (uint64_t)1 << (e & 63);
    if (b) bits[e >> 6] |= mask;
    else bits[e >> 6] &= ~mask;
}

static int get_bit(const uint64_t *bits, int64_t e)
{
    return (int)((bits[e >> 6] >> (e & 63)) & 1u);
}

/* C[z] on elements [b, e): writes the sign bits, returns the scale. */
float orc_compress(int64_t b, int64_t e, const float *z, uint64_t *bits)
{
    int64_t len = e - b;
    if (len <= 0) return 0.0f;
    double sum_sq = 0.0;
    for (int64_t idx = b; idx < e; ++idx) {
        double zd = (double)z[idx];
        sum_sq += zd * zd;
    }
    for (int64_t idx = b; idx < e; ++idx) set_bit(bits, idx, sign_bit(z[idx]));
    return (float)sqrt(sum_sq / (double)len);
}

/* Decoded value of element e of a compressed message: +scale or -scale. */
float orc_decode(const uint64_t *bits, int64_t e, float scale)
{
    return get_bit(bits, e) ? scale : -scale;
}

/* Decoded message over elements [b, e): out[idx] = +scale or -scale. */
void orc_decode_range(int64_t b, int64_t e, const uint64_t *bits, float scale, float *out)
{
    for (int64_t idx = b; idx < e; ++idx) out[idx] = orc_decode(bits, idx, scale);
}

/* ------------------------------------------------------------------------ */
/* Warm-up: original Adam, eq. (alg:v) of Section 3.3, on the averaged      */
/* data-parallel gradient (problem statement (main)).  The paper disables   */
/* bias correction; bias_correction != 0 gives the textbook Kingma-Ba form. */
/* Works on elements [b, e).  g has n rows of stride g_ld.                   */
/* ------------------------------------------------------------------------ */
void orc_warmup_range(int64_t b, int64_t e, float *x, float *m, float *v,
                      const float *g, int64_t g_ld, int32_t n,
                      float lr, float beta1, float beta2, float eps,
                      int32_t bias_correction, int64_t t)
{
    const float one_minus_beta1 = 1.0f - beta1;
    const float one_minus_beta2 = 1.0f - beta2;
    float bc1 = 1.0f, bc2 = 1.0f;
    if (bias_correction) {
        bc1 = (float)(1.0 - pow((double)beta1, (double)t));
        bc2 = (float)(1.0 - pow((double)beta2, (double)t));
    }
    for (int64_t idx = b; idx < e; ++idx) {
        double sum = 0.0;
        for (int32_t i = 0; i < n; ++i) sum += (double)g[(int64_t)i * g_ld + idx];
        float g_avg = (float)(sum / (double)n);

        float m_new = beta1 * m[idx];
        m_new = m_new + one_minus_beta1 * g_avg;
        float g_sq = g_avg * g_avg;
        float v_new = beta2 * v[idx];
        v_new = v_new + one_minus_beta2 * g_sq;
        m[idx] = m_new;
        v[idx] = v_new;

        float m_hat = m_new, v_hat = v_new;
        if (bias_correction) {
            m_hat = m_new / bc1;
            v_hat = v_new / bc2;
        }
        float denom = sqrtf(v_hat) + eps;
        float ratio = m_hat / denom;
        float step = lr * ratio;
        x[idx] = x[idx] - step;
    }
}

/* The l1 norm of v over [b, e) in binary64, index order (the warm-up's
 * variance-stability indicator ||v||_1 of Section 7.1). */
double orc_l1_norm_range(int64_t b, int64_t e, const float *v)
{
    double s = 0.0;
    for (int64_t idx = b; idx < e; ++idx) s += fabs((double)v[idx]);
    return s;
}

/* ------------------------------------------------------------------------ */
/* Compression stage, Algorithm 1, one segment [b, e) at a time (each       */
/* segment is an independent parameter-server problem).                      */
/* ------------------------------------------------------------------------ */

/* Worker i: momentum from the shared m_{t-1} and the local gradient, error
 * compensation, compression, and the new worker error.
 *   m_i   = beta1 * m + (1 - beta1) * g_i
 *   z     = m_i + delta_i            (compensated momentum)
 *   m_hat = C[z]                     (bits + scale; returned scale)
 *   delta_i <- z - m_hat                                                  */
float orc_worker_segment(int64_t b, int64_t e, float beta1,
                         const float *m, const float *g_i,
                         float *delta_i, uint64_t *bits_i, float *z_scratch)
{
    const float one_minus_beta1 = 1.0f - beta1;
    for (int64_t idx = b; idx < e; ++idx) {
        float m_i = beta1 * m[idx];
        m_i = m_i + one_minus_beta1 * g_i[idx];
        z_scratch[idx] = m_i + delta_i[idx];
    }
    float scale = orc_compress(b, e, z_scratch, bits_i);
    for (int64_t idx = b; idx < e; ++idx) {
        float m_hat = orc_decode(bits_i, idx, scale);
        delta_i[idx] = z_scratch[idx] - m_hat;
    }
    return scale;
}

/* Server: average of the n decoded worker messages (binary64 sum in worker
 * order, one rounding), server error compensation, recompression, new
 * server error.
 *   avg     = (1/n) sum_i m_hat_i
 *   z_bar   = avg + delta_bar
 *   m_bar   = C[z_bar]               (bits + scale; returned scale)
 *   delta_bar <- z_bar - m_bar
 * Worker i's bits are row i of wbits (stride bits_ld words, addressed by the
 * same global word index as the element); its scale for this segment is
 * wscale[i * scale_stride].                                               */
float orc_server_segment(int64_t b, int64_t e, int32_t n,
                         const uint64_t *wbits, int64_t bits_ld,
                         const float *wscale, int64_t scale_stride,
                         float *delta_bar, uint64_t *bits_out, float *z_scratch)
{
    for (int64_t idx = b; idx < e; ++idx) {
        double sum = 0.0;
        for (int32_t i = 0; i < n; ++i)
            sum += (double)orc_decode(wbits + (int64_t)i * bits_ld, idx,
                                      wscale[(int64_t)i * scale_stride]);
        float avg = (float)(sum / (double)n);
        z_scratch[idx] = avg + delta_bar[idx];
    }
    float scale = orc_compress(b, e, z_scratch, bits_out);
    for (int64_t idx = b; idx < e; ++idx) {
        float m_bar = orc_decode(bits_out, idx, scale);
        delta_bar[idx] = z_scratch[idx] - m_bar;
    }
    return scale;
}

/* Every worker: decode the broadcast m_bar, set m = m_bar, and take the
 * preconditioned step with the frozen variance:
 *   x <- x - lr * m_bar / sqrt(v_frozen + eps)
 * (eps under the root: the paper's Algorithm 1 shows no eps at all; this is
 * the placement the implementation fixes).  m may be NULL.                */
void orc_update_segment(int64_t b, int64_t e, const uint64_t *bits, float scale,
                        float lr, float eps, float *x, float *m,
                        const float *v_frozen)
{
    for (int64_t idx = b; idx < e; ++idx) {
        float m_bar = orc_decode(bits, idx, scale);
        float denom = sqrtf(v_frozen[idx] + eps);
        float ratio = m_bar / denom;
        float step = lr * ratio;
        x[idx] = x[idx] - step;
        if (m) m[idx] = m_bar;
    }
}

/* One whole compression-stage step over a layout of K tensors and n workers
 * (all n workers simulated in this process).  Buffers are flat over the
 * padded length D: g and delta have n rows (strides g_ld, delta_ld), wbits
 * has n rows of W = D/64 words, wscales has n rows of K*n scales; sbits has
 * W words and sscales K*n scales.  z_scratch holds D floats.              */
void orc_step(const int64_t *numel, int32_t K, int32_t n,
              const int64_t *seg_begin, const int64_t *seg_end,
              float *x, float *m, const float *v_frozen,
              const float *g, int64_t g_ld, float *delta, int64_t delta_ld,
              float *delta_bar, uint64_t *wbits, int64_t W, float *wscales,
              uint64_t *sbits, float *sscales,
              float lr, float beta1, float eps, float *z_scratch)
{
    (void)numel;
    const int64_t S = (int64_t)K * n;
    /* workers (each reads the shared momentum m of the previous step) */
    for (int32_t i = 0; i < n; ++i)
        for (int64_t q = 0; q < S; ++q)
            wscales[(int64_t)i * S + q] = orc_worker_segment(
                seg_begin[q], seg_end[q], beta1, m, g + (int64_t)i * g_ld,
                delta + (int64_t)i * delta_ld, wbits + (int64_t)i * W, z_scratch);
    /* servers: server j owns segments (k, j) of every tensor k */
    for (int64_t q = 0; q < S; ++q)
        sscales[q] = orc_server_segment(seg_begin[q], seg_end[q], n, wbits, W,
                                        wscales + q, S, delta_bar, sbits, z_scratch);
    /* every worker decodes the gathered result and updates x and m */
    for (int64_t q = 0; q < S; ++q)
        orc_update_segment(seg_begin[q], seg_end[q], sbits, sscales[q], lr, eps,
                           x, m, v_frozen);
}

/* The same step with the identity compressor (the paper's "1-bit Adam
 * (32-bits)" variant of Section 7.2: variance frozen, no compression).  With
 * C = identity every error stays zero and the step is momentum SGD on the
 * averaged gradient with the frozen preconditioner. Elements [b, e).       */
void orc_step_uncompressed_range(int64_t b, int64_t e, int32_t n,
                                 float *x, float *m, const float *v_frozen,
                                 const float *g, int64_t g_ld,
                                 float lr, float beta1, float eps)
{
    const float one_minus_beta1 = 1.0f - beta1;
    for (int64_t idx = b; idx < e; ++idx) {
        double sum = 0.0;
        for (int32_t i = 0; i < n; ++i) {
            float m_i = beta1 * m[idx];
            m_i = m_i + one_minus_beta1 * g[(int64_t)i * g_ld + idx];
            sum += (double)m_i;
        }
        float m_bar = (float)(sum / (double)n);
        float denom = sqrtf(v_frozen[idx] + eps);
        float ratio = m_bar / denom;
        float step = lr * ratio;
        x[idx] = x[idx] - step;
        m[idx] = m_bar;
    }
}
