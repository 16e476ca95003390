/*
 * zo_oracle.c -- plain, slow, single-threaded CPU oracle of 0/1 Adam.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file; only the tests, the smoke check and the CPU-baseline leg of
 * the benchmark use it.  It shares no source with the HIP library.
 *
 * What it computes (Lu, Li, Zhang, De Sa, He, "Maximizing Communication
 * Efficiency for Large-scale Training via 0/1 Adam", arXiv 2202.06009):
 *   - Algorithm 4 (the frozen-variance framework with compressed gradients,
 *     of which 1-bit Adam is the case T_v = a prefix of the steps), one step
 *     given the averaged gradient, see zr_fv_step;
 *   - Algorithm 1 (0/1 Adam) for one worker, step by step, in the paper's
 *     order: momentum, model, buffer; then the sync block (1bit-AllReduce of
 *     the buffer, momentum approximation, model from the anchor, reset); then
 *     the variance block (update or keep the stale variance).
 *   - Algorithm 2 (error-feedback 1bit-AllReduce) as the 1bit-AllReduce of
 *     Algorithm 1: the worker half (compress z + delta, keep the new error)
 *     and the server half (average the W compressed buffers, add the server
 *     error, compress again, keep the new server error).
 *   - Equation 3 (the 1-bit compressor C[a] = (|a|_1 / n) sign(a)), applied
 *     independently to every chunk of the flat shard.
 *
 * Precision.  The decisions the method takes (a sign bit per coordinate)
 * depend on floating-point values, so this oracle computes in the precision
 * of the GPU kernels, IEEE binary32, with every rounding pinned:
 *   - no FMA contraction (built with -ffp-contract=off), IEEE sqrtf and '/';
 *   - constants c1 = 1 - beta1 and c2 = 1 - beta2 are formed in binary32;
 *   - the per-chunk L1 norm is a balanced pairwise tree in index order,
 *     zero-padded to the next power of two;
 *   - the server's sum over workers is carried out in binary64 and checked to
 *     be exact (TwoSum residual zero at every addition), then divided by W in
 *     binary64 and rounded once to binary32.
 * Everything else is the literal expression of the algorithm, one rounding
 * per operation, evaluated left to right as written below.
 *
 * Readings taken where the paper is silent or ambiguous (each is restated at
 * the place it is used):
 *   - momentum index: the model and buffer lines use the freshly updated
 *     momentum m_{t+1/2} (the literal m_t is kept behind a flag; with
 *     synchronisation at every step it freezes m at zero);
 *   - after a sync at step t the next interval starts at t+1: the anchor is
 *     the model produced by that sync and the learning-rate sum Gamma covers
 *     exactly the steps whose updates are in the buffer u;
 *   - the server line of Algorithm 2 averages the compressed buffers of the
 *     current step (its "t+1" subscript is read as "t");
 *   - sign(0) = +1, for +0 and -0 alike;
 *   - sign bits are packed LSB-first into 64-bit words; every chunk starts a
 *     new word; pad bits are zero.
 *
 * Parity pins: every function here is pinned by the not-GPU tests against
 * closed forms, invariants, brute force or an independent fp64 Adam; none is
 * "parity unpinned".
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#if defined(__FAST_MATH__) || defined(__FP_FAST_FMAF)
#error "the oracle must be built without fast-math and without FMA contraction"
#endif

#define ZR_OK 0
#define ZR_EINVAL -1
#define ZR_EINEXACT -6

/* ------------------------------------------------------------------------ */
/* Layout: segments split into chunks, chunks own whole 64-bit words.        */
/* ------------------------------------------------------------------------ */

/* Number of chunks produced by cutting every segment into pieces of at most
 * `chunk` elements (the compressor of Equation 3 is applied per chunk). */
int64_t zr_count_chunks(int32_t nseg, const int64_t *seg_off, int32_t chunk)
{
    int64_t total = 0;
    for (int32_t s = 0; s < nseg; ++s) {
        int64_t len = seg_off[s + 1] - seg_off[s];
        total += (len + chunk - 1) / chunk;
    }
    return total;
}

/* Fill the chunk table: start index, length and first packed word of every
 * chunk.  Returns the total number of 64-bit words. */
int64_t zr_build_chunks(int32_t nseg, const int64_t *seg_off, int32_t chunk,
                        int64_t *cstart, int64_t *clen, int64_t *cword)
{
    int64_t c = 0, word = 0;
    for (int32_t s = 0; s < nseg; ++s) {
        for (int64_t pos = seg_off[s]; pos < seg_off[s + 1]; pos += chunk) {
            int64_t len = seg_off[s + 1] - pos;
            if (len > chunk) len = chunk;
            cstart[c] = pos;
            clen[c] = len;
            cword[c] = word;
            word += (len + 63) / 64;
            ++c;
        }
    }
    return word;
}

/* ------------------------------------------------------------------------ */
/* Equation 3 on one chunk.                                                  */
/* ------------------------------------------------------------------------ */

/* Pairwise sum of |a[0..n)| over a virtual array of length `span` (a power of
 * two, span >= n) whose tail beyond n holds zeros: T(lo half) + T(hi half). */
static float tree_abs(const float *a, int64_t n, int64_t span)
{
    if (n <= 0) return 0.0f;
    if (span == 1) return fabsf(a[0]);
    int64_t half = span / 2;
    int64_t nlo = n < half ? n : half;
    float lo = tree_abs(a, nlo, half);
    float hi = tree_abs(a + half, n - nlo, half);
    return lo + hi;
}

static int64_t next_pow2(int64_t n)
{
    int64_t p = 1;
    while (p < n) p *= 2;
    return p;
}

/* The L1 norm of a chunk as the balanced pairwise tree in index order. */
float zr_tree_abs_sum(const float *a, int64_t n)
{
    return tree_abs(a, n, next_pow2(n));
}

/* C[a] of Equation 3 for one chunk of length n: the shared magnitude
 * s = |a|_1 / n, and sign(a) with sign(0) = +1 (bit 1 means +1). */
float zr_compress_chunk(const float *a, int64_t n, uint8_t *bit)
{
    float l1 = zr_tree_abs_sum(a, n);
    float s = l1 / (float)n;
    for (int64_t j = 0; j < n; ++j) bit[j] = (a[j] >= 0.0f) ? 1 : 0;
    return s;
}

/* ------------------------------------------------------------------------ */
/* Packing: element j of a chunk -> word j/64, bit j%64 (LSB first).         */
/* ------------------------------------------------------------------------ */

void zr_pack_chunk(const uint8_t *bit, int64_t n, uint64_t *words)
{
    int64_t nw = (n + 63) / 64;
    for (int64_t w = 0; w < nw; ++w) words[w] = 0;
    for (int64_t j = 0; j < n; ++j)
        if (bit[j]) words[j / 64] |= (uint64_t)1 << (j % 64);
}

void zr_unpack_chunk(const uint64_t *words, int64_t n, uint8_t *bit)
{
    for (int64_t j = 0; j < n; ++j) bit[j] = (uint8_t)((words[j / 64] >> (j % 64)) & 1u);
}

/* ------------------------------------------------------------------------ */
/* Algorithm 2, worker half: compress z + delta, keep the new error.         */
/* ------------------------------------------------------------------------ */

/* For every chunk: a = z + delta; (s, sign) = C[a]; delta <- a - s*sign.
 * Writes the packed signs (nwords words) and one scale per chunk. */
int zr_ef_compress(int64_t nchunks, const int64_t *cstart, const int64_t *clen,
                   const int64_t *cword, const float *z, float *delta,
                   uint64_t *words, float *scales)
{
    for (int64_t c = 0; c < nchunks; ++c) {
        int64_t n = clen[c], base = cstart[c];
        float *a = (float *)malloc((size_t)n * sizeof(float));
        uint8_t *bit = (uint8_t *)malloc((size_t)n);
        if (!a || !bit) { free(a); free(bit); return ZR_EINVAL; }
        for (int64_t j = 0; j < n; ++j) a[j] = z[base + j] + delta[base + j];
        float s = zr_compress_chunk(a, n, bit);
        for (int64_t j = 0; j < n; ++j)
            delta[base + j] = bit[j] ? (a[j] - s) : (a[j] + s);
        zr_pack_chunk(bit, n, words + cword[c]);
        scales[c] = s;
        free(a);
        free(bit);
    }
    return ZR_OK;
}

/* ------------------------------------------------------------------------ */
/* Algorithm 2, server half.                                                 */
/* ------------------------------------------------------------------------ */

/* Exact sum check: Knuth's TwoSum error term of a + b. */
static double two_sum_err(double a, double b, double s)
{
    double bb = s - a;
    return (a - (s - bb)) + (b - bb);
}

/* The average over W workers of their decompressed buffers, for the element
 * at position j of chunk c:  (1/W) * sum_w (+-S_w[c]).  The sum is exact in
 * binary64 (checked), the division is binary64, the result rounded once to
 * binary32.  Returns ZR_EINEXACT if an addition was not exact. */
static int server_average(int32_t W, int64_t nwords_stride, int64_t nchunks_stride,
                          const uint64_t *words, const float *scales,
                          int64_t c, int64_t word_of_elem, int bitpos, float *out)
{
    double sum = 0.0;
    for (int32_t w = 0; w < W; ++w) {
        uint64_t word = words[(int64_t)w * nwords_stride + word_of_elem];
        double sw = (double)scales[(int64_t)w * nchunks_stride + c];
        double term = ((word >> bitpos) & 1u) ? sw : -sw;
        double s = sum + term;
        if (two_sum_err(sum, term, s) != 0.0) return ZR_EINEXACT;
        sum = s;
    }
    *out = (float)(sum / (double)W);
    return ZR_OK;
}

/* Server half of Algorithm 2 over the chunks [c0, c1): for each element,
 * b = avg_w(C[z_w + delta_w]) + server_delta; (s, sign) = C[b] per chunk;
 * server_delta <- b - s*sign.  `words` is [W][nwords_stride], slot w holding
 * worker w's packed signs indexed by global word minus cword[c0]; `scales` is
 * [W][nchunks_stride] indexed by chunk minus c0.  `srv_delta` covers the
 * elements of the range, indexed by element minus cstart[c0].  The server
 * output words/scales are indexed by global word and global chunk.  `avg`
 * (optional) receives the binary32 averages, indexed like srv_delta. */
int zr_server(int32_t W, int64_t c0, int64_t c1, const int64_t *cstart,
              const int64_t *clen, const int64_t *cword,
              const uint64_t *words, int64_t nwords_stride,
              const float *scales, int64_t nchunks_stride,
              float *srv_delta, uint64_t *srv_words, float *srv_scales, float *avg)
{
    int64_t ebase = cstart[c0], wbase = cword[c0];
    for (int64_t c = c0; c < c1; ++c) {
        int64_t n = clen[c];
        float *b = (float *)malloc((size_t)n * sizeof(float));
        uint8_t *bit = (uint8_t *)malloc((size_t)n);
        if (!b || !bit) { free(b); free(bit); return ZR_EINVAL; }
        for (int64_t j = 0; j < n; ++j) {
            float a;
            int rc = server_average(W, nwords_stride, nchunks_stride, words, scales,
                                    c - c0, cword[c] - wbase + j / 64, (int)(j % 64), &a);
            if (rc != ZR_OK) { free(b); free(bit); return rc; }
            int64_t e = cstart[c] + j - ebase;
            if (avg) avg[e] = a;
            b[j] = a + srv_delta[e];
        }
        float s = zr_compress_chunk(b, n, bit);
        for (int64_t j = 0; j < n; ++j) {
            int64_t e = cstart[c] + j - ebase;
            srv_delta[e] = bit[j] ? (b[j] - s) : (b[j] + s);
        }
        zr_pack_chunk(bit, n, srv_words + cword[c]);
        srv_scales[c] = s;
        free(b);
        free(bit);
    }
    return ZR_OK;
}

/* Decompress a packed buffer: out_j = sign_j * S[c] (exact). */
void zr_decompress(int64_t nchunks, const int64_t *cstart, const int64_t *clen,
                   const int64_t *cword, const uint64_t *words, const float *scales,
                   float *out)
{
    for (int64_t c = 0; c < nchunks; ++c)
        for (int64_t j = 0; j < clen[c]; ++j) {
            int bit = (int)((words[cword[c] + j / 64] >> (j % 64)) & 1u);
            out[cstart[c] + j] = bit ? scales[c] : -scales[c];
        }
}

/* Uncompressed average of W dense buffers (the "compression off" switch):
 * binary64 sum in worker order, checked exact, divided by W, rounded once. */
int zr_dense_average(int32_t W, int64_t n, const float *z, float *out)
{
    for (int64_t j = 0; j < n; ++j) {
        double sum = 0.0;
        for (int32_t w = 0; w < W; ++w) {
            double term = (double)z[(int64_t)w * n + j];
            double s = sum + term;
            if (two_sum_err(sum, term, s) != 0.0) return ZR_EINEXACT;
            sum = s;
        }
        out[j] = (float)(sum / (double)W);
    }
    return ZR_OK;
}

/* ------------------------------------------------------------------------ */
/* Algorithm 1 for one worker.                                               */
/* ------------------------------------------------------------------------ */

typedef struct {
    float beta1, beta2, eps;
    float c1, c2;              /* 1 - beta1, 1 - beta2, formed in binary32 */
    int32_t literal_momentum;  /* 1: model/buffer lines use the old m_t */
} zr_params;

typedef struct {
    float *x, *m, *v, *u, *anchor;
    float gamma_sum;           /* Gamma: sum of the learning rates folded into u */
} zr_state;

void zr_params_init(zr_params *p, float beta1, float beta2, float eps, int32_t literal)
{
    p->beta1 = beta1;
    p->beta2 = beta2;
    p->eps = eps;
    p->c1 = 1.0f - beta1;
    p->c2 = 1.0f - beta2;
    p->literal_momentum = literal;
}

/* Momentum, model and buffer lines of Algorithm 1 (every step):
 *   m_{t+1/2} = beta1 m_t + (1 - beta1) g_t
 *   x_{t+1/2} = x_t - gamma_t m / sqrt(v_t + eps)
 *   u_{t+1/2} = u_t + gamma_t m
 * with m = m_{t+1/2} (or m_t under the literal reading).  Gamma += gamma_t.
 * The x written here is superseded by the reconstruction at a sync step. */
void zr_half_step(const zr_params *p, zr_state *st, int64_t n, float gamma, const float *g)
{
    st->gamma_sum = st->gamma_sum + gamma;
    for (int64_t j = 0; j < n; ++j) {
        float m_old = st->m[j];
        float m_new = p->beta1 * m_old + p->c1 * g[j];
        float m_used = p->literal_momentum ? m_old : m_new;
        float step = gamma * m_used;
        float den = sqrtf(st->v[j] + p->eps);
        st->x[j] = st->x[j] - step / den;
        st->u[j] = st->u[j] + step;
        st->m[j] = m_new;
    }
}

/* Sync lines of Algorithm 1 given the averaged buffer ubar:
 *   m_{t+1} = ubar / Gamma
 *   x_{t+1} = x_{t'} - ubar / sqrt(v_t + eps)
 *   u_{t+1} = 0,  t' = t  (the anchor becomes x_{t+1}, Gamma restarts). */
void zr_sync_dense(const zr_params *p, zr_state *st, int64_t n, const float *ubar)
{
    float gsum = st->gamma_sum;
    for (int64_t j = 0; j < n; ++j) {
        float den = sqrtf(st->v[j] + p->eps);
        st->m[j] = ubar[j] / gsum;
        st->x[j] = st->anchor[j] - ubar[j] / den;
        st->anchor[j] = st->x[j];
        st->u[j] = 0.0f;
    }
    st->gamma_sum = 0.0f;
}

/* Variance lines of Algorithm 1 at t in T_v:
 *   v_{t+1} = beta2 v_t + (1 - beta2) gbar_t^2. */
void zr_variance(const zr_params *p, zr_state *st, int64_t n, const float *gbar)
{
    for (int64_t j = 0; j < n; ++j)
        st->v[j] = p->beta2 * st->v[j] + p->c2 * (gbar[j] * gbar[j]);
}

/* ------------------------------------------------------------------------ */
/* Algorithm 4: 1-bit communication with a frozen variance (no local steps). */
/* ------------------------------------------------------------------------ */

/* One step of Algorithm 4 given the averaged gradient gbar: the
 * full-precision average at t in T_v (update_v = 1), else the compressed
 * average of Algorithm 2 applied to the gradients (update_v = 0).  The
 * listing's lines in its order:
 *   v_{t+1} = beta2 v_t + (1 - beta2) gbar^2   (t in T_v;  else v_{t+1} = v_t)
 *   m_{t+1} = beta1 m_t + (1 - beta1) gbar
 *   x_{t+1} = x_t - gamma_t m_t / sqrt(v_t + eps)
 * The model line uses m_t and v_t as printed, as Equation 2 does: nothing
 * here degenerates, so the listing is taken literally. */
void zr_fv_step(const zr_params *p, float *x, float *m, float *v, int64_t n, float gamma,
                const float *gbar, int32_t update_v)
{
    for (int64_t j = 0; j < n; ++j) {
        float v_old = v[j], m_old = m[j];
        if (update_v) v[j] = p->beta2 * v_old + p->c2 * (gbar[j] * gbar[j]);
        m[j] = p->beta1 * m_old + p->c1 * gbar[j];
        float step = gamma * m_old;
        float den = sqrtf(v_old + p->eps);
        x[j] = x[j] - step / den;
    }
}

