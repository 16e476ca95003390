/*
 * zo_adam.h -- C ABI of the MI355X (gfx950) hot path of 0/1 Adam.
 *
 * 0/1 Adam (Lu, Li, Zhang, De Sa, He, arXiv 2202.06009), Algorithm 1, with the
 * error-feedback 1bit-AllReduce of Algorithm 2 and the 1-bit compressor of
 * Equation 3, for ONE worker's flat binary32 parameter shard of length d.
 * The other W-1 workers are represented only by their packed sign buffers and
 * scales, which the caller places in device memory (slots 1..W-1 of a W-slot
 * buffer); this worker writes its own into slot 0.
 *
 * Conventions shared by every entry point
 *   - Device pointers are caller-owned HIP device allocations.  Float vectors
 *     of shard length (state, avg_debug, and g and gbar when binary32) must
 *     be 16-byte aligned, binary16 / bfloat16 g and gbar 8-byte aligned,
 *     packed word buffers 8-byte aligned, scale buffers 4-byte aligned
 *     (ZO_EALIGN otherwise).  The library never frees or reallocates them.
 *   - The gradient inputs g and gbar have the element type grad_dtype of
 *     the configuration (binary32 by default; binary16 or bfloat16, as in
 *     the paper's FP16 training, are widened exactly to binary32 on load).
 *   - Every call validates all of its arguments on the host before enqueueing
 *     anything; a rejected call returns a negative status and changes nothing.
 *   - Calls are asynchronous on the stream given to zo_adam_init (or
 *     zo_set_stream): each hot-path call (zo_local_step, zo_compress_pack_ef,
 *     zo_unpack_average, zo_sync_update, zo_variance_update,
 *     zo_fullprec_step) returns after enqueueing one kernel; zo_read_state
 *     enqueues one and zo_materialize up to three elementwise kernels.
 *     Device faults surface at the caller's synchronisation.
 *   - No entry point after zo_adam_init allocates memory.
 *   - The hot-path calls may be recorded into a HIP graph (stream capture):
 *     each enqueues one kernel and no memset or copy.  A replay repeats the
 *     recorded arguments (step scalars, the implicit-state modes of deferred
 *     writes), so it stands for later steps only where those repeat, e.g. a
 *     steady local/sync alternation at a constant learning rate; the host's
 *     step counter does not advance on replays.
 *   - A handle is not thread-safe; use one handle per stream.
 *   - Arithmetic is IEEE binary32 with one rounding per operation, no FMA
 *     contraction, correctly rounded division and square root, no flushing of
 *     denormals; the per-chunk L1 norm is the balanced pairwise tree over the
 *     chunk in index order; the server's average over workers is the exact
 *     binary64 sum S divided by W in binary64 and rounded to binary32, which
 *     is RN32(S / W): for a binary64 S and an integer W the intermediate
 *     binary64 quotient never lands on a binary32 midpoint unless S / W does.
 *
 * Layout
 *   - The shard is a list of segments (one per parameter tensor); every
 *     segment is cut into chunks of at most `chunk` elements; Equation 3 is
 *     applied to each chunk on its own.
 *   - Packed signs: chunk c owns ceil(len_c / 64) uint64 words starting at
 *     word_c = sum of the word counts of the chunks before it; element j of
 *     the chunk is bit j % 64 of word j / 64 (LSB first); bit 1 means +1;
 *     sign(0) = +1 for +0 and -0; pad bits are written as 0 and ignored on
 *     input.  One binary32 scale per chunk.
 *   - A W-slot packed buffer is uint64[W][wstride], scales float[W][cstride],
 *     where wstride / cstride are the word / chunk counts of the server range
 *     (all words / all chunks for the single server).
 */
#ifndef ZO_ADAM_H
#define ZO_ADAM_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes. */
enum {
    ZO_OK = 0,
    ZO_EINVAL = -1,   /* bad argument: null pointer, size, hyper-parameter, step */
    ZO_EALIGN = -2,   /* pointer not 16-byte aligned / segment offset not a multiple of 4 */
    ZO_ESTATE = -3,   /* call out of order for the current step */
    ZO_EHIP = -4,     /* HIP runtime error (text via zo_last_hip_error) */
    ZO_ENOMEM = -5,   /* host or device allocation failed in zo_adam_init */
    ZO_ESCRATCH = -6  /* zo_adam_init_static: the configuration exceeds its static scratch */
};

/* Element types of the gradient inputs (zo_config.grad_dtype). */
enum { ZO_DTYPE_F32 = 0, ZO_DTYPE_F16 = 1, ZO_DTYPE_BF16 = 2 };

/* Algorithms (zo_config.algorithm). */
enum {
    ZO_ALG_ZERO_ONE_ADAM = 0,     /* Algorithm 1 with Algorithm 2 (0/1 Adam) */
    ZO_ALG_FROZEN_VARIANCE = 1    /* Algorithm 4 with Algorithm 2: 1-bit compressed
                                     gradients, variance updated only in T_v, no local
                                     steps; 1-bit Adam is T_v = {0, ..., T0 - 1} */
};

typedef struct zo_adam zo_adam;   /* opaque handle */

/*
 * Configuration (host memory, read during zo_adam_init only).
 *   beta1, beta2   Adam decay factors, each in [0, 1) (Algorithm 1 inputs).
 *   eps            numerical constant added inside the square root, >= 0.
 *   world          number of workers n = W >= 1 (the average of Algorithm 2).
 *   chunk          compression chunk length C in [1, 16384].  Chunks then
 *                  start at segment offsets plus multiples of C; when C is not a
 *                  multiple of 4 the chunk kernels access elements one by one
 *                  (slower) and the server uses its plain form.
 *   n              shard length d >= 0.
 *   nseg, seg_off  nseg >= 1 segments; seg_off[0] = 0, seg_off[nseg] = n,
 *                  non-decreasing, every offset a multiple of 4.
 *   ntv, tv        the variance-update step set T_v: strictly increasing
 *                  0-based step indices (ntv may be 0).
 *   ntu, tu        the synchronisation step set T_u, likewise.
 *   srv_chunk_begin, srv_chunk_end
 *                  chunk range [begin, end) that this GPU serves in the
 *                  server half of Algorithm 2; end < 0 means "to the last
 *                  chunk" (begin = 0, end = -1 is the single server).
 *   defer_sync_writes
 *                  0: zo_sync_update writes m, x, anchor and u = 0 (x, m and
 *                  u are always current in their buffers).  Nonzero: it
 *                  writes only the anchor (12 bytes per parameter less) and a
 *                  copy of the server's packed words and scales into the
 *                  library's own memory (allocated by zo_adam_init): the new
 *                  model is held in `anchor`, u is +0 by definition and m is
 *                  the server's average over Gamma, which the next call
 *                  rebuilds from the 1-bit copy (reading 1/8 byte per
 *                  parameter instead of 4).
 *                  The next zo_local_step reads the model from the anchor and
 *                  writes x and m, and neither reads nor writes u (8 bytes less):
 *                  u is then +0 + gamma_t m_{t+1} in binary32, the one
 *                  product it added, so the next call that needs u (a local
 *                  step, which writes it, or a fused compress) forms it from
 *                  the m it reads anyway (4 bytes less).  A local step at a
 *                  sync step (the unfused path) always writes u.
 *                  zo_read_state gives the current x, m or u; zo_materialize
 *                  writes them out.  The arithmetic, and so every value, is
 *                  the same in both modes.
 *   algorithm      ZO_ALG_ZERO_ONE_ADAM (default 0) or ZO_ALG_FROZEN_VARIANCE.
 *                  The latter requires ntu = 0 and defer_sync_writes = 0; its
 *                  steps are zo_fullprec_step at t in T_v and, at every other
 *                  t, zo_compress_pack_ef (with the gradient), zo_unpack_average
 *                  and zo_sync_update (gbar = NULL).  st.u and st.anchor are
 *                  unused and may be NULL.
 *   grad_dtype     ZO_DTYPE_F32 (default 0), ZO_DTYPE_F16 or ZO_DTYPE_BF16:
 *                  the element type of every g and gbar argument.  All
 *                  arithmetic stays binary32 (16-bit values widen exactly).
 */
typedef struct zo_config {
    float beta1, beta2, eps;
    int32_t world;
    int32_t chunk;
    int64_t n;
    int32_t nseg;
    const int64_t *seg_off;
    int32_t ntv;
    const int64_t *tv;
    int32_t ntu;
    const int64_t *tu;
    int64_t srv_chunk_begin, srv_chunk_end;
    int32_t defer_sync_writes;
    int32_t algorithm;
    int32_t grad_dtype;
} zo_config;

/*
 * Optimizer state (device memory, caller-owned, binary32).
 *   x        model, float[n]; holds x_0 at init.
 *   m, v, u  momentum, variance, local-step buffer, float[n].
 *   err      worker compression error delta (Algorithm 2), float[n].
 *   srv_err  server compression error (Algorithm 2), float[elements of the
 *            server range].
 *   anchor   model at the most recent synchronisation x_{t'}, float[n].
 */
typedef struct zo_state {
    float *x, *m, *v, *u, *err, *srv_err, *anchor;
} zo_state;

/*
 * zo_adam_init -- set up the handle (Algorithm 1, its "Require" line).
 * Validates the configuration, builds the chunk table and copies it to the
 * device, and allocates one flag byte per server chunk and, with
 * defer_sync_writes, the copy of the server's packed words and scales (the
 * only device allocations the library makes), then enqueues on `stream`:
 * m = v = u = err = srv_err = 0 and anchor = x.  Gamma = 0, next step t = 0.
 * Returns ZO_OK and *h, or an error (then *h is NULL).
 */
int zo_adam_init(zo_adam **h, const zo_config *cfg, const zo_state *st, hipStream_t stream);

/*
 * zo_adam_init_static -- zo_adam_init for callers that cannot allocate
 * (code recorded under HIP graph capture, tight serving loops, harnesses that
 * forbid allocation): the same handle, arguments, validation, initial state
 * and results, but no device or host memory is allocated.  The chunk table,
 * the exactness flags and, with defer_sync_writes, the copy of the server's
 * output live in the library's static device array of 4 MiB (each GPU the
 * library runs on holds one until the process ends), the handle and its
 * schedules in a static host slot of the current device.
 * Limits: one live handle from zo_adam_init_static per device at a time
 * (ZO_ESTATE while one exists; zo_adam_destroy frees the slot; a later one
 * reuses the array and starts from a cleared state); 20 bytes per chunk plus
 * one per server chunk, plus 8 per packed word and 4 per chunk with
 * defer_sync_writes, must fit the 4 MiB (about 190,000 chunks without
 * deferred writes), and T_v and T_u at most 65536 steps each, else
 * ZO_ESCRATCH.  Calls on such a handle from several host threads race, as on
 * any handle.  zo_chunk_table reads the table back from the device.
 */
int zo_adam_init_static(zo_adam **h, const zo_config *cfg, const zo_state *st,
                        hipStream_t stream);

/* Release the handle and its device memory.  Waits for the stream. */
int zo_adam_destroy(zo_adam *h);

/* Change the stream later calls enqueue on.  Work already enqueued on the
 * previous stream is not waited for: the caller orders the two streams (an
 * event recorded on the old one and waited on by the new one) before the next
 * call, since every call reads what the previous one wrote.  zo_adam_destroy
 * waits only for the current stream. */
int zo_set_stream(zo_adam *h, hipStream_t stream);

/*
 * zo_local_step -- the momentum, model and buffer lines of Algorithm 1 for
 * step t (must be the handle's next step), elementwise over the shard:
 *   m' = beta1 m + (1 - beta1) g;  p = gamma m';
 *   x <- x - p / sqrt(v + eps);  u <- u + p;  m <- m';  Gamma <- Gamma + gamma.
 * The momentum used in the model and buffer lines is the fresh m' (the literal
 * subscript t would freeze the momentum when every step synchronises).
 *   gamma   learning rate gamma_t > 0, finite.
 *   g       device [n] of grad_dtype, this worker's stochastic gradient g_t.
 *   gbar    NULL, or device [n] of grad_dtype with the full-precision average gradient
 *           of step t when t is in T_v and t is not in T_u: the variance line
 *           v <- beta2 v + (1 - beta2) gbar^2 is then fused (v_t is used above
 *           before it is overwritten).  Passing gbar when t is not in T_v, or
 *           when t is in T_u, is ZO_EINVAL.
 * At t not in T_u this completes step t (unless the variance update is still
 * due).  At t in T_u it is the unfused first half of a sync step:
 * zo_compress_pack_ef with g = NULL must follow.
 */
int zo_local_step(zo_adam *h, int64_t t, float gamma, const void *g, const void *gbar);

/*
 * zo_compress_pack_ef -- worker half of Algorithm 2 applied to the buffer
 * u_{t+1/2} at a sync step t in T_u (the 1bit-AllReduce line of Algorithm 1),
 * with Equation 3 per chunk:
 *   a = u_{t+1/2} + err;  s_c = |a|_1 / len_c (pairwise tree);
 *   bit_j = (a_j >= 0);  err_j <- a_j - s_c (bit 1) or a_j + s_c (bit 0).
 * With g != NULL the momentum/buffer lines are fused: u_{t+1/2} = u + gamma m'
 * with m' = beta1 m + (1 - beta1) g, and Gamma += gamma; x, m and u are not
 * written (the reconstruction supersedes them).  With g == NULL the call must
 * follow zo_local_step(t) and u already holds u_{t+1/2} (gamma is ignored).
 * ZO_ALG_FROZEN_VARIANCE, t not in T_v: a = g + err (the compressed
 * AllReduce of the gradient in Algorithm 4); g is required and gamma = gamma_t
 * is kept for zo_sync_update.
 *   packed0  device uint64[words]: this worker's packed signs (slot 0).
 *   scales0  device float[nchunks]: this worker's scales (slot 0).
 */
int zo_compress_pack_ef(zo_adam *h, int64_t t, float gamma, const void *g,
                        uint64_t *packed0, float *scales0);

/*
 * zo_unpack_average -- server half of Algorithm 2 over the server chunk
 * range, at sync step t, after zo_compress_pack_ef(t).  For each element:
 *   avg = RN32( (sum_w (bit_w ? +S_w : -S_w)) / W )  (sum exact),
 *   b = avg + srv_err;  per chunk s = |b|_1 / len_c;  sigma = (b >= 0);
 *   srv_err <- b - s sigma.
 * The line's "t+1" subscript on the averaged buffers is read as "t" (the
 * error update on the same line uses t).
 *   packed      device uint64[W][wstride]: slot w = worker w, slot 0 = own.
 *   scales      device float[W][cstride], likewise.
 *   srv_packed  device uint64[words] indexed by global word; only the server
 *               range's words are written.
 *   srv_scales  device float[nchunks] indexed by global chunk (range only).
 *   avg_debug   NULL, or device float[range elements] receiving avg.
 * The exact sum needs the nonzero scales of a chunk to span at most
 * 29 - ceil(log2 W) binary exponents; chunks that violate it are counted
 * (zo_inexact_chunks) and still produce the binary64 result.
 */
int zo_unpack_average(zo_adam *h, int64_t t, const uint64_t *packed, const float *scales,
                      uint64_t *srv_packed, float *srv_scales, float *avg_debug);

/*
 * zo_sync_update -- the sync lines of Algorithm 1 at step t, after
 * zo_unpack_average(t) (on a multi-GPU run, after the server outputs of all
 * ranges have been gathered into srv_packed / srv_scales):
 *   ubar = sigma s (the server's compressed average);
 *   m <- ubar / Gamma;  x <- anchor - ubar / sqrt(v_t + eps);
 *   anchor <- x;  u <- 0;  Gamma <- 0  (the next interval starts at t + 1).
 *   srv_packed  device uint64[words], srv_scales device float[nchunks].
 *   gbar        as in zo_local_step: fused variance line when t is in T_v.
 * With defer_sync_writes, x and u are not written (see zo_config).
 * ZO_ALG_FROZEN_VARIANCE: gbar_t = sigma s is the step's gradient in
 * Algorithm 4's momentum and model lines, v is kept (t is not in T_v):
 *   m <- beta1 m + (1 - beta1) gbar_t;  x <- x - gamma_t m_t / sqrt(v_t + eps)
 * with the momentum m_t and variance v_t from before the step, as the listing
 * writes them; gbar must be NULL.
 */
int zo_sync_update(zo_adam *h, int64_t t, const uint64_t *srv_packed, const float *srv_scales,
                   const void *gbar);

/*
 * zo_fullprec_step -- ZO_ALG_FROZEN_VARIANCE, t in T_v: one step of
 * Algorithm 4 with the full-precision AllReduce output gbar (device [n] of
 * grad_dtype):
 *   v <- beta2 v + (1 - beta2) gbar^2;  m <- beta1 m + (1 - beta1) gbar;
 *   x <- x - gamma m_t / sqrt(v_t + eps)   (m_t, v_t from before the step).
 * ZO_EINVAL on a ZO_ALG_ZERO_ONE_ADAM handle; ZO_ESTATE if t is not the next
 * step or not in T_v.
 */
int zo_fullprec_step(zo_adam *h, int64_t t, float gamma, const void *gbar);

/*
 * zo_variance_update -- the variance line of Algorithm 1 for t in T_v when it
 * was not fused: v <- beta2 v + (1 - beta2) gbar^2, after the other calls of
 * step t.  gbar: device [n] of grad_dtype, the full-precision AllReduce
 * output.
 */
int zo_variance_update(zo_adam *h, int64_t t, const void *gbar);

/*
 * zo_materialize -- with defer_sync_writes, write out what is implicit:
 * x <- anchor, u <- +0 or +0 + gamma m, and m from the server copy (a few
 * elementwise kernels on the handle's stream, only for what is pending).  Between steps
 * only (ZO_ESTATE otherwise); changes no value of the optimizer state.  The
 * next steps run as after an eager zo_sync_update.
 */
int zo_materialize(zo_adam *h);

/* State vectors for zo_read_state. */
enum { ZO_STATE_X = 0, ZO_STATE_M = 1, ZO_STATE_U = 2 };

/*
 * zo_read_state -- the current value of x, m or u (which = ZO_STATE_*) into
 * out (device float[n], 16-byte aligned, async on the handle's stream),
 * wherever deferred sync writes keep it.  Between steps only (ZO_ESTATE
 * otherwise); changes nothing.  ZO_STATE_U is ZO_EINVAL under
 * ZO_ALG_FROZEN_VARIANCE (no buffer).
 */
int zo_read_state(zo_adam *h, int32_t which, float *out);

/* ---- queries (host only; never touch the device unless stated) ---------- */
/* Where the current state is: *x_now = the device buffer that holds x
 * (st.x, or st.anchor after a deferred zo_sync_update); *u_mode = 0 when
 * st.u holds u, 1 when u is +0 everywhere, 2 when u = +0 + (*u_gamma) * m
 * elementwise in binary32 (st.u stale in modes 1 and 2; *u_gamma is 0 in modes
 * 0 and 1).  Any pointer may be NULL. */
int zo_state_location(const zo_adam *h, float **x_now, int32_t *u_mode, float *u_gamma);
int64_t zo_num_chunks(const zo_adam *h);
int64_t zo_packed_words(const zo_adam *h);
/* Server range: first chunk, chunk count, first word, word count, first
 * element, element count (any pointer may be NULL). */
int zo_server_range(const zo_adam *h, int64_t *chunk0, int64_t *nchunks, int64_t *word0,
                    int64_t *nwords, int64_t *elem0, int64_t *nelems);
/* Copy the chunk table to host arrays of nchunks entries (any may be NULL). */
int zo_chunk_table(const zo_adam *h, int64_t *start, int64_t *len, int64_t *word);
float zo_gamma_sum(const zo_adam *h);
int64_t zo_next_step(const zo_adam *h);
/* Number of server-range chunks whose scales broke the exact-sum condition
 * in at least one zo_unpack_average since zo_adam_init (a chunk's flag is
 * never cleared; synchronises the stream). */
int zo_inexact_chunks(zo_adam *h, int64_t *count);
const char *zo_strerror(int status);
const char *zo_last_hip_error(const zo_adam *h);

/* ---- diagnostics --------------------------------------------------------- */
/* Elementwise q = a / b and r = sqrt(a) on the device, with the same binary32
 * division and square root the kernels use (device float[n] each; async on
 * `stream`).  Lets a test compare them with the host's IEEE operations. */
int zo_diag_divsqrt(const float *a, const float *b, float *q, float *r, int64_t n,
                    hipStream_t stream);

/* Copy float[n] (n a multiple of 4, 16-byte aligned) with the loads and
 * stores of the streaming kernels: nontemporal != 0 selects nontemporal
 * accesses.  A reference kernel of known size for HBM byte counters. */
int zo_diag_copy(const float *src, float *dst, int64_t n, int nontemporal, hipStream_t stream);

/* dst[w][i] = (sum over r of src[r][i]) + w for i < n: nsrc in [1, 6] read
 * streams and ndst in [1, 5] write streams of float[n] (n a multiple of 4,
 * 16-byte aligned device buffers; src and dst are host arrays of device
 * pointers), one float4 per thread with nontemporal accesses like the
 * streaming kernels.  A dst may be one of the srcs (the array is then read
 * and rewritten in place: each thread stores after all of its loads, and the
 * sum uses the old values); two dsts may not be the same buffer (ZO_EINVAL),
 * and buffers may not otherwise overlap.  Timing it measures the HBM rate
 * reachable by a kernel with the same mix of arrays. */
int zo_diag_stream(const float *const *src, int32_t nsrc, float *const *dst, int32_t ndst,
                   int64_t n, hipStream_t stream);

/* The memory accesses of zo_unpack_average's kernel without its arithmetic,
 * on h's server range: per chunk one workgroup in the server's shape and
 * order, each lane reading its packed dword of the chunk from all `world`
 * rows of `packed` (laid out as for zo_unpack_average), then the chunk's
 * server error (the srv_err buffer of h's state) loaded and stored back
 * unchanged with the server's nontemporal accesses: the error keeps its
 * bits.  Timing it measures the HBM rate the server's access pattern can
 * reach.  Enqueued on h's stream; no state-machine effect (any phase).
 * Chunks of at most 1024 elements (several chunks per workgroup) are not
 * covered: ZO_EINVAL. */
int zo_diag_server_pattern(zo_adam *h, const uint64_t *packed);

/* ---- planning helpers (pure host; usable without a GPU) ----------------- */
/* Validate a configuration exactly as zo_adam_init does. */
int zo_config_check(const zo_config *cfg);
/* Chunk count of a segment table, or a negative status. */
int64_t zo_plan_num_chunks(int32_t nseg, const int64_t *seg_off, int32_t chunk);
/* Fill a chunk table (arrays of zo_plan_num_chunks entries); returns the
 * total packed word count or a negative status. */
int64_t zo_plan_chunks(int32_t nseg, const int64_t *seg_off, int32_t chunk, int64_t *start,
                       int64_t *len, int64_t *word);

#ifdef __cplusplus
}
#endif

#endif /* ZO_ADAM_H */
