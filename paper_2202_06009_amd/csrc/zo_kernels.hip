// zo_kernels.hip -- gfx950 kernels of the 0/1 Adam hot path.
//
// Paper: Lu et al., "Maximizing Communication Efficiency for Large-scale
// Training via 0/1 Adam" (arXiv 2202.06009): Algorithm 1 (0/1 Adam),
// Algorithm 2 (error-feedback 1bit-AllReduce), Equation 3 (1-bit compressor).
//
// Every kernel streams HBM: nothing is a contraction, so nothing uses MFMA.
// Arithmetic is binary32 with one rounding per operation (the library is
// built with -ffp-contract=off; division and sqrtf are the correctly rounded
// lowerings), so any implementation that follows the same operation order
// reproduces the results bit for bit.
//
// Memory access
//   * every state vector is read and written once per step with 16-byte
//     nontemporal loads and stores where a wave's access covers whole cache
//     lines (each byte is touched once: keeping it out of the caches leaves
//     them to the small shared data); lane-strided accesses, where a lane
//     walks its own line in several loads, stay plain so that the line is
//     fetched once;
//   * elementwise kernels give one float4 to each thread of a grid that covers
//     the whole shard, so the workgroups in flight cover a compact, contiguous
//     address window; the reconstruction uses the same shape within chunks
//     (one 256-thread workgroup per 1024-element block of a chunk);
//   * chunk kernels (compress, server) need a chunk's L1 norm before any of its
//     outputs can be written, so one workgroup owns a whole chunk and keeps it
//     in registers: one pass over HBM.
//
// Chunk layout in a workgroup: L lanes per chunk (a power of two <= 1024);
// lane lc holds, for each block k < V, the four elements 4*L*k + 4*lc + {0..3},
// so a block of 4L elements is one contiguous, coalesced span per buffer.
// The chunk's L1 norm is the in-lane (|a0|+|a1|)+(|a2|+|a3|), an xor butterfly
// over the lanes of a wave (partners l and l^o hold adjacent index ranges),
// then an in-order tree over the chunk's waves and over its blocks: exactly the
// balanced pairwise tree over the chunk in index order (the zero padding
// beyond the chunk length adds +0 and changes no bit).  Packed signs: dword j
// of a chunk holds elements 32j..32j+31, assembled by an OR butterfly over 8
// lanes (4 bits per lane) and stored by every 8th lane.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "zo_internal.h"

namespace zo {

typedef float f4v __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------------------
// streaming access helpers
// ---------------------------------------------------------------------------

__device__ __forceinline__ f4v ldnt(const float *p, int64_t i4)
{
    return __builtin_nontemporal_load(reinterpret_cast<const f4v *>(p) + i4);
}

__device__ __forceinline__ void stnt(float *p, int64_t i4, f4v v)
{
    __builtin_nontemporal_store(v, reinterpret_cast<f4v *>(p) + i4);
}

typedef uint32_t u2v __attribute__((ext_vector_type(2)));

// Four elements i4*4 .. i4*4+3 of a gradient array of element type GT
// (binary32, or binary16 / bfloat16 widened exactly), as a float4.  The type
// is a template argument: a run-time switch would leave loads of different
// widths pending across a branch merge, and the compiler then waits for all
// of them before the next load.
template <int GT>
__device__ __forceinline__ f4v ldg4(const void *p, int64_t i4)
{
    if constexpr (GT == GT_F32) {
        return ldnt(static_cast<const float *>(p), i4);
    } else {
        const u2v w = __builtin_nontemporal_load(static_cast<const u2v *>(p) + i4);
        f4v r;
#pragma unroll
        for (int q = 0; q < 2; ++q) {
            if constexpr (GT == GT_BF16) {
                r[2 * q] = __uint_as_float(w[q] << 16);
                r[2 * q + 1] = __uint_as_float(w[q] & 0xFFFF0000u);
            } else {
                r[2 * q] = (float)__builtin_bit_cast(_Float16, (uint16_t)(w[q] & 0xFFFFu));
                r[2 * q + 1] = (float)__builtin_bit_cast(_Float16, (uint16_t)(w[q] >> 16));
            }
        }
        return r;
    }
}

// Calls f(integral_constant<GT>) for a run-time gradient type.
template <class F>
static hipError_t with_grad_type(int gt, F &&f)
{
    switch (gt) {
    case GT_F32: return f(std::integral_constant<int, GT_F32>{});
    case GT_F16: return f(std::integral_constant<int, GT_F16>{});
    case GT_BF16: return f(std::integral_constant<int, GT_BF16>{});
    default: return hipErrorInvalidValue;
    }
}

// Momentum / model / buffer lines of Algorithm 1 for one element, with the
// fresh momentum in the model and buffer lines.
__device__ __forceinline__ void local_elem(float g, float &m, float &x, float v, float &u,
                                           const Scalars &s)
{
    float mn = s.b1 * m + s.c1 * g;
    float p = s.gamma * mn;
    float den = sqrtf(v + s.eps);
    x = x - p / den;
    u = u + p;
    m = mn;
}

// Variance line of Algorithm 1.
__device__ __forceinline__ float var_elem(float v, float gb, const Scalars &s)
{
    return s.b2 * v + s.c2 * (gb * gb);
}

// ---------------------------------------------------------------------------
// a1 (+a2): local step, one float4 per thread
// ---------------------------------------------------------------------------

// The chunk c and the offset e (a multiple of 4) in it of this thread's
// float4; false when the thread has none.
__device__ __forceinline__ bool chunk_slot(Chunks ch, int64_t nchunks, int bpc, int lb,
                                           int64_t &c, int &e)
{
    if (bpc > 1) {
        c = (int64_t)blockIdx.x / bpc;
        e = 1024 * (int)(blockIdx.x - c * bpc) + 4 * (int)threadIdx.x;
    } else {
        c = (int64_t)blockIdx.x * (256 / lb) + threadIdx.x / lb;
        e = 4 * (int)(threadIdx.x % lb);
    }
    return c < nchunks && e < ch.len[c];
}

// The momentum of float4 e/4 of chunk c after a deferred reconstruction:
// (sign bit ? S_c : -S_c) / Gamma from the library's copy of the server output
// (the reconstruction's own expression).
__device__ __forceinline__ f4v m_from_copy(const SrvCopy &sm, const Chunks &ch, int64_t c, int e)
{
    const uint32_t bits = sm.words32[2 * ch.word[c] + (e >> 5)] >> (e & 31);
    // (-S)/Gamma = -(S/Gamma): a rounded quotient is odd in its dividend, so
    // one division per chunk gives every element's value
    const float mq = sm.scales[c] / sm.gamma_m;
    f4v r;
#pragma unroll
    for (int q = 0; q < 4; ++q) r[q] = ((bits >> q) & 1u) ? mq : -mq;
    return r;
}

// The buffer before this step, per BufferIn (m_old: the momentum read).
template <int UIN>
__device__ __forceinline__ f4v buffer_in(const float *u, int64_t i4, f4v m_old, const Scalars &s)
{
    if constexpr (UIN == U_MEM) {
        return ldnt(u, i4);
    } else if constexpr (UIN == U_ZERO) {
        return f4v{0.f, 0.f, 0.f, 0.f};
    } else {
        f4v r;
#pragma unroll
        for (int q = 0; q < 4; ++q) r[q] = 0.0f + s.gamma_u * m_old[q];
        return r;
    }
}

// The model is read from x_src (x itself, or the anchor when the last
// synchronisation left the model there) and written to x.  UIN: where u is
// (BufferIn).  WU: write u (false only with U_ZERO: the new u = +0 + gamma m'
// is then left implicit, U_GM for the next call).
// UIN = U_ZERO runs over the chunk grid (chunk_slot) and takes m from the
// server copy; the other variants run one float4 per thread over the shard.
template <bool VAR, int UIN, bool WU, int GT>
__global__ __launch_bounds__(256) void k_local(const void *__restrict__ g, float *__restrict__ m,
                                               const float *x_src, float *x,
                                               float *__restrict__ v, float *__restrict__ u,
                                               const void *__restrict__ gbar, int64_t n4,
                                               Scalars s, Chunks ch, int64_t nchunks, int bpc,
                                               int lb, SrvCopy sm)
{
    int64_t i;
    f4v mm;
    if constexpr (UIN == U_ZERO) {
        int64_t c;
        int e;
        if (!chunk_slot(ch, nchunks, bpc, lb, c, e)) return;
        i = (ch.start[c] + e) >> 2;
        mm = m_from_copy(sm, ch, c, e);
    } else {
        i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
        if (i >= n4) return;
        mm = ldnt(m, i);
    }
    f4v gg = ldg4<GT>(g, i), xx = ldnt(x_src, i), vv = ldnt(v, i);
    f4v uu = buffer_in<UIN>(u, i, mm, s);
    f4v gb;
    if (VAR) gb = ldg4<GT>(gbar, i);
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        float mc = mm[c], xc = xx[c], uc = uu[c];
        local_elem(gg[c], mc, xc, vv[c], uc, s);
        mm[c] = mc;
        xx[c] = xc;
        uu[c] = uc;
    }
    stnt(m, i, mm);
    stnt(x, i, xx);
    if (WU) stnt(u, i, uu);
    if (VAR) {
#pragma unroll
        for (int c = 0; c < 4; ++c) vv[c] = var_elem(vv[c], gb[c], s);
        stnt(v, i, vv);
    }
}

// a2 standalone.
template <int GT>
__global__ __launch_bounds__(256) void k_var(float *__restrict__ v, const void *__restrict__ gbar,
                                             int64_t n4, Scalars s)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n4) return;
    f4v vv = ldnt(v, i), gb = ldg4<GT>(gbar, i);
#pragma unroll
    for (int c = 0; c < 4; ++c) vv[c] = var_elem(vv[c], gb[c], s);
    stnt(v, i, vv);
}

// ---------------------------------------------------------------------------
// chunk machinery
// ---------------------------------------------------------------------------

// Sum over the lanes of a chunk that share a wave: xor butterfly.
template <int L>
__device__ __forceinline__ float wave_tree(float x)
{
#pragma unroll
    for (int o = 1; o < (L < 64 ? L : 64); o <<= 1) x = x + __shfl_xor(x, o);
    return x;
}

template <int L>
__device__ __forceinline__ uint32_t wave_or8(uint32_t x)
{
#pragma unroll
    for (int o = 1; o < (L < 8 ? L : 8); o <<= 1) x |= (uint32_t)__shfl_xor((int)x, o);
    return x;
}

// The chunk's pairwise L1 tree from each lane's per-block partial sums (the
// in-lane level).  Returns the total to every lane of the chunk.  Every
// thread of the workgroup must call it (it synchronises when L > 64).  `lds`
// holds (blockDim / 64) * V floats.
template <int L, int V>
__device__ __forceinline__ float chunk_tree(float (&part)[V], float *lds)
{
#pragma unroll
    for (int k = 0; k < V; ++k) part[k] = wave_tree<L>(part[k]);
    if constexpr (L <= 64) {
        // the chunk's lanes share a wave: the in-order tree over its blocks
#pragma unroll
        for (int h = 1; h < V; h <<= 1) {
#pragma unroll
            for (int k = 0; k + h < V; k += 2 * h) part[k] = part[k] + part[k + h];
        }
        return part[0];
    } else {
        constexpr int NW = L / 64;  // waves per chunk
        const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
        __syncthreads();  // lds may still be read by a previous call
        if (lane == 0) {
#pragma unroll
            for (int k = 0; k < V; ++k) lds[wave * V + k] = part[k];
        }
        __syncthreads();
        const int base = (wave / NW) * NW;
        float bs[V];
#pragma unroll
        for (int k = 0; k < V; ++k) {
            float t[NW];
#pragma unroll
            for (int w = 0; w < NW; ++w) t[w] = lds[(base + w) * V + k];
#pragma unroll
            for (int h = 1; h < NW; h <<= 1) {
#pragma unroll
                for (int w = 0; w + h < NW; w += 2 * h) t[w] = t[w] + t[w + h];
            }
            bs[k] = t[0];
        }
#pragma unroll
        for (int h = 1; h < V; h <<= 1) {
#pragma unroll
            for (int k = 0; k + h < V; k += 2 * h) bs[k] = bs[k] + bs[k + h];
        }
        return bs[0];
    }
}

__device__ __forceinline__ float abs4(f4v a)
{
    return (fabsf(a[0]) + fabsf(a[1])) + (fabsf(a[2]) + fabsf(a[3]));
}

__device__ __forceinline__ uint32_t sign4(f4v a)
{
    return (a[0] >= 0.0f ? 1u : 0u) | (a[1] >= 0.0f ? 2u : 0u) | (a[2] >= 0.0f ? 4u : 0u) |
           (a[3] >= 0.0f ? 8u : 0u);
}

__device__ __forceinline__ float ef_elem(float a, float s)
{
    return a >= 0.0f ? a - s : a + s;
}

// Equation 3 with error feedback on one chunk whose values `a` are in the
// lanes' registers (zeros beyond `len`): writes the new error, the packed
// signs (all 2*ceil(len/64) dwords of the chunk) and the scale.
// get_a(k) returns block k of a (from registers or from where the caller
// stashed it); part[k] = abs4 of it, formed by the caller.
template <int L, int V, class GetA>
__device__ __forceinline__ void compress_chunk_from(const float (&part_in)[V], GetA get_a, int lc,
                                                    int len, bool active,
                                                    float *__restrict__ err, int64_t err_e0,
                                                    uint32_t *__restrict__ words32,
                                                    float *scale_out, float *lds)
{
    float part[V];
#pragma unroll
    for (int k = 0; k < V; ++k) part[k] = part_in[k];
    const float tot = chunk_tree<L, V>(part, lds);
    const float s = tot / (float)len;
    const int ndw = 2 * ((len + 63) >> 6);
    uint32_t pend = 0;  // L < 8: several blocks share a dword
#pragma unroll
    for (int k = 0; k < V; ++k) {
        const int e = 4 * L * k + 4 * lc;
        const bool valid = active && e < len;
        uint32_t nib = 0;
        if (valid) {
            const f4v ak = get_a(k);
            f4v d;
#pragma unroll
            for (int c = 0; c < 4; ++c) d[c] = ef_elem(ak[c], s);
            stnt(err, (err_e0 + e) >> 2, d);
            nib = sign4(ak);
        }
        const uint32_t dw = wave_or8<L>(nib << (4 * (lc & 7)));
        if constexpr (L >= 8) {
            // lanes 8q..8q+7 hold dword 4Lk/32 + q
            if (active && (lc & 7) == 0) {
                const int j = e >> 5;
                if (j < ndw) words32[j] = dw;
            }
        } else {
            pend |= dw << ((4 * L * k) & 31);
            if (((4 * L * (k + 1)) & 31) == 0 || k == V - 1) {
                const int j = (4 * L * k) >> 5;
                if (active && lc == 0 && j < ndw) words32[j] = pend;
                pend = 0;
            }
        }
    }
    // the chunk's last word may hold a dword of pad bits only, past the lanes
    constexpr int kCovered = (4 * L * V + 31) / 32;
    if (active && lc == 0 && kCovered < ndw) words32[kCovered] = 0u;
    if (active && lc == 0) *scale_out = s;
}

template <int L, int V>
__device__ __forceinline__ void compress_chunk(f4v (&a)[V], int lc, int len, bool active,
                                               float *__restrict__ err, int64_t err_e0,
                                               uint32_t *__restrict__ words32, float *scale_out,
                                               float *lds)
{
    float part[V];
#pragma unroll
    for (int k = 0; k < V; ++k) part[k] = abs4(a[k]);
    compress_chunk_from<L, V>(part, [&](int k) { return a[k]; }, lc, len, active, err, err_e0,
                              words32, scale_out, lds);
}

// ---------------------------------------------------------------------------
// a3: worker compress + error feedback + pack (fused with the momentum and
// buffer lines when g != nullptr)
// ---------------------------------------------------------------------------

// UIN (with FUSED only; U_MEM otherwise): where u is (BufferIn).  GT: element
// type of g when FUSED, else of u (binary32 u, or the gradient itself under
// Algorithm 4).
template <int L, int V, bool FUSED, int UIN, int GT>
__global__ __launch_bounds__(L > 256 ? L : 256, V > 1 ? 8 : 1) void k_sync1(
    const void *__restrict__ g, const float *__restrict__ m, const void *__restrict__ u,
    float *__restrict__ err, Chunks ch, int64_t nchunks, uint32_t *__restrict__ packed32,
    float *__restrict__ scales, Scalars s, SrvCopy sm)
{
    __shared__ float lds[64];
    // With several blocks per lane, a is parked in LDS across the chunk's
    // reduction instead of in registers: that keeps a 1024-lane chunk within
    // 64 registers, so two chunks share a CU.
    constexpr bool kStash = V > 1;
    __shared__ f4v stash[kStash ? L * V : 1];
    constexpr int CPW = L >= 256 ? 1 : 256 / L;
    const int lc = threadIdx.x % L;
    const int64_t c = (int64_t)blockIdx.x * CPW + threadIdx.x / L;
    const bool active = c < nchunks;
    const int len = active ? ch.len[c] : 0;
    const int64_t e0 = active ? ch.start[c] : 0;
    f4v a[kStash ? 1 : V];
    float part[V];
#pragma unroll
    for (int k = 0; k < V; ++k) {
        const int e = 4 * L * k + 4 * lc;
        f4v ak = f4v{0.f, 0.f, 0.f, 0.f};
        if (e < len) {
            const int64_t i4 = (e0 + e) >> 2;
            const f4v dd = ldnt(err, i4);
            f4v uu;
            if (FUSED) {
                const f4v gg = ldg4<GT>(g, i4);
                const f4v mm = UIN == U_ZERO ? m_from_copy(sm, ch, c, e) : ldnt(m, i4);
                uu = buffer_in<UIN>(static_cast<const float *>(u), i4, mm, s);
#pragma unroll
                for (int q = 0; q < 4; ++q) uu[q] = uu[q] + s.gamma * (s.b1 * mm[q] + s.c1 * gg[q]);
            } else {
                uu = ldg4<GT>(u, i4);
            }
#pragma unroll
            for (int q = 0; q < 4; ++q) ak[q] = uu[q] + dd[q];
        }
        part[k] = abs4(ak);
        if constexpr (kStash)
            stash[k * L + lc] = ak;
        else
            a[k] = ak;
    }
    compress_chunk_from<L, V>(
        part, [&](int k) { return kStash ? stash[k * L + lc] : a[kStash ? 0 : k]; }, lc, len,
        active, err, e0, packed32 + 2 * (active ? ch.word[c] : 0), scales + (active ? c : 0), lds);
}

// ---------------------------------------------------------------------------
// a4: server -- unpack W workers, exact average, server error feedback, pack
// ---------------------------------------------------------------------------

// Exact-sum condition for one chunk's scales (see zo_unpack_average): every
// partial sum of +-S_w is a multiple of the smallest ulp among the nonzero
// scales and below W * 2^(largest exponent + 1), so it is exact in binary64
// when that span fits 53 bits.  Evaluated by the first min(L, 64) lanes of the
// chunk; returns 1 when violated (or a scale is not finite).
template <int L>
__device__ __forceinline__ uint32_t inexact_flag(const float *__restrict__ sc, int64_t cstride,
                                                 int W, int lc)
{
    constexpr int LW = L < 64 ? L : 64;
    int lo = 1 << 20, hi = -(1 << 20), bad = 0;
    if (lc < LW) {
        for (int w = lc; w < W; w += LW) {
            uint32_t b = __float_as_uint(sc[cstride * w]) & 0x7FFFFFFFu;
            if (b == 0) continue;
            int f = (int)(b >> 23);
            if (f == 255) { bad = 1; continue; }
            int l, h;
            if (f == 0) {
                l = -149;
                h = (31 - __clz((int)b)) - 149;
            } else {
                l = f - 150;
                h = f - 127;
            }
            lo = min(lo, l);
            hi = max(hi, h);
        }
    }
#pragma unroll
    for (int o = 1; o < LW; o <<= 1) {
        lo = min(lo, __shfl_xor(lo, o));
        hi = max(hi, __shfl_xor(hi, o));
        bad |= __shfl_xor(bad, o);
    }
    int lg = 0;
    while ((1 << lg) < W) ++lg;
    if (hi < lo) return (uint32_t)bad;  // every scale is zero
    return (uint32_t)(bad || (hi + 1 + lg - lo > 53));
}

// Plain server: per element, per worker, select +-S_w and add in binary64.
// Kept for worker counts whose lookup tables do not fit in LDS.
template <int L, int V>
__global__ __launch_bounds__(L > 256 ? L : 256) void k_srv_plain(
    const uint32_t *__restrict__ packed32, const float *__restrict__ scales, int W,
    int64_t wstride, int64_t cstride, Chunks ch, int64_t c0, int64_t nch, int64_t word0,
    int64_t elem0, float *__restrict__ srv_err, uint32_t *__restrict__ srv_packed32,
    float *__restrict__ srv_scales, float *__restrict__ avg_out, uint8_t *__restrict__ flags,
    double inv_w, int w_pow2)
{
    __shared__ float lds[64];
    constexpr int CPW = L >= 256 ? 1 : 256 / L;
    const int lc = threadIdx.x % L;
    const int64_t cr = (int64_t)blockIdx.x * CPW + threadIdx.x / L;  // chunk within range
    const bool active = cr < nch;
    const int64_t c = c0 + (active ? cr : 0);
    const int len = active ? ch.len[c] : 0;
    const int64_t el = active ? ch.start[c] - elem0 : 0;  // element offset in range
    const int64_t wd = active ? ch.word[c] - word0 : 0;   // word offset in range
    f4v b[V];
#pragma unroll
    for (int k = 0; k < V; ++k) {
        const int e = 4 * L * k + 4 * lc;
        b[k] = f4v{0.f, 0.f, 0.f, 0.f};
        if (e < len) {
            double acc[4] = {0.0, 0.0, 0.0, 0.0};
            const int64_t dwi = 2 * wd + (e >> 5);
            const int sh = e & 31;
            for (int w = 0; w < W; ++w) {
                const uint32_t bits = packed32[2 * wstride * w + dwi] >> sh;
                const double sw = (double)scales[cstride * w + cr];
#pragma unroll
                for (int q = 0; q < 4; ++q) acc[q] += ((bits >> q) & 1u) ? sw : -sw;
            }
            f4v av;
#pragma unroll
            for (int q = 0; q < 4; ++q)
                av[q] = w_pow2 ? (float)(acc[q] * inv_w) : (float)(acc[q] / (double)W);
            if (avg_out) stnt(avg_out, (el + e) >> 2, av);
            const f4v d = ldnt(srv_err, (el + e) >> 2);
#pragma unroll
            for (int q = 0; q < 4; ++q) b[k][q] = av[q] + d[q];
        }
    }
    compress_chunk<L, V>(b, lc, len, active, srv_err, el,
                         srv_packed32 + 2 * (active ? ch.word[c] : 0), srv_scales + c, lds);
    // sticky: a flag once set stays set until the handle is recreated
    const uint32_t f = inexact_flag<L>(scales + (active ? cr : 0), cstride, W, lc);
    if (active && lc == 0 && f) flags[cr] = 1;
}

// Server with a lookup table per group of 8 workers ("four Russians"): for a
// chunk, T_g[b] = sum_{k<8} (bit k of b ? +S_{8g+k} : -S_{8g+k}) in binary64
// for all 256 bytes b; an element's sum over W workers is then the sum over
// groups of T_g[byte of its 8 workers' bits].  Under the exact-sum condition
// every partial sum is exact, so any grouping gives the bits of the
// sequential sum.  Lane mapping: one lane owns the 32 elements of one packed
// dword per round (round r, lane lc -> dword r*LD + lc of the chunk); the
// 8 x 32 bit block of a worker group is transposed in registers so that byte c
// of register k holds element 8c+k's 8 worker bits.

// Swap the bits selected by m << s in x with the bits selected by m in y
// (a delta swap written as two bit-field inserts).
__device__ __forceinline__ void swap_bits(uint32_t &x, uint32_t &y, int s, uint32_t m)
{
    const uint32_t xs = x >> s, ys = y << s;
    y = (xs & m) | (y & ~m);
    x = (ys & (m << s)) | (x & ~(m << s));
}

__device__ __forceinline__ void transpose8x32(uint32_t (&x)[8])
{
#pragma unroll
    for (int k = 0; k < 4; ++k) swap_bits(x[k], x[k + 4], 4, 0x0F0F0F0Fu);
    swap_bits(x[0], x[2], 2, 0x33333333u);
    swap_bits(x[1], x[3], 2, 0x33333333u);
    swap_bits(x[4], x[6], 2, 0x33333333u);
    swap_bits(x[5], x[7], 2, 0x33333333u);
#pragma unroll
    for (int k = 0; k < 8; k += 2) swap_bits(x[k], x[k + 1], 1, 0x55555555u);
}

// Byte C of x times 8 (a table offset in bytes) in one SDWA instruction.
template <int C>
__device__ __forceinline__ uint32_t byte_x8(uint32_t x)
{
    uint32_t r;
    if constexpr (C == 0)
        asm("v_lshlrev_b32_sdwa %0, 3, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD "
            "src1_sel:BYTE_0" : "=v"(r) : "v"(x));
    else if constexpr (C == 1)
        asm("v_lshlrev_b32_sdwa %0, 3, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD "
            "src1_sel:BYTE_1" : "=v"(r) : "v"(x));
    else if constexpr (C == 2)
        asm("v_lshlrev_b32_sdwa %0, 3, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD "
            "src1_sel:BYTE_2" : "=v"(r) : "v"(x));
    else
        asm("v_lshlrev_b32_sdwa %0, 3, %1 dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:DWORD "
            "src1_sel:BYTE_3" : "=v"(r) : "v"(x));
    __builtin_assume(r < 2048u);  // lets the table base fold into the LDS offset
    return r;
}

// Workgroups are dealt to the GPU's 8 XCDs round-robin (workgroup i to XCD
// i % 8), and each XCD has its own L2.  With the grid padded to a multiple
// of 8 workgroups, block i takes block number (i % 8) * (grid / 8) + i / 8:
// every XCD walks a contiguous run of blocks in order, so neighbouring
// chunks share its L2 (in every worker's row the cache line that straddles
// two chunks' words, and each line holding 32 chunks' scales).
constexpr int kXcds = 8;

__device__ __forceinline__ int64_t xcd_block()
{
    const int64_t per = gridDim.x / kXcds;
    return (int64_t)(blockIdx.x % kXcds) * per + blockIdx.x / kXcds;
}

static inline unsigned xcd_grid(unsigned blocks)
{
    return (blocks + kXcds - 1) / kXcds * kXcds;
}

// Load the 8 dwords of worker group g (workers beyond W read as 0).  Plain
// loads: the nontemporal hint measured no faster for these dword accesses.
// a value the whole wave agrees on, moved to scalar registers: a load at
// p + wave_uniform(off) + lane is then addressed as scalar base + lane offset
__device__ __forceinline__ int64_t wave_uniform(int64_t v)
{
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)(uint64_t)v);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)((uint64_t)v >> 32));
    return (int64_t)(((uint64_t)hi << 32) | lo);
}

// Dword lc of the chunk for the 8 workers of group g: worker w's words start
// at dword off + ws*w.  UNIFORM: the whole wave is on one chunk, so the row
// offsets are scalars and each load costs one address add.
template <bool UNIFORM>
__device__ __forceinline__ void load_group(uint32_t (&x)[8], const uint32_t *packed32, int64_t off,
                                           int64_t ws, int g, int W, uint32_t lc)
{
    int64_t r[8];
#pragma unroll
    for (int k = 0; k < 8; ++k)
        r[k] = UNIFORM ? wave_uniform(off + ws * (8 * g + k)) : off + ws * (8 * g + k);
    if (8 * g + 8 <= W) {
#pragma unroll
        for (int k = 0; k < 8; ++k) x[k] = packed32[r[k] + lc];
    } else {
#pragma unroll
        for (int k = 0; k < 8; ++k) x[k] = 8 * g + k < W ? packed32[r[k] + lc] : 0u;
    }
}

// Worker groups whose packed words are loaded ahead of the one being summed
// (HBM latency is hidden by bytes in flight, and the table lookups leave
// registers for only a few groups).
constexpr int kSrvPrefetch = 2;

// Chunks of fewer than 64 dwords (several chunks per wave) look up the two
// 16-entry half tables of each group directly instead of building the
// 256-entry table from them: the build would cost as much as the lookups, and
// the smaller tables leave LDS for more waves per CU.
constexpr bool srv_nibble(int LD) { return LD < 64; }

// Chunks per workgroup of the LUT server: enough chunks to fill a wave when a
// chunk has fewer than 64 dwords, as long as their tables fit in 64 KB.
constexpr int srv_chunks_per_block(int LD, int G)
{
    const int fill = LD >= 64 ? 1 : 64 / LD;
    const int per = srv_nibble(LD) ? 256 : 32;  // chunks of G groups' tables in 64 KB, times G
    const int fit = per / G > 1 ? per / G : 1;
    int c = fill < fit ? fill : fit;
    while (c & (c - 1)) c &= c - 1;  // a power of two (G need not be one)
    return c;
}

// Eight table lookups (byte C of the eight transposed registers) added to
// their accumulators.  The empty asm consumes the eight sums: the adds, and so
// the table reads, of one batch complete before the next batch's reads are
// issued (otherwise the scheduler hoists every read of the unrolled groups and
// their results, two registers each, spill).
template <int C>
__device__ __forceinline__ void lookup8(double (&acc)[32], const uint32_t (&x)[8], const char *tg)
{
#pragma unroll
    for (int k = 0; k < 8; ++k)
        acc[8 * C + k] += *reinterpret_cast<const double *>(tg + byte_x8<C>(x[k]));
    asm volatile(""
                 : "+v"(acc[8 * C + 0]), "+v"(acc[8 * C + 1]), "+v"(acc[8 * C + 2]),
                   "+v"(acc[8 * C + 3]), "+v"(acc[8 * C + 4]), "+v"(acc[8 * C + 5]),
                   "+v"(acc[8 * C + 6]), "+v"(acc[8 * C + 7])
                 :
                 : "memory");
}

// The same for the half tables at hg (16 entries for the low nibble of a
// worker byte, workers 8g..8g+3, then 16 for the high nibble): two lookups per
// element; every partial sum is exact, so the order of the adds does not
// matter.
template <int C>
__device__ __forceinline__ void lookup8_nib(double (&acc)[32], const uint32_t (&x)[8],
                                            const char *hg)
{
#pragma unroll
    for (int k = 0; k < 8; ++k) {
        // nibble times 8 (a byte offset into its 128-byte table)
        const uint32_t lo = C == 0 ? (x[k] << 3) & 0x78u : (x[k] >> (8 * C - 3)) & 0x78u;
        const uint32_t hi = (x[k] >> (8 * C + 1)) & 0x78u;
        acc[8 * C + k] += *reinterpret_cast<const double *>(hg + lo);
        acc[8 * C + k] += *reinterpret_cast<const double *>(hg + 128 + hi);
    }
    asm volatile(""
                 : "+v"(acc[8 * C + 0]), "+v"(acc[8 * C + 1]), "+v"(acc[8 * C + 2]),
                   "+v"(acc[8 * C + 3]), "+v"(acc[8 * C + 4]), "+v"(acc[8 * C + 5]),
                   "+v"(acc[8 * C + 6]), "+v"(acc[8 * C + 7])
                 :
                 : "memory");
}

// Float4 slot of the transpose buffer that holds float4 t of a chunk (t = e/4).
// Lane j writes the slots 8j..8j+7 of its dword; lanes then read slots in
// coalesced order.  XOR-ing the slot's low three bits with bits 1..3 of j makes
// both the writes and the reads of 16 consecutive lanes hit 16 distinct
// 16-byte bank groups.
__device__ __forceinline__ int xpose_slot(int t)
{
    return 8 * (t >> 3) + ((t & 7) ^ ((t >> 4) & 7));
}

// LD lanes per chunk (one packed dword each), G groups of 8 workers (a
// compile-time count; groups past the last worker hold zero tables), CPW
// chunks per workgroup.  The tables of chunk q of the workgroup start at byte
// q*G*2048 of `tab` (with half tables, q*G*256 of `half`); with one chunk per
// workgroup the offset of every lookup is an immediate.  With half tables the
// register budget is held to the waves per SIMD that the workgroups' LDS
// allows, at most four (at 1024-element chunks and W = 32: four, with a
// 20-byte spill; 74 instead of 81 us on the ResNet-50 shape).
constexpr int srv_lut_waves(int LD, int G)
{
    if (!srv_nibble(LD)) return 1;  // no bound beyond the workgroup size
    const int cpw = srv_chunks_per_block(LD, G);
    const int lds = cpw * LD * 128 + cpw * G * (256 + 32) + 256;  // transpose, tables, scales, tree
    const int per_cu = 160 * 1024 / lds;                         // one-wave workgroups per CU
    const int per_simd = (per_cu + 3) / 4;
    return per_simd < 1 ? 1 : (per_simd > 4 ? 4 : per_simd);
}

template <int LD, int G>
__global__ __launch_bounds__(LD > 64 ? LD : 64)
__attribute__((amdgpu_waves_per_eu(srv_lut_waves(LD, G)))) void k_srv_lut(
    const uint32_t *__restrict__ packed32, const float *__restrict__ scales, int W,
    int64_t wstride, int64_t cstride, Chunks ch, int64_t c0, int64_t nch, int64_t word0,
    int64_t elem0, float *__restrict__ srv_err, uint32_t *__restrict__ srv_packed32,
    float *__restrict__ srv_scales, float *__restrict__ avg_out, uint8_t *__restrict__ flags,
    double inv_w, int w_pow2)
{
    constexpr int CPW = srv_chunks_per_block(LD, G);
    constexpr bool kNib = srv_nibble(LD);
    // static arrays: their LDS addresses are link-time constants, so the group
    // offset of every lookup is an instruction immediate.  The tables are dead
    // once the sums are formed; the same memory then transposes the averages.
    constexpr int kTabBytes = kNib ? 0 : CPW * G * 256 * 8;
    constexpr int kXposeBytes = CPW * LD * 32 * 4;
    __shared__ double uni[(kTabBytes > kXposeBytes ? kTabBytes : kXposeBytes) / 8];
    __shared__ float sc[CPW * G * 8];  // W <= 8G
    __shared__ double half[CPW * G * 32];  // per group: 16 sums of workers 0-3, 16 of 4-7
    __shared__ float tree[64];
    double *tab = uni;

    const int q = CPW == 1 ? 0 : (int)threadIdx.x / LD;
    const int lc = CPW == 1 ? (int)threadIdx.x : (int)threadIdx.x % LD;
    const int64_t cbase = xcd_block() * CPW;
    const int64_t cr = cbase + q;
    const bool active = cr < nch;
    const int64_t c = c0 + (active ? cr : 0);
    const int len = active ? ch.len[c] : 0;
    const int64_t el = active ? ch.start[c] - elem0 : 0;
    const int64_t wd = active ? ch.word[c] - word0 : 0;

    // lane lc sums the 32 elements of dword lc of the chunk, if the chunk has it
    const int ndw_data = (len + 31) >> 5;
    const bool has_dw = lc < ndw_data;
    const int64_t ws = 2 * wstride;
    const int64_t off = 2 * wd;
    constexpr bool kUni = LD >= 64;  // a wave never spans two chunks
    uint32_t ring[kSrvPrefetch + 1][8];
    // the first groups' packed words are in flight while the tables are built
    if (has_dw) {
#pragma unroll
        for (int g = 0; g < kSrvPrefetch && g < G; ++g)
            load_group<kUni>(ring[g], packed32, off, ws, g, W, lc);
    }

    // stage the scales of the workgroup's chunks, then build the tables
    for (int i = threadIdx.x; i < CPW * W; i += blockDim.x) {
        const int qq = i / W, w = i - qq * W;
        sc[i] = (cbase + qq < nch) ? scales[cstride * w + cbase + qq] : 0.0f;
    }
    __syncthreads();
    // T_g[b] = H_g,0[b & 15] + H_g,1[b >> 4], with H_g,h[n] the signed sum of
    // workers 8g+4h .. 8g+4h+3 (every partial sum is exact, so the split is
    // too)
    for (int i = threadIdx.x; i < CPW * G * 32; i += blockDim.x) {
        const int qq = i / (G * 32), g = (i >> 5) % G, h = (i >> 4) & 1, nb = i & 15;
        double t = 0.0;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int w = 8 * g + 4 * h + k;
            if (w < W) {
                const double sw = (double)sc[qq * W + w];
                t += ((nb >> k) & 1) ? sw : -sw;
            }
        }
        half[i] = t;
    }
    __syncthreads();
    if constexpr (!kNib) {
        // CPW * G * 256 entries over LD * CPW threads, kPer = the ceiling of
        // their ratio each (a thread past the last entry repeats one from the
        // start: the same value written twice), in batches
        // of at most 8 whose reads are all issued before the first add (a
        // narrow workgroup has thousands of entries per thread: one batch at
        // a time keeps them out of scratch memory)
        constexpr int kTotal = CPW * G * 256, kThreads = LD * CPW;
        constexpr int kPer = (kTotal + kThreads - 1) / kThreads;
        constexpr int kBatch = kPer < 8 ? kPer : 8;
#pragma unroll 1
        for (int k0 = 0; k0 < kPer; k0 += kBatch) {
            double lo[kBatch], hi[kBatch];
#pragma unroll
            for (int k = 0; k < kBatch; ++k) {
                const int i = ((int)threadIdx.x + (k0 + k) * kThreads) % kTotal;
                const int qg = i >> 8, b = i & 255;  // qg = chunk * G + group
                lo[k] = half[32 * qg + (b & 15)];
                hi[k] = half[32 * qg + 16 + (b >> 4)];
            }
#pragma unroll
            for (int k = 0; k < kBatch; ++k)
                tab[((int)threadIdx.x + (k0 + k) * kThreads) % kTotal] = lo[k] + hi[k];
        }
        __syncthreads();
    }
    const char *mytab = kNib ? reinterpret_cast<const char *>(half) + (size_t)q * G * 256
                             : reinterpret_cast<const char *>(tab) + (size_t)q * G * 2048;

    // the server error of the lane's elements in the compress layout (lane lc
    // holds the float4s lc + LD*k, k < 8, of its chunk); loaded while the last
    // group's lookups run
    f4v serr[8];
    auto load_serr = [&]() {
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            const int e = 4 * LD * k + 4 * lc;
            serr[k] = e < len ? ldnt(srv_err, (el + e) >> 2) : f4v{0.f, 0.f, 0.f, 0.f};
        }
    };

    // the sum over workers of the lane's 32 elements
    double acc[32];
#pragma unroll
    for (int i = 0; i < 32; ++i) acc[i] = 0.0;
    if (has_dw) {
#pragma unroll
        for (int g = 0; g < G; ++g) {
            if (g + kSrvPrefetch < G)
                load_group<kUni>(ring[(g + kSrvPrefetch) % (kSrvPrefetch + 1)], packed32, off,
                                 ws, g + kSrvPrefetch, W, lc);
            uint32_t (&cur)[8] = ring[g % (kSrvPrefetch + 1)];
            transpose8x32(cur);
            if constexpr (kNib) {
                const char *hg = mytab + g * 256;
                lookup8_nib<0>(acc, cur, hg);
                lookup8_nib<1>(acc, cur, hg);
                lookup8_nib<2>(acc, cur, hg);
                if (g == G - 1) load_serr();
                lookup8_nib<3>(acc, cur, hg);
            } else {
                const char *tg = mytab + g * 2048;
                lookup8<0>(acc, cur, tg);
                lookup8<1>(acc, cur, tg);
                lookup8<2>(acc, cur, tg);
                if (g == G - 1) load_serr();
                lookup8<3>(acc, cur, tg);
            }
        }
    } else {
        load_serr();
    }
    {
        // sticky: a flag once set stays set until the handle is recreated
        const uint32_t f = inexact_flag<LD>(sc + q * W, 1, W, lc);
        if (active && lc == 0 && f) flags[cr] = 1;
    }

    // averages -> LDS, then back in the coalesced layout of the compress step
    __syncthreads();  // every lookup is done: the tables may be overwritten
    f4v *xp = reinterpret_cast<f4v *>(uni) + (size_t)q * LD * 8;
#pragma unroll
    for (int p = 0; p < 8; ++p) {
        f4v av;
#pragma unroll
        for (int qq = 0; qq < 4; ++qq)
            av[qq] = w_pow2 ? (float)(acc[4 * p + qq] * inv_w) : (float)(acc[4 * p + qq] / (double)W);
        xp[xpose_slot(8 * lc + p)] = av;
    }
    __syncthreads();
    f4v bv[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
        const int e = 4 * LD * k + 4 * lc;
        bv[k] = f4v{0.f, 0.f, 0.f, 0.f};
        if (e < len) {
            const f4v av = xp[xpose_slot(LD * k + lc)];
            if (avg_out) stnt(avg_out, (el + e) >> 2, av);
#pragma unroll
            for (int qq = 0; qq < 4; ++qq) bv[k][qq] = av[qq] + serr[k][qq];
        }
    }
    // Equation 3 with the server error
    compress_chunk<LD, 8>(bv, lc, len, active, srv_err, el,
                          srv_packed32 + 2 * (active ? ch.word[c] : 0), srv_scales + c, tree);
}

// ---------------------------------------------------------------------------
// a5 (+a2): reconstruct momentum and model from the server's compressed
// average; reset the buffer; move the anchor.  No reduction, so the grid is
// cut into 256-thread workgroups over <= 1024-element blocks of one chunk
// (bpc blocks per chunk) or, for short chunks, several chunks per workgroup
// (lb lanes per chunk).
// ---------------------------------------------------------------------------

// DEFER: only m and the anchor are written; the new model is the new anchor
// and u is +0, both left implicit until the next local step writes them.

template <bool VAR, bool DEFER, int GT>
__global__ __launch_bounds__(256) void k_recon(const uint32_t *__restrict__ srv_packed32,
                                               const float *__restrict__ srv_scales, Chunks ch,
                                               int64_t nchunks, int bpc, int lb,
                                               float *__restrict__ m, float *__restrict__ x,
                                               float *__restrict__ v, float *__restrict__ u,
                                               float *__restrict__ anchor,
                                               const void *__restrict__ gbar, float gsum,
                                               Scalars s, SrvCopy sm)
{
    int64_t c;
    int e;
    if (!chunk_slot(ch, nchunks, bpc, lb, c, e)) return;
    const int64_t i4 = (ch.start[c] + e) >> 2;
    const float sc = srv_scales[c];
    const int64_t wd = 2 * ch.word[c] + (e >> 5);
    const uint32_t dw = srv_packed32[wd];
    const uint32_t bits = dw >> (e & 31);
    if (DEFER) {
        // the copy the next step rebuilds m from (one thread per dword)
        if ((e & 31) == 0) sm.words32[wd] = dw;
        if (e == 0) sm.scales[c] = sc;
    }
    const f4v vv = ldnt(v, i4), an = ldnt(anchor, i4);
    f4v gb;
    if (VAR) gb = ldg4<GT>(gbar, i4);
    f4v mm, xx, nv;
    const float mq = sc / gsum;  // odd in sc, so one division serves both signs
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const float ub = ((bits >> q) & 1u) ? sc : -sc;
        mm[q] = ((bits >> q) & 1u) ? mq : -mq;
        xx[q] = an[q] - ub / sqrtf(vv[q] + s.eps);
        if (VAR) nv[q] = var_elem(vv[q], gb[q], s);
    }
    stnt(anchor, i4, xx);
    if (!DEFER) {
        stnt(m, i4, mm);
        stnt(x, i4, xx);
        stnt(u, i4, f4v{0.f, 0.f, 0.f, 0.f});
    }
    if (VAR) stnt(v, i4, nv);
}

// ---------------------------------------------------------------------------
// Algorithm 4 (frozen variance, compressed gradients; 1-bit Adam when T_v is a
// prefix): one step given the averaged gradient gbar, in the listing's order
//   v' = beta2 v + (1 - beta2) gbar^2 (t in T_v only);  m' = beta1 m + (1 - beta1) gbar;
//   x' = x - gamma m / sqrt(v + eps)   (the model line uses m_t and v_t)
// ---------------------------------------------------------------------------

__device__ __forceinline__ void fv_elem(float gb, float &x, float &m, float &v, bool full,
                                        const Scalars &s)
{
    const float v_old = v, m_old = m;
    if (full) v = var_elem(v_old, gb, s);
    m = s.b1 * m_old + s.c1 * gb;
    const float step = s.gamma * m_old;
    const float den = sqrtf(v_old + s.eps);
    x = x - step / den;
}

// t in T_v: gbar is the full-precision average.  One float4 per thread.
template <int GT>
__global__ __launch_bounds__(256) void k_fv_full(const void *__restrict__ gbar,
                                                 float *__restrict__ x, float *__restrict__ m,
                                                 float *__restrict__ v, int64_t n4, Scalars s)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n4) return;
    const f4v gb = ldg4<GT>(gbar, i);
    f4v xx = ldnt(x, i), mm = ldnt(m, i), vv = ldnt(v, i);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        float xc = xx[q], mc = mm[q], vc = vv[q];
        fv_elem(gb[q], xc, mc, vc, true, s);
        xx[q] = xc;
        mm[q] = mc;
        vv[q] = vc;
    }
    stnt(x, i, xx);
    stnt(m, i, mm);
    stnt(v, i, vv);
}

// t outside T_v: gbar = sigma * s of the server's packed words (v kept).
__global__ __launch_bounds__(256) void k_fv_apply(const uint32_t *__restrict__ srv_packed32,
                                                  const float *__restrict__ srv_scales, Chunks ch,
                                                  int64_t nchunks, int bpc, int lb,
                                                  float *__restrict__ x, float *__restrict__ m,
                                                  const float *__restrict__ v, Scalars s)
{
    int64_t c;
    int e;
    if (!chunk_slot(ch, nchunks, bpc, lb, c, e)) return;
    const int64_t i4 = (ch.start[c] + e) >> 2;
    const float sc = srv_scales[c];
    const uint32_t bits = srv_packed32[2 * ch.word[c] + (e >> 5)] >> (e & 31);
    const f4v vv = ldnt(v, i4);
    f4v xx = ldnt(x, i4), mm = ldnt(m, i4);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        float xc = xx[q], mc = mm[q], vc = vv[q];
        fv_elem(((bits >> q) & 1u) ? sc : -sc, xc, mc, vc, false, s);
        xx[q] = xc;
        mm[q] = mc;
    }
    stnt(x, i4, xx);
    stnt(m, i4, mm);
}

// dst = +0, one float4 per thread (u after a deferred reset).
__global__ __launch_bounds__(256) void k_zero(float *__restrict__ dst, int64_t n4)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n4) return;
    stnt(dst, i, f4v{0.f, 0.f, 0.f, 0.f});
}

// ---------------------------------------------------------------------------
// diagnostic: the division and square root the kernels use
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(256) void k_divsqrt(const float *__restrict__ a,
                                                 const float *__restrict__ b,
                                                 float *__restrict__ q, float *__restrict__ r,
                                                 int64_t n)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    q[i] = a[i] / b[i];
    r[i] = sqrtf(a[i]);
}

// Plain copy, one float4 per thread, with the same (nontemporal or plain)
// loads and stores as the streaming kernels: the reference for HBM byte
// counters.
template <bool NT>
__global__ __launch_bounds__(256) void k_copy(const float *__restrict__ src, float *__restrict__ dst,
                                              int64_t n4)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n4) return;
    if (NT)
        stnt(dst, i, ldnt(src, i));
    else
        reinterpret_cast<f4v *>(dst)[i] = reinterpret_cast<const f4v *>(src)[i];
}

// R read streams and S write streams of float4, one float4 per thread per
// stream, nontemporal: the achievable HBM rate of a streaming kernel's mix of
// arrays (every write depends on every read, so no load is dead, and a thread
// issues its stores after all of its loads: a dst that is also a src is
// updated in place, like the optimizer states a kernel reads and rewrites).
template <int R, int S>
__global__ __launch_bounds__(256) void k_stream(StreamPtrs p, int64_t n4)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n4) return;
    f4v acc = f4v{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const f4v a = ldnt(p.src[r], i);
#pragma unroll
        for (int q = 0; q < 4; ++q) acc[q] = acc[q] + a[q];
    }
#pragma unroll
    for (int w = 0; w < S; ++w) {
        f4v o;
#pragma unroll
        for (int q = 0; q < 4; ++q) o[q] = acc[q] + (float)w;
        stnt(p.dst[w], i, o);
    }
}

// The memory accesses of k_srv_lut without its arithmetic: per chunk of the
// server range one workgroup of LD lanes in the same XCD-aware order, each lane
// reading its dword of the chunk from all W workers' rows, then the chunk's
// server error loaded and stored back unchanged with the kernel's nontemporal
// accesses and float4 layout.  The error keeps its bits; timing it measures
// the rate the server's access pattern can reach.
template <int LD>
__global__ __launch_bounds__(LD) void k_srv_pattern(const uint32_t *__restrict__ packed32, int W,
                                                    int64_t wstride, Chunks ch, int64_t c0,
                                                    int64_t nch, int64_t word0, int64_t elem0,
                                                    float *__restrict__ srv_err)
{
    const int lc = (int)threadIdx.x;
    const int64_t cr = xcd_block();
    if (cr >= nch) return;
    const int64_t c = c0 + cr;
    const int len = ch.len[c];
    const int64_t el = ch.start[c] - elem0;
    const int64_t wd = ch.word[c] - word0;
    uint32_t x = 0;
    if (lc < (len + 31) >> 5) {
        const uint32_t *p = packed32 + 2 * wd + lc;
        const int64_t ws = 2 * wstride;
#pragma unroll 8
        for (int w = 0; w < W; ++w) x ^= p[ws * w];
    }
    asm volatile("" ::"v"(x));  // the loads are not dead
    f4v v[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
        const int e = 4 * LD * k + 4 * lc;
        if (e < len) v[k] = ldnt(srv_err, (el + e) >> 2);
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) {
        const int e = 4 * LD * k + 4 * lc;
        if (e < len) stnt(srv_err, (el + e) >> 2, v[k]);
    }
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------

static inline int next_pow2(int v)
{
    int p = 1;
    while (p < v) p <<= 1;
    return p;
}

// Lanes per chunk and blocks per lane of the compress kernels: one float4 per
// lane and block, up to 1024 lanes (16 waves) per chunk.
Geometry geometry_for(int chunk)
{
    const int lanes = (chunk + 3) / 4;
    if (lanes <= 256) return Geometry{next_pow2(lanes), 1};
    const int L = next_pow2(lanes) < 1024 ? next_pow2(lanes) : 1024;
    return Geometry{L, next_pow2((lanes + L - 1) / L)};
}

static inline unsigned grid_for(int64_t items, int64_t per_block)
{
    return (unsigned)((items + per_block - 1) / per_block);
}

// Calls f(integral_constant<L>, integral_constant<V>) for a supported geometry.
template <class F>
static hipError_t with_geometry(Geometry geo, F &&f)
{
    using std::integral_constant;
    if (geo.V == 1) {
        switch (geo.L) {
        case 1: return f(integral_constant<int, 1>{}, integral_constant<int, 1>{});
        case 2: return f(integral_constant<int, 2>{}, integral_constant<int, 1>{});
        case 4: return f(integral_constant<int, 4>{}, integral_constant<int, 1>{});
        case 8: return f(integral_constant<int, 8>{}, integral_constant<int, 1>{});
        case 16: return f(integral_constant<int, 16>{}, integral_constant<int, 1>{});
        case 32: return f(integral_constant<int, 32>{}, integral_constant<int, 1>{});
        case 64: return f(integral_constant<int, 64>{}, integral_constant<int, 1>{});
        case 128: return f(integral_constant<int, 128>{}, integral_constant<int, 1>{});
        case 256: return f(integral_constant<int, 256>{}, integral_constant<int, 1>{});
        case 512: return f(integral_constant<int, 512>{}, integral_constant<int, 1>{});
        case 1024: return f(integral_constant<int, 1024>{}, integral_constant<int, 1>{});
        default: return hipErrorInvalidValue;
        }
    }
    if (geo.L != 1024) return hipErrorInvalidValue;
    switch (geo.V) {
    case 2: return f(integral_constant<int, 1024>{}, integral_constant<int, 2>{});
    case 4: return f(integral_constant<int, 1024>{}, integral_constant<int, 4>{});
    default: return hipErrorInvalidValue;
    }
}

template <int L>
static inline unsigned chunk_block() { return L > 256 ? L : 256; }
template <int L>
static inline int64_t chunks_per_block() { return L >= 256 ? 1 : 256 / L; }

// Grid of the chunk-mapped elementwise kernels (see chunk_slot): bpc
// 256-thread workgroups per chunk of more than 1024 elements, else several
// chunks of lb lanes per workgroup.
int64_t chunk_slots(int chunk, int64_t nchunks, int &bpc, int &lb)
{
    const int lanes = (chunk + 3) / 4;
    if (lanes > 256) {
        bpc = (lanes + 255) / 256;
        lb = 256;
        return nchunks * bpc;
    }
    bpc = 1;
    lb = next_pow2(lanes);
    return (nchunks + (256 / lb) - 1) / (256 / lb);
}

hipError_t launch_local(bool var, int u_in, bool write_u, const void *g, float *m,
                        const float *x_src, float *x, float *v, float *u, const void *gbar,
                        int64_t n, const Scalars &s, int gt, const Chunks &ch, int64_t nchunks,
                        int chunk, const SrvCopy &sm, hipStream_t st)
{
    const int64_t n4 = n / 4;
    if (n4 == 0) return hipSuccess;
    if (!write_u && u_in != U_ZERO) return hipErrorInvalidValue;
    int bpc = 1, lb = 1;
    // U_ZERO: the chunk grid; otherwise one float4 per thread
    const int64_t blocks = u_in == U_ZERO ? chunk_slots(chunk, nchunks, bpc, lb) : grid_for(n4, 256);
    if (blocks == 0) return hipSuccess;
    const dim3 grid((unsigned)blocks), block(256);
    return with_grad_type(gt, [&](auto T) {
        constexpr int GT = decltype(T)::value;
        auto go = [&](auto kernel) {
            hipLaunchKernelGGL(kernel, grid, block, 0, st, g, m, x_src, x, v, u, gbar, n4, s, ch,
                               nchunks, bpc, lb, sm);
            return hipGetLastError();
        };
#define ZO_LOCAL(VAR_)                                                                        \
    switch (u_in * 2 + (write_u ? 1 : 0)) {                                                   \
    case U_MEM * 2 + 1: return go(k_local<VAR_, U_MEM, true, GT>);                            \
    case U_ZERO * 2 + 1: return go(k_local<VAR_, U_ZERO, true, GT>);                          \
    case U_ZERO * 2 + 0: return go(k_local<VAR_, U_ZERO, false, GT>);                         \
    case U_GM * 2 + 1: return go(k_local<VAR_, U_GM, true, GT>);                              \
    default: return hipErrorInvalidValue;                                                     \
    }
        if (var) {
            ZO_LOCAL(true)
        } else {
            ZO_LOCAL(false)
        }
#undef ZO_LOCAL
    });
}

// m = (bit ? S_c : -S_c) / Gamma from the server copy, over the chunk grid.
__global__ __launch_bounds__(256) void k_m_from_copy(float *__restrict__ m, Chunks ch,
                                                     int64_t nchunks, int bpc, int lb,
                                                     SrvCopy sm)
{
    int64_t c;
    int e;
    if (!chunk_slot(ch, nchunks, bpc, lb, c, e)) return;
    stnt(m, (ch.start[c] + e) >> 2, m_from_copy(sm, ch, c, e));
}

hipError_t launch_m_from_copy(float *m, const Chunks &ch, int64_t nchunks, int chunk,
                              const SrvCopy &sm, hipStream_t st)
{
    if (nchunks == 0) return hipSuccess;
    int bpc, lb;
    const int64_t blocks = chunk_slots(chunk, nchunks, bpc, lb);
    hipLaunchKernelGGL(k_m_from_copy, dim3((unsigned)blocks), dim3(256), 0, st, m, ch, nchunks,
                       bpc, lb, sm);
    return hipGetLastError();
}

// u = +0 + gamma_u * m, one float4 per thread.
__global__ __launch_bounds__(256) void k_u_from_m(float *__restrict__ u,
                                                  const float *__restrict__ m, int64_t n4,
                                                  float gamma_u)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n4) return;
    const f4v mm = ldnt(m, i);
    f4v r;
#pragma unroll
    for (int q = 0; q < 4; ++q) r[q] = 0.0f + gamma_u * mm[q];
    stnt(u, i, r);
}

hipError_t launch_u_from_m(float *u, const float *m, int64_t n, float gamma_u, hipStream_t st)
{
    const int64_t n4 = n / 4;
    if (n4 == 0) return hipSuccess;
    hipLaunchKernelGGL(k_u_from_m, dim3(grid_for(n4, 256)), dim3(256), 0, st, u, m, n4, gamma_u);
    return hipGetLastError();
}

hipError_t launch_zero(float *dst, int64_t n, hipStream_t st)
{
    const int64_t n4 = n / 4;
    if (n4 == 0) return hipSuccess;
    hipLaunchKernelGGL(k_zero, dim3(grid_for(n4, 256)), dim3(256), 0, st, dst, n4);
    return hipGetLastError();
}

hipError_t launch_var(float *v, const void *gbar, int64_t n, const Scalars &s, int gt,
                      hipStream_t st)
{
    const int64_t n4 = n / 4;
    if (n4 == 0) return hipSuccess;
    return with_grad_type(gt, [&](auto T) {
        constexpr int GT = decltype(T)::value;
        hipLaunchKernelGGL((k_var<GT>), dim3(grid_for(n4, 256)), dim3(256), 0, st, v, gbar, n4,
                           s);
        return hipGetLastError();
    });
}

hipError_t launch_sync1(Geometry geo, bool fused, int u_in, const void *g, const float *m,
                        const void *u, float *err, const Chunks &ch, int64_t nchunks,
                        uint64_t *packed, float *scales, const Scalars &s, int gt, int ut,
                        const SrvCopy &sm, hipStream_t st)
{
    if (nchunks == 0) return hipSuccess;
    if (u_in != U_MEM && !fused) return hipErrorInvalidValue;
    if (fused && ut != GT_F32) return hipErrorInvalidValue;
    return with_grad_type(fused ? gt : ut, [&](auto T) {
        constexpr int GT = decltype(T)::value;
        return with_geometry(geo, [&](auto Lc, auto Vc) {
            constexpr int L = decltype(Lc)::value, V = decltype(Vc)::value;
            const dim3 grid(grid_for(nchunks, chunks_per_block<L>())), block(chunk_block<L>());
            uint32_t *p32 = reinterpret_cast<uint32_t *>(packed);
            auto go = [&](auto kernel) {
                hipLaunchKernelGGL(kernel, grid, block, 0, st, g, m, u, err, ch, nchunks, p32,
                                   scales, s, sm);
                return hipGetLastError();
            };
            if (!fused) return go(k_sync1<L, V, false, U_MEM, GT>);
            switch (u_in) {
            case U_MEM: return go(k_sync1<L, V, true, U_MEM, GT>);
            case U_ZERO: return go(k_sync1<L, V, true, U_ZERO, GT>);
            case U_GM: return go(k_sync1<L, V, true, U_GM, GT>);
            default: return hipErrorInvalidValue;
            }
        });
    });
}

// Lanes per chunk and rounds of the LUT server: one lane per packed dword,
// up to 512 lanes per chunk.
static inline Geometry srv_geometry_for(int chunk)
{
    const int dws = (chunk + 31) / 32;
    if (dws <= 512) return Geometry{next_pow2(dws), 1};
    return Geometry{512, next_pow2((dws + 511) / 512)};
}

static constexpr size_t kSrvLdsMax = 96 * 1024;

template <int LD, int G>
static hipError_t go_srv_lut(const uint64_t *packed, const float *scales, int W, int64_t wstride,
                             int64_t cstride, const Chunks &ch, int64_t c0, int64_t nch,
                             int64_t word0, int64_t elem0, float *srv_err, uint64_t *srv_packed,
                             float *srv_scales, float *avg, uint8_t *flags, double inv_w,
                             int pow2, hipStream_t st)
{
    constexpr int CPW = srv_chunks_per_block(LD, G);
    hipLaunchKernelGGL((k_srv_lut<LD, G>), dim3(xcd_grid(grid_for(nch, CPW))), dim3(LD * CPW), 0, st,
                       reinterpret_cast<const uint32_t *>(packed), scales, W, wstride, cstride,
                       ch, c0, nch, word0, elem0, srv_err, reinterpret_cast<uint32_t *>(srv_packed),
                       srv_scales, avg, flags, inv_w, pow2);
    return hipGetLastError();
}

template <int G>
static hipError_t srv_lut_ld(int LD, const uint64_t *packed, const float *scales, int W,
                             int64_t wstride, int64_t cstride, const Chunks &ch, int64_t c0,
                             int64_t nch, int64_t word0, int64_t elem0, float *srv_err,
                             uint64_t *srv_packed, float *srv_scales, float *avg, uint8_t *flags,
                             double inv_w, int pow2, hipStream_t st)
{
#define ZO_SRV_LD(L)                                                                           \
    case L:                                                                                    \
        return go_srv_lut<L, G>(packed, scales, W, wstride, cstride, ch, c0, nch, word0, elem0, \
                                srv_err, srv_packed, srv_scales, avg, flags, inv_w, pow2, st);
    if constexpr ((G & (G - 1)) != 0) {
        // groups counted exactly only for chunks of at least 64 dwords
        switch (LD) {
            ZO_SRV_LD(64) ZO_SRV_LD(128) ZO_SRV_LD(256) ZO_SRV_LD(512)
        default: return hipErrorInvalidValue;
        }
    } else {
        switch (LD) {
            ZO_SRV_LD(1) ZO_SRV_LD(2) ZO_SRV_LD(4) ZO_SRV_LD(8) ZO_SRV_LD(16) ZO_SRV_LD(32)
            ZO_SRV_LD(64) ZO_SRV_LD(128) ZO_SRV_LD(256) ZO_SRV_LD(512)
        default: return hipErrorInvalidValue;
        }
    }
#undef ZO_SRV_LD
}

hipError_t launch_srv(Geometry geo, int algo, const uint64_t *packed, const float *scales, int W,
                      int64_t wstride, int64_t cstride, const Chunks &ch, int64_t c0,
                      int64_t nch, int64_t word0, int64_t elem0, float *srv_err,
                      uint64_t *srv_packed, float *srv_scales, float *avg, uint8_t *flags,
                      int chunk, hipStream_t st)
{
    if (nch == 0) return hipSuccess;
    const Geometry sg = srv_geometry_for(chunk);
    // worker groups of 8 (the last one may be partial); chunks of fewer than
    // 64 dwords round the count up to a power of two (fewer instantiations,
    // the extra groups' tables are zero)
    const int G = sg.L >= 64 ? (W + 7) / 8 : next_pow2((W + 7) / 8);
    const int cpw = srv_chunks_per_block(sg.L, G);
    const size_t tab = srv_nibble(sg.L) ? 0 : (size_t)cpw * G * 2048;
    const size_t xpose = (size_t)cpw * sg.L * 128;
    const size_t lds = (tab > xpose ? tab : xpose) + (size_t)cpw * G * 32 + (size_t)cpw * G * 256 + 256;
    const bool pow2 = (W & (W - 1)) == 0;
    const double inv_w = 1.0 / (double)W;
    const bool lut = algo != SRV_PLAIN && sg.V == 1 && G <= 16 && lds <= kSrvLdsMax;
    if (!lut) {
        return with_geometry(geo, [&](auto Lc, auto Vc) {
            constexpr int L = decltype(Lc)::value, V = decltype(Vc)::value;
            hipLaunchKernelGGL((k_srv_plain<L, V>), dim3(grid_for(nch, chunks_per_block<L>())),
                               dim3(chunk_block<L>()), 0, st,
                               reinterpret_cast<const uint32_t *>(packed), scales, W, wstride,
                               cstride, ch, c0, nch, word0, elem0, srv_err,
                               reinterpret_cast<uint32_t *>(srv_packed), srv_scales, avg, flags,
                               inv_w, pow2 ? 1 : 0);
            return hipGetLastError();
        });
    }
    switch (G) {
    case 1: return srv_lut_ld<1>(sg.L, packed, scales, W, wstride, cstride, ch, c0, nch, word0, elem0, srv_err, srv_packed, srv_scales, avg, flags, inv_w, pow2, st);
    case 2: return srv_lut_ld<2>(sg.L, packed, scales, W, wstride, cstride, ch, c0, nch, word0, elem0, srv_err, srv_packed, srv_scales, avg, flags, inv_w, pow2, st);
    case 3: return srv_lut_ld<3>(sg.L, packed, scales, W, wstride, cstride, ch, c0, nch, word0, elem0, srv_err, srv_packed, srv_scales, avg, flags, inv_w, pow2, st);
    case 4: return srv_lut_ld<4>(sg.L, packed, scales, W, wstride, cstride, ch, c0, nch, word0, elem0, srv_err, srv_packed, srv_scales, avg, flags, inv_w, pow2, st);
    case 5: return srv_lut_ld<5>(sg.L, packed, scales, W, wstride, cstride, ch, c0, nch, word0, elem0, srv_err, srv_packed, srv_scales, avg, flags, inv_w, pow2, st);
    case 6: return srv_lut_ld<6>(sg.L, packed, scales, W, wstride, cstride, ch, c0, nch, word0, elem0, srv_err, srv_packed, srv_scales, avg, flags, inv_w, pow2, st);
    case 7: return srv_lut_ld<7>(sg.L, packed, scales, W, wstride, cstride, ch, c0, nch, word0, elem0, srv_err, srv_packed, srv_scales, avg, flags, inv_w, pow2, st);
    case 8: return srv_lut_ld<8>(sg.L, packed, scales, W, wstride, cstride, ch, c0, nch, word0, elem0, srv_err, srv_packed, srv_scales, avg, flags, inv_w, pow2, st);
    case 9: return srv_lut_ld<9>(sg.L, packed, scales, W, wstride, cstride, ch, c0, nch, word0, elem0, srv_err, srv_packed, srv_scales, avg, flags, inv_w, pow2, st);
    case 10: return srv_lut_ld<10>(sg.L, packed, scales, W, wstride, cstride, ch, c0, nch, word0, elem0, srv_err, srv_packed, srv_scales, avg, flags, inv_w, pow2, st);
    case 11: return srv_lut_ld<11>(sg.L, packed, scales, W, wstride, cstride, ch, c0, nch, word0, elem0, srv_err, srv_packed, srv_scales, avg, flags, inv_w, pow2, st);
    case 12: return srv_lut_ld<12>(sg.L, packed, scales, W, wstride, cstride, ch, c0, nch, word0, elem0, srv_err, srv_packed, srv_scales, avg, flags, inv_w, pow2, st);
    case 13: return srv_lut_ld<13>(sg.L, packed, scales, W, wstride, cstride, ch, c0, nch, word0, elem0, srv_err, srv_packed, srv_scales, avg, flags, inv_w, pow2, st);
    case 14: return srv_lut_ld<14>(sg.L, packed, scales, W, wstride, cstride, ch, c0, nch, word0, elem0, srv_err, srv_packed, srv_scales, avg, flags, inv_w, pow2, st);
    case 15: return srv_lut_ld<15>(sg.L, packed, scales, W, wstride, cstride, ch, c0, nch, word0, elem0, srv_err, srv_packed, srv_scales, avg, flags, inv_w, pow2, st);
    case 16: return srv_lut_ld<16>(sg.L, packed, scales, W, wstride, cstride, ch, c0, nch, word0, elem0, srv_err, srv_packed, srv_scales, avg, flags, inv_w, pow2, st);
    default: return hipErrorInvalidValue;
    }
}


hipError_t launch_fv_full(const void *gbar, float *x, float *m, float *v, int64_t n,
                          const Scalars &s, int gt, hipStream_t st)
{
    const int64_t n4 = n / 4;
    if (n4 == 0) return hipSuccess;
    return with_grad_type(gt, [&](auto T) {
        constexpr int GT = decltype(T)::value;
        hipLaunchKernelGGL((k_fv_full<GT>), dim3(grid_for(n4, 256)), dim3(256), 0, st, gbar, x, m,
                           v, n4, s);
        return hipGetLastError();
    });
}

hipError_t launch_fv_apply(const uint64_t *srv_packed, const float *srv_scales, const Chunks &ch,
                           int64_t nchunks, float *x, float *m, const float *v, const Scalars &s,
                           int chunk, hipStream_t st)
{
    if (nchunks == 0) return hipSuccess;
    int bpc, lb;
    const int64_t grid = chunk_slots(chunk, nchunks, bpc, lb);
    hipLaunchKernelGGL(k_fv_apply, dim3((unsigned)grid), dim3(256), 0, st,
                       reinterpret_cast<const uint32_t *>(srv_packed), srv_scales, ch, nchunks,
                       bpc, lb, x, m, v, s);
    return hipGetLastError();
}

hipError_t launch_recon(Geometry geo, bool var, bool defer, const uint64_t *srv_packed,
                        const float *srv_scales, const Chunks &ch, int64_t nchunks, float *m,
                        float *x, float *v, float *u, float *anchor, const void *gbar,
                        float gsum, const Scalars &s, int gt, int chunk, const SrvCopy &sm,
                        hipStream_t st)
{
    (void)geo;
    if (nchunks == 0) return hipSuccess;
    int bpc, lb;
    const int64_t grid = chunk_slots(chunk, nchunks, bpc, lb);
    const uint32_t *p32 = reinterpret_cast<const uint32_t *>(srv_packed);
    const dim3 g3((unsigned)grid), b3(256);
    return with_grad_type(gt, [&](auto T) {
        constexpr int GT = decltype(T)::value;
        if (var && defer)
            hipLaunchKernelGGL((k_recon<true, true, GT>), g3, b3, 0, st, p32, srv_scales, ch,
                               nchunks, bpc, lb, m, x, v, u, anchor, gbar, gsum, s, sm);
        else if (var)
            hipLaunchKernelGGL((k_recon<true, false, GT>), g3, b3, 0, st, p32, srv_scales, ch,
                               nchunks, bpc, lb, m, x, v, u, anchor, gbar, gsum, s, sm);
        else if (defer)
            hipLaunchKernelGGL((k_recon<false, true, GT>), g3, b3, 0, st, p32, srv_scales, ch,
                               nchunks, bpc, lb, m, x, v, u, anchor, gbar, gsum, s, sm);
        else
            hipLaunchKernelGGL((k_recon<false, false, GT>), g3, b3, 0, st, p32, srv_scales, ch,
                               nchunks, bpc, lb, m, x, v, u, anchor, gbar, gsum, s, sm);
        return hipGetLastError();
    });
}

template <int R>
static hipError_t stream_r(int S, const StreamPtrs &p, int64_t n4, hipStream_t st)
{
    const dim3 grid(grid_for(n4, 256)), block(256);
    switch (S) {
    case 1: hipLaunchKernelGGL((k_stream<R, 1>), grid, block, 0, st, p, n4); break;
    case 2: hipLaunchKernelGGL((k_stream<R, 2>), grid, block, 0, st, p, n4); break;
    case 3: hipLaunchKernelGGL((k_stream<R, 3>), grid, block, 0, st, p, n4); break;
    case 4: hipLaunchKernelGGL((k_stream<R, 4>), grid, block, 0, st, p, n4); break;
    case 5: hipLaunchKernelGGL((k_stream<R, 5>), grid, block, 0, st, p, n4); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_stream(int R, int S, const StreamPtrs &p, int64_t n, hipStream_t st)
{
    const int64_t n4 = n / 4;
    if (n4 == 0) return hipSuccess;
    switch (R) {
    case 1: return stream_r<1>(S, p, n4, st);
    case 2: return stream_r<2>(S, p, n4, st);
    case 3: return stream_r<3>(S, p, n4, st);
    case 4: return stream_r<4>(S, p, n4, st);
    case 5: return stream_r<5>(S, p, n4, st);
    case 6: return stream_r<6>(S, p, n4, st);
    default: return hipErrorInvalidValue;
    }
}

hipError_t launch_srv_pattern(int chunk, const uint64_t *packed, int W, int64_t wstride,
                              const Chunks &ch, int64_t c0, int64_t nch, int64_t word0,
                              int64_t elem0, float *srv_err, hipStream_t st)
{
    const Geometry sg = srv_geometry_for(chunk);
    if (sg.V != 1 || sg.L < 64) return hipErrorInvalidValue;
    if (nch == 0) return hipSuccess;
    const dim3 grid(xcd_grid(grid_for(nch, 1)));
    const uint32_t *p = reinterpret_cast<const uint32_t *>(packed);
    switch (sg.L) {
    case 64: hipLaunchKernelGGL(k_srv_pattern<64>, grid, dim3(64), 0, st, p, W, wstride, ch, c0, nch, word0, elem0, srv_err); break;
    case 128: hipLaunchKernelGGL(k_srv_pattern<128>, grid, dim3(128), 0, st, p, W, wstride, ch, c0, nch, word0, elem0, srv_err); break;
    case 256: hipLaunchKernelGGL(k_srv_pattern<256>, grid, dim3(256), 0, st, p, W, wstride, ch, c0, nch, word0, elem0, srv_err); break;
    case 512: hipLaunchKernelGGL(k_srv_pattern<512>, grid, dim3(512), 0, st, p, W, wstride, ch, c0, nch, word0, elem0, srv_err); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_copy(const float *src, float *dst, int64_t n, bool nt, hipStream_t st)
{
    const int64_t n4 = n / 4;
    if (n4 == 0) return hipSuccess;
    if (nt)
        hipLaunchKernelGGL(k_copy<true>, dim3(grid_for(n4, 256)), dim3(256), 0, st, src, dst, n4);
    else
        hipLaunchKernelGGL(k_copy<false>, dim3(grid_for(n4, 256)), dim3(256), 0, st, src, dst, n4);
    return hipGetLastError();
}

hipError_t launch_divsqrt(const float *a, const float *b, float *q, float *r, int64_t n,
                          hipStream_t st)
{
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_divsqrt, dim3(grid_for(n, 256)), dim3(256), 0, st, a, b, q, r, n);
    return hipGetLastError();
}

}  // namespace zo
