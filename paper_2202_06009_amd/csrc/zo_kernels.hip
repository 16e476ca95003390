// zo_kernels.hip -- gfx950 kernels of the 0/1 Adam hot path.
//
// Paper: Lu et al., "Maximizing Communication Efficiency for Large-scale
// Training via 0/1 Adam" (arXiv 2202.06009): Algorithm 1 (0/1 Adam),
// Algorithm 2 (error-feedback 1bit-AllReduce), Equation 3 (1-bit compressor).
//
// Every kernel is HBM-streaming: no contraction, so no MFMA.  Arithmetic is
// binary32 with one rounding per operation (the library is built with
// -ffp-contract=off; division and sqrtf are the correctly rounded lowerings),
// so results are reproducible bit for bit by any implementation that follows
// the same operation order.
//
// Data layout
//   * state vectors are flat float[n], n a multiple of 4, accessed as float4;
//   * chunk kernels map one chunk onto L lanes (L a power of two <= 256) of a
//     256-thread workgroup; lane lc of the chunk holds, for each block k < V,
//     the four elements 4*L*k + 4*lc + {0,1,2,3}.  A block of 4L elements is
//     therefore one contiguous, coalesced 16*L-byte span per buffer;
//   * per-chunk L1 norm: in-lane (|a0|+|a1|)+(|a2|+|a3|), then an xor
//     butterfly over the lanes of a wave (pairs partner lanes l and l^o, i.e.
//     adjacent index ranges), then an in-order tree over the chunk's waves and
//     over its blocks.  That is exactly the balanced pairwise tree over the
//     chunk in index order; the zero padding beyond the chunk length adds +0
//     and changes no bit;
//   * packed signs: dword j of a chunk's words holds elements 32j..32j+31,
//     assembled by an OR butterfly over 8 lanes (4 bits per lane) and stored
//     by every 8th lane.
#include <hip/hip_runtime.h>
#include <stdint.h>
#include <type_traits>

#include "zo_internal.h"

namespace zo {

// ---------------------------------------------------------------------------
// elementwise helpers
// ---------------------------------------------------------------------------

__device__ __forceinline__ float4 ld4(const float *p, int64_t i4)
{
    return reinterpret_cast<const float4 *>(p)[i4];
}

__device__ __forceinline__ void st4(float *p, int64_t i4, float4 v)
{
    reinterpret_cast<float4 *>(p)[i4] = v;
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
// a1 (+a2): local step, grid-stride over float4
// ---------------------------------------------------------------------------

template <bool VAR>
__global__ __launch_bounds__(256) void k_local(const float *__restrict__ g, float *__restrict__ m,
                                               float *__restrict__ x, float *__restrict__ v,
                                               float *__restrict__ u,
                                               const float *__restrict__ gbar, int64_t n4,
                                               Scalars s)
{
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride) {
        float4 gg = ld4(g, i), mm = ld4(m, i), xx = ld4(x, i), vv = ld4(v, i), uu = ld4(u, i);
        local_elem(gg.x, mm.x, xx.x, vv.x, uu.x, s);
        local_elem(gg.y, mm.y, xx.y, vv.y, uu.y, s);
        local_elem(gg.z, mm.z, xx.z, vv.z, uu.z, s);
        local_elem(gg.w, mm.w, xx.w, vv.w, uu.w, s);
        st4(m, i, mm);
        st4(x, i, xx);
        st4(u, i, uu);
        if (VAR) {
            float4 gb = ld4(gbar, i);
            vv.x = var_elem(vv.x, gb.x, s);
            vv.y = var_elem(vv.y, gb.y, s);
            vv.z = var_elem(vv.z, gb.z, s);
            vv.w = var_elem(vv.w, gb.w, s);
            st4(v, i, vv);
        }
    }
}

// a2 standalone.
__global__ __launch_bounds__(256) void k_var(float *__restrict__ v, const float *__restrict__ gbar,
                                             int64_t n4, Scalars s)
{
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride) {
        float4 vv = ld4(v, i), gb = ld4(gbar, i);
        vv.x = var_elem(vv.x, gb.x, s);
        vv.y = var_elem(vv.y, gb.y, s);
        vv.z = var_elem(vv.z, gb.z, s);
        vv.w = var_elem(vv.w, gb.w, s);
        st4(v, i, vv);
    }
}

// ---------------------------------------------------------------------------
// chunk machinery
// ---------------------------------------------------------------------------

// Sum over the L lanes of a chunk that share a wave (L <= 64): xor butterfly.
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

// The chunk's pairwise L1 tree, given each lane's per-block partial sums
// (the in-lane level).  Returns the total to every lane of the chunk.  All
// threads of the workgroup must call it (it synchronises when L > 64).
template <int L, int V>
__device__ __forceinline__ float chunk_tree(float (&part)[V], float *lds)
{
#pragma unroll
    for (int k = 0; k < V; ++k) part[k] = wave_tree<L>(part[k]);
    if constexpr (L <= 64) {
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
            if constexpr (NW == 2) {
                bs[k] = lds[base * V + k] + lds[(base + 1) * V + k];
            } else {
                bs[k] = (lds[base * V + k] + lds[(base + 1) * V + k]) +
                        (lds[(base + 2) * V + k] + lds[(base + 3) * V + k]);
            }
        }
#pragma unroll
        for (int w = 1; w < V; w <<= 1) {
#pragma unroll
            for (int k = 0; k + w < V; k += 2 * w) bs[k] = bs[k] + bs[k + w];
        }
        return bs[0];
    }
}

__device__ __forceinline__ float abs4(float4 a)
{
    return (fabsf(a.x) + fabsf(a.y)) + (fabsf(a.z) + fabsf(a.w));
}

__device__ __forceinline__ uint32_t sign4(float4 a)
{
    return (a.x >= 0.0f ? 1u : 0u) | (a.y >= 0.0f ? 2u : 0u) | (a.z >= 0.0f ? 4u : 0u) |
           (a.w >= 0.0f ? 8u : 0u);
}

__device__ __forceinline__ float ef_elem(float a, float s)
{
    return a >= 0.0f ? a - s : a + s;
}

// Equation 3 with error feedback on one chunk whose values `a` are in the
// lanes' registers (zeros beyond `len`): writes the new error, the packed
// signs (all 2*ceil(len/64) dwords of the chunk) and the scale.
template <int L, int V>
__device__ __forceinline__ void compress_chunk(float4 (&a)[V], int lc, int len, bool active,
                                               float *__restrict__ err, int64_t err_e0,
                                               uint32_t *__restrict__ words32, float *scale_out,
                                               float *lds)
{
    float part[V];
#pragma unroll
    for (int k = 0; k < V; ++k) part[k] = abs4(a[k]);
    const float tot = chunk_tree<L, V>(part, lds);
    const float s = tot / (float)len;
    const int ndw = 2 * ((len + 63) >> 6);
#pragma unroll
    for (int k = 0; k < V; ++k) {
        const int e = 4 * L * k + 4 * lc;
        const bool valid = active && e < len;
        uint32_t nib = 0;
        if (valid) {
            float4 d;
            d.x = ef_elem(a[k].x, s);
            d.y = ef_elem(a[k].y, s);
            d.z = ef_elem(a[k].z, s);
            d.w = ef_elem(a[k].w, s);
            st4(err, (err_e0 + e) >> 2, d);
            nib = sign4(a[k]);
        }
        uint32_t dw = wave_or8<L>(nib << (4 * (lc & 7)));
        if (active && (lc & 7) == 0) {
            const int j = e >> 5;
            if (j < ndw) words32[j] = dw;
            if (L <= 8 && ndw > 1) words32[1] = 0u;
        }
    }
    if (active && lc == 0) *scale_out = s;
}

// ---------------------------------------------------------------------------
// a3: worker compress + error feedback + pack (fused with the momentum and
// buffer lines when g != nullptr)
// ---------------------------------------------------------------------------

template <int L, int V, bool FUSED>
__global__ __launch_bounds__(256) void k_sync1(const float *__restrict__ g,
                                               const float *__restrict__ m,
                                               const float *__restrict__ u,
                                               float *__restrict__ err, Chunks ch,
                                               int64_t nchunks, uint32_t *__restrict__ packed32,
                                               float *__restrict__ scales, Scalars s)
{
    __shared__ float lds[64];
    constexpr int CPW = 256 / L;
    const int lc = threadIdx.x % L;
    const int64_t c = (int64_t)blockIdx.x * CPW + threadIdx.x / L;
    const bool active = c < nchunks;
    const int len = active ? ch.len[c] : 0;
    const int64_t e0 = active ? ch.start[c] : 0;
    float4 a[V];
#pragma unroll
    for (int k = 0; k < V; ++k) {
        const int e = 4 * L * k + 4 * lc;
        a[k] = make_float4(0.f, 0.f, 0.f, 0.f);
        if (e < len) {
            const int64_t i4 = (e0 + e) >> 2;
            float4 uu = ld4(u, i4), dd = ld4(err, i4);
            if (FUSED) {
                float4 gg = ld4(g, i4), mm = ld4(m, i4);
                uu.x = uu.x + s.gamma * (s.b1 * mm.x + s.c1 * gg.x);
                uu.y = uu.y + s.gamma * (s.b1 * mm.y + s.c1 * gg.y);
                uu.z = uu.z + s.gamma * (s.b1 * mm.z + s.c1 * gg.z);
                uu.w = uu.w + s.gamma * (s.b1 * mm.w + s.c1 * gg.w);
            }
            a[k].x = uu.x + dd.x;
            a[k].y = uu.y + dd.y;
            a[k].z = uu.z + dd.z;
            a[k].w = uu.w + dd.w;
        }
    }
    compress_chunk<L, V>(a, lc, len, active, err, e0, packed32 + 2 * (active ? ch.word[c] : 0),
                         scales + (active ? c : 0), lds);
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
template <int L, int V>
__global__ __launch_bounds__(256) void k_srv_plain(const uint32_t *__restrict__ packed32,
                                                   const float *__restrict__ scales, int W,
                                                   int64_t wstride, int64_t cstride,
                                                   Chunks ch, int64_t c0, int64_t nch,
                                                   int64_t word0, int64_t elem0,
                                                   float *__restrict__ srv_err,
                                                   uint32_t *__restrict__ srv_packed32,
                                                   float *__restrict__ srv_scales,
                                                   float *__restrict__ avg_out,
                                                   uint8_t *__restrict__ flags)
{
    __shared__ float lds[64];
    constexpr int CPW = 256 / L;
    const int lc = threadIdx.x % L;
    const int64_t cr = (int64_t)blockIdx.x * CPW + threadIdx.x / L;  // chunk within range
    const bool active = cr < nch;
    const int64_t c = c0 + (active ? cr : 0);
    const int len = active ? ch.len[c] : 0;
    const int64_t el = active ? ch.start[c] - elem0 : 0;      // element offset in range
    const int64_t wd = active ? ch.word[c] - word0 : 0;       // word offset in range
    float4 b[V];
#pragma unroll
    for (int k = 0; k < V; ++k) {
        const int e = 4 * L * k + 4 * lc;
        b[k] = make_float4(0.f, 0.f, 0.f, 0.f);
        if (e < len) {
            double acc0 = 0.0, acc1 = 0.0, acc2 = 0.0, acc3 = 0.0;
            const int64_t dwi = 2 * wd + (e >> 5);
            const int sh = e & 31;
            for (int w = 0; w < W; ++w) {
                const uint32_t bits = packed32[2 * wstride * w + dwi] >> sh;
                const double sw = (double)scales[cstride * w + cr];
                acc0 += (bits & 1u) ? sw : -sw;
                acc1 += (bits & 2u) ? sw : -sw;
                acc2 += (bits & 4u) ? sw : -sw;
                acc3 += (bits & 8u) ? sw : -sw;
            }
            float4 av;
            av.x = (float)(acc0 / (double)W);
            av.y = (float)(acc1 / (double)W);
            av.z = (float)(acc2 / (double)W);
            av.w = (float)(acc3 / (double)W);
            if (avg_out) st4(avg_out, (el + e) >> 2, av);
            float4 d = ld4(srv_err, (el + e) >> 2);
            b[k].x = av.x + d.x;
            b[k].y = av.y + d.y;
            b[k].z = av.z + d.z;
            b[k].w = av.w + d.w;
        }
    }
    compress_chunk<L, V>(b, lc, len, active, srv_err, el,
                         srv_packed32 + 2 * (active ? ch.word[c] : 0), srv_scales + c, lds);
    const uint32_t f = inexact_flag<L>(scales + (active ? cr : 0), cstride, W, lc);
    if (active && lc == 0) flags[cr] = (uint8_t)f;
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
__device__ __forceinline__ void transpose8x32(uint32_t (&x)[8])
{
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        uint32_t t = ((x[k] >> 4) ^ x[k + 4]) & 0x0F0F0F0Fu;
        x[k + 4] ^= t;
        x[k] ^= t << 4;
    }
#pragma unroll
    for (int k = 0; k < 8; k += (k & 1) ? 3 : 1) {   // pairs (0,2) (1,3) (4,6) (5,7)
        uint32_t t = ((x[k] >> 2) ^ x[k + 2]) & 0x33333333u;
        x[k + 2] ^= t;
        x[k] ^= t << 2;
    }
#pragma unroll
    for (int k = 0; k < 8; k += 2) {
        uint32_t t = ((x[k] >> 1) ^ x[k + 1]) & 0x55555555u;
        x[k + 1] ^= t;
        x[k] ^= t << 1;
    }
}

// In-lane pairwise tree of |v[0..32)| in index order.
__device__ __forceinline__ float tree32_abs(const float (&v)[32])
{
    float t[32];
#pragma unroll
    for (int i = 0; i < 32; ++i) t[i] = fabsf(v[i]);
#pragma unroll
    for (int w = 1; w < 32; w <<= 1) {
#pragma unroll
        for (int i = 0; i + w < 32; i += 2 * w) t[i] = t[i] + t[i + w];
    }
    return t[0];
}

template <int LD, int R>
__global__ __launch_bounds__(256) void k_srv_lut(const uint32_t *__restrict__ packed32,
                                                 const float *__restrict__ scales, int W, int G,
                                                 int64_t wstride, int64_t cstride, Chunks ch,
                                                 int64_t c0, int64_t nch, int64_t word0,
                                                 int64_t elem0, float *__restrict__ srv_err,
                                                 uint32_t *__restrict__ srv_packed32,
                                                 float *__restrict__ srv_scales,
                                                 float *__restrict__ avg_out,
                                                 uint8_t *__restrict__ flags, int cpw,
                                                 double inv_w, int w_pow2)
{
    extern __shared__ double dyn_lds[];
    double *tab = dyn_lds;                                   // [cpw][G][256]
    float *sc = reinterpret_cast<float *>(tab + (size_t)cpw * G * 256);  // [cpw][W]
    float *tree = sc + (((size_t)cpw * W + 3) & ~(size_t)3); // [64]

    const int q = threadIdx.x / LD, lc = threadIdx.x % LD;
    const int64_t cbase = (int64_t)blockIdx.x * cpw;
    const int64_t cr = cbase + q;
    const bool active = cr < nch;
    const int64_t c = c0 + (active ? cr : 0);
    const int len = active ? ch.len[c] : 0;
    const int64_t el = active ? ch.start[c] - elem0 : 0;
    const int64_t wd = active ? ch.word[c] - word0 : 0;

    // stage the scales of the workgroup's chunks, then build the tables
    for (int i = threadIdx.x; i < cpw * W; i += blockDim.x) {
        const int qq = i / W, w = i - qq * W;
        sc[i] = (cbase + qq < nch) ? scales[cstride * w + cbase + qq] : 0.0f;
    }
    __syncthreads();
    for (int i = threadIdx.x; i < cpw * G * 256; i += blockDim.x) {
        const int qq = i / (G * 256), g = (i >> 8) % G, b = i & 255;
        double t = 0.0;
#pragma unroll
        for (int k = 0; k < 8; ++k) {
            const int w = 8 * g + k;
            if (w < W) {
                const double sw = (double)sc[qq * W + w];
                t += ((b >> k) & 1) ? sw : -sw;
            }
        }
        tab[i] = t;
    }
    __syncthreads();
    const double *mytab = tab + (size_t)q * G * 256;

    const int ndw_data = (len + 31) >> 5;
    float bv[R][32];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int j = r * LD + lc;
        double acc[32];
#pragma unroll
        for (int i = 0; i < 32; ++i) acc[i] = 0.0;
        if (j < ndw_data) {
            const uint32_t *src = packed32 + 2 * wd + j;
            const int64_t ws = 2 * wstride;
            for (int g = 0; g < G; ++g) {
                uint32_t x[8];
#pragma unroll
                for (int k = 0; k < 8; ++k) {
                    const int w = 8 * g + k;
                    x[k] = (w < W) ? src[ws * w] : 0u;
                }
                transpose8x32(x);
                const double *tg = mytab + g * 256;
#pragma unroll
                for (int cc = 0; cc < 4; ++cc) {
#pragma unroll
                    for (int k = 0; k < 8; ++k) acc[8 * cc + k] += tg[(x[k] >> (8 * cc)) & 0xFFu];
                }
            }
        }
#pragma unroll
        for (int i4 = 0; i4 < 8; ++i4) {
            const int e = 32 * j + 4 * i4;
            if (e < len) {
                float4 av;
                if (w_pow2) {
                    av.x = (float)(acc[4 * i4 + 0] * inv_w);
                    av.y = (float)(acc[4 * i4 + 1] * inv_w);
                    av.z = (float)(acc[4 * i4 + 2] * inv_w);
                    av.w = (float)(acc[4 * i4 + 3] * inv_w);
                } else {
                    av.x = (float)(acc[4 * i4 + 0] / (double)W);
                    av.y = (float)(acc[4 * i4 + 1] / (double)W);
                    av.z = (float)(acc[4 * i4 + 2] / (double)W);
                    av.w = (float)(acc[4 * i4 + 3] / (double)W);
                }
                if (avg_out) st4(avg_out, (el + e) >> 2, av);
                const float4 d = ld4(srv_err, (el + e) >> 2);
                bv[r][4 * i4 + 0] = av.x + d.x;
                bv[r][4 * i4 + 1] = av.y + d.y;
                bv[r][4 * i4 + 2] = av.z + d.z;
                bv[r][4 * i4 + 3] = av.w + d.w;
            } else {
#pragma unroll
                for (int i = 0; i < 4; ++i) bv[r][4 * i4 + i] = 0.0f;
            }
        }
    }

    // Equation 3 with the server error, in the same lane layout
    float part[R];
#pragma unroll
    for (int r = 0; r < R; ++r) part[r] = tree32_abs(bv[r]);
    const float tot = chunk_tree<LD, R>(part, tree);
    const float s = tot / (float)len;
    const int ndw = 2 * ((len + 63) >> 6);
    uint32_t *dst = srv_packed32 + 2 * (active ? ch.word[c] : 0);
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int j = r * LD + lc;
        uint32_t bits = 0;
#pragma unroll
        for (int i4 = 0; i4 < 8; ++i4) {
            const int e = 32 * j + 4 * i4;
            if (active && e < len) {
                float4 bb = make_float4(bv[r][4 * i4], bv[r][4 * i4 + 1], bv[r][4 * i4 + 2],
                                        bv[r][4 * i4 + 3]);
                float4 d;
                d.x = ef_elem(bb.x, s);
                d.y = ef_elem(bb.y, s);
                d.z = ef_elem(bb.z, s);
                d.w = ef_elem(bb.w, s);
                st4(srv_err, (el + e) >> 2, d);
                bits |= sign4(bb) << (4 * i4);
            }
        }
        if (active && j < ndw) dst[j] = bits;
    }
    if (LD * R == 1 && active && ndw > 1) dst[1] = 0u;
    if (active && lc == 0) srv_scales[c] = s;
    const uint32_t f = inexact_flag<LD>(scales + (active ? cr : 0), cstride, W, lc);
    if (active && lc == 0) flags[cr] = (uint8_t)f;
}

// ---------------------------------------------------------------------------
// a5 (+a2): reconstruct momentum and model from the server's compressed
// average; reset the buffer; move the anchor
// ---------------------------------------------------------------------------

template <int L, int V, bool VAR>
__global__ __launch_bounds__(256) void k_recon(const uint32_t *__restrict__ srv_packed32,
                                               const float *__restrict__ srv_scales, Chunks ch,
                                               int64_t nchunks, float *__restrict__ m,
                                               float *__restrict__ x, float *__restrict__ v,
                                               float *__restrict__ u,
                                               float *__restrict__ anchor,
                                               const float *__restrict__ gbar, float gsum,
                                               Scalars s)
{
    constexpr int CPW = 256 / L;
    const int lc = threadIdx.x % L;
    const int64_t c = (int64_t)blockIdx.x * CPW + threadIdx.x / L;
    if (c >= nchunks) return;
    const int len = ch.len[c];
    const int64_t e0 = ch.start[c];
    const float sc = srv_scales[c];
    const uint32_t *wp = srv_packed32 + 2 * ch.word[c];
#pragma unroll
    for (int k = 0; k < V; ++k) {
        const int e = 4 * L * k + 4 * lc;
        if (e < len) {
            const int64_t i4 = (e0 + e) >> 2;
            const uint32_t bits = wp[e >> 5] >> (e & 31);
            float4 ub;
            ub.x = (bits & 1u) ? sc : -sc;
            ub.y = (bits & 2u) ? sc : -sc;
            ub.z = (bits & 4u) ? sc : -sc;
            ub.w = (bits & 8u) ? sc : -sc;
            float4 vv = ld4(v, i4), an = ld4(anchor, i4);
            float4 mm, xx;
            mm.x = ub.x / gsum;
            mm.y = ub.y / gsum;
            mm.z = ub.z / gsum;
            mm.w = ub.w / gsum;
            xx.x = an.x - ub.x / sqrtf(vv.x + s.eps);
            xx.y = an.y - ub.y / sqrtf(vv.y + s.eps);
            xx.z = an.z - ub.z / sqrtf(vv.z + s.eps);
            xx.w = an.w - ub.w / sqrtf(vv.w + s.eps);
            st4(m, i4, mm);
            st4(x, i4, xx);
            st4(anchor, i4, xx);
            st4(u, i4, make_float4(0.f, 0.f, 0.f, 0.f));
            if (VAR) {
                float4 gb = ld4(gbar, i4);
                vv.x = var_elem(vv.x, gb.x, s);
                vv.y = var_elem(vv.y, gb.y, s);
                vv.z = var_elem(vv.z, gb.z, s);
                vv.w = var_elem(vv.w, gb.w, s);
                st4(v, i4, vv);
            }
        }
    }
}

}  // namespace zo

// ---------------------------------------------------------------------------
// diagnostic: the division and square root the kernels use
// ---------------------------------------------------------------------------

namespace zo {

__global__ __launch_bounds__(256) void k_divsqrt(const float *__restrict__ a,
                                                 const float *__restrict__ b,
                                                 float *__restrict__ q, float *__restrict__ r,
                                                 int64_t n)
{
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
        q[i] = a[i] / b[i];
        r[i] = sqrtf(a[i]);
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

Geometry geometry_for(int chunk)
{
    const int lanes = (chunk + 3) / 4;
    if (lanes <= 256) return Geometry{next_pow2(lanes), 1};
    return Geometry{256, next_pow2((lanes + 255) / 256)};
}

static inline unsigned stream_grid(int64_t n4)
{
    int64_t blocks = (n4 + 255) / 256;
    const int64_t cap = 256 * 64;  // 64 workgroups per CU, then grid-stride
    if (blocks > cap) blocks = cap;
    return (unsigned)(blocks < 1 ? 1 : blocks);
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
        default: return hipErrorInvalidValue;
        }
    }
    if (geo.L != 256) return hipErrorInvalidValue;
    switch (geo.V) {
    case 2: return f(integral_constant<int, 256>{}, integral_constant<int, 2>{});
    case 4: return f(integral_constant<int, 256>{}, integral_constant<int, 4>{});
    case 8: return f(integral_constant<int, 256>{}, integral_constant<int, 8>{});
    case 16: return f(integral_constant<int, 256>{}, integral_constant<int, 16>{});
    default: return hipErrorInvalidValue;
    }
}

hipError_t launch_local(bool var, const float *g, float *m, float *x, float *v, float *u,
                        const float *gbar, int64_t n, const Scalars &s, hipStream_t st)
{
    const int64_t n4 = n / 4;
    if (n4 == 0) return hipSuccess;
    if (var)
        hipLaunchKernelGGL(k_local<true>, dim3(stream_grid(n4)), dim3(256), 0, st, g, m, x, v, u,
                           gbar, n4, s);
    else
        hipLaunchKernelGGL(k_local<false>, dim3(stream_grid(n4)), dim3(256), 0, st, g, m, x, v,
                           u, gbar, n4, s);
    return hipGetLastError();
}

hipError_t launch_var(float *v, const float *gbar, int64_t n, const Scalars &s, hipStream_t st)
{
    const int64_t n4 = n / 4;
    if (n4 == 0) return hipSuccess;
    hipLaunchKernelGGL(k_var, dim3(stream_grid(n4)), dim3(256), 0, st, v, gbar, n4, s);
    return hipGetLastError();
}

hipError_t launch_sync1(Geometry geo, bool fused, const float *g, const float *m, const float *u,
                        float *err, const Chunks &ch, int64_t nchunks, uint64_t *packed,
                        float *scales, const Scalars &s, hipStream_t st)
{
    if (nchunks == 0) return hipSuccess;
    return with_geometry(geo, [&](auto Lc, auto Vc) {
        constexpr int L = decltype(Lc)::value, V = decltype(Vc)::value;
        const unsigned grid = (unsigned)((nchunks + (256 / L) - 1) / (256 / L));
        uint32_t *p32 = reinterpret_cast<uint32_t *>(packed);
        if (fused)
            hipLaunchKernelGGL((k_sync1<L, V, true>), dim3(grid), dim3(256), 0, st, g, m, u, err,
                               ch, nchunks, p32, scales, s);
        else
            hipLaunchKernelGGL((k_sync1<L, V, false>), dim3(grid), dim3(256), 0, st, g, m, u,
                               err, ch, nchunks, p32, scales, s);
        return hipGetLastError();
    });
}

// Lanes per chunk and rounds of the LUT server: one lane per packed dword.
static inline Geometry srv_geometry_for(int chunk)
{
    const int dws = (chunk + 31) / 32;
    if (dws <= 256) return Geometry{next_pow2(dws), 1};
    return Geometry{256, next_pow2((dws + 255) / 256)};
}

static constexpr size_t kSrvLdsMax = 64 * 1024;

hipError_t launch_srv(Geometry geo, int algo, const uint64_t *packed, const float *scales, int W,
                      int64_t wstride, int64_t cstride, const Chunks &ch, int64_t c0,
                      int64_t nch, int64_t word0, int64_t elem0, float *srv_err,
                      uint64_t *srv_packed, float *srv_scales, float *avg, uint8_t *flags,
                      int chunk, hipStream_t st)
{
    if (nch == 0) return hipSuccess;
    const int G = (W + 7) / 8;
    const size_t per_chunk = (size_t)G * 256 * 8 + (size_t)W * 4 + 16;
    const Geometry sg = srv_geometry_for(chunk);
    const bool lut = algo != SRV_PLAIN && sg.V <= 2 && per_chunk + 256 <= kSrvLdsMax;
    if (!lut) {
        return with_geometry(geo, [&](auto Lc, auto Vc) {
            constexpr int L = decltype(Lc)::value, V = decltype(Vc)::value;
            const unsigned grid = (unsigned)((nch + (256 / L) - 1) / (256 / L));
            hipLaunchKernelGGL((k_srv_plain<L, V>), dim3(grid), dim3(256), 0, st,
                               reinterpret_cast<const uint32_t *>(packed), scales, W, wstride,
                               cstride, ch, c0, nch, word0, elem0, srv_err,
                               reinterpret_cast<uint32_t *>(srv_packed), srv_scales, avg, flags);
            return hipGetLastError();
        });
    }
    int cpw = 256 / sg.L;
    while (cpw > 1 && (size_t)cpw * per_chunk + 256 > kSrvLdsMax) cpw >>= 1;
    const size_t lds = (size_t)cpw * ((size_t)G * 256 * 8) + (((size_t)cpw * W + 3) & ~(size_t)3) * 4 +
                       64 * 4;
    const bool pow2 = (W & (W - 1)) == 0;
    const double inv_w = 1.0 / (double)W;
    const unsigned grid = (unsigned)((nch + cpw - 1) / cpw);
    const unsigned block = (unsigned)(sg.L * cpw);
    auto go = [&](auto Lc, auto Rc) {
        constexpr int L = decltype(Lc)::value, Rr = decltype(Rc)::value;
        hipLaunchKernelGGL((k_srv_lut<L, Rr>), dim3(grid), dim3(block), lds, st,
                           reinterpret_cast<const uint32_t *>(packed), scales, W, G, wstride,
                           cstride, ch, c0, nch, word0, elem0, srv_err,
                           reinterpret_cast<uint32_t *>(srv_packed), srv_scales, avg, flags, cpw,
                           inv_w, pow2 ? 1 : 0);
        return hipGetLastError();
    };
    using std::integral_constant;
    if (sg.V == 2) return go(integral_constant<int, 256>{}, integral_constant<int, 2>{});
    switch (sg.L) {
    case 1: return go(integral_constant<int, 1>{}, integral_constant<int, 1>{});
    case 2: return go(integral_constant<int, 2>{}, integral_constant<int, 1>{});
    case 4: return go(integral_constant<int, 4>{}, integral_constant<int, 1>{});
    case 8: return go(integral_constant<int, 8>{}, integral_constant<int, 1>{});
    case 16: return go(integral_constant<int, 16>{}, integral_constant<int, 1>{});
    case 32: return go(integral_constant<int, 32>{}, integral_constant<int, 1>{});
    case 64: return go(integral_constant<int, 64>{}, integral_constant<int, 1>{});
    case 128: return go(integral_constant<int, 128>{}, integral_constant<int, 1>{});
    case 256: return go(integral_constant<int, 256>{}, integral_constant<int, 1>{});
    default: return hipErrorInvalidValue;
    }
}

hipError_t launch_recon(Geometry geo, bool var, const uint64_t *srv_packed,
                        const float *srv_scales, const Chunks &ch, int64_t nchunks, float *m,
                        float *x, float *v, float *u, float *anchor, const float *gbar,
                        float gsum, const Scalars &s, hipStream_t st)
{
    if (nchunks == 0) return hipSuccess;
    return with_geometry(geo, [&](auto Lc, auto Vc) {
        constexpr int L = decltype(Lc)::value, V = decltype(Vc)::value;
        const unsigned grid = (unsigned)((nchunks + (256 / L) - 1) / (256 / L));
        const uint32_t *p32 = reinterpret_cast<const uint32_t *>(srv_packed);
        if (var)
            hipLaunchKernelGGL((k_recon<L, V, true>), dim3(grid), dim3(256), 0, st, p32,
                               srv_scales, ch, nchunks, m, x, v, u, anchor, gbar, gsum, s);
        else
            hipLaunchKernelGGL((k_recon<L, V, false>), dim3(grid), dim3(256), 0, st, p32,
                               srv_scales, ch, nchunks, m, x, v, u, anchor, gbar, gsum, s);
        return hipGetLastError();
    });
}

hipError_t launch_divsqrt(const float *a, const float *b, float *q, float *r, int64_t n,
                          hipStream_t st)
{
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(k_divsqrt, dim3(stream_grid((n + 3) / 4)), dim3(256), 0, st, a, b, q, r, n);
    return hipGetLastError();
}

}  // namespace zo
