// zo_device.h -- device code shared by the gfx950 kernels of the 0/1 Adam hot
// path: streaming access helpers, the per-element lines of Algorithm 1, the
// chunk machinery of Equation 3 (pairwise L1 tree, error feedback, sign
// packing) and the bodies of the chunk-mapped kernels, each for two access
// shapes: chunks whose elements start and end on 16-byte boundaries (every
// chunk length a multiple of 4: one float4 access per lane and block) and
// chunks that do not (the same lane layout, four element accesses with the
// tail past the chunk masked).  The kernel entry points live in
// zo_kernels.hip (aligned), zo_kernels_ua.hip (unaligned) and zo_server.hip;
// this header holds only inline and template code.
#pragma once

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


// Where a lane's four consecutive elements are.  At4: elements 4*i4 .. 4*i4+3,
// one 16-byte access.  At1: elements e .. e+3 of a chunk whose elements need
// not sit on a 16-byte boundary, of which the first nv (1..4) are inside the
// chunk: four element accesses, elements past the chunk read as +0 and never
// written.
struct At4 {
    int64_t i4;
};
struct At1 {
    int64_t e;
    int nv;
};
template <bool AL>
using At = std::conditional_t<AL, At4, At1>;

// The place of the four elements from element index e (a multiple of 4 when
// AL), `left` of them (>= 1) up to the end of the chunk.
template <bool AL>
__device__ __forceinline__ At<AL> at(int64_t e, int left)
{
    if constexpr (AL) {
        return At4{e >> 2};
    } else {
        return At1{e, left < 4 ? left : 4};
    }
}

__device__ __forceinline__ f4v ld(const float *p, At4 a) { return ldnt(p, a.i4); }
__device__ __forceinline__ f4v ld(const float *p, At1 a)
{
    f4v r;
#pragma unroll
    for (int q = 0; q < 4; ++q) r[q] = q < a.nv ? __builtin_nontemporal_load(p + a.e + q) : 0.0f;
    return r;
}

__device__ __forceinline__ void st(float *p, At4 a, f4v v) { stnt(p, a.i4, v); }
__device__ __forceinline__ void st(float *p, At1 a, f4v v)
{
#pragma unroll
    for (int q = 0; q < 4; ++q)
        if (q < a.nv) __builtin_nontemporal_store(v[q], p + a.e + q);
}

// Gradient elements of type GT widened to binary32 (see ldg4).
template <int GT>
__device__ __forceinline__ f4v ldg(const void *p, At4 a) { return ldg4<GT>(p, a.i4); }
template <int GT>
__device__ __forceinline__ f4v ldg(const void *p, At1 a)
{
    f4v r;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        if (q >= a.nv) {
            r[q] = 0.0f;
        } else if constexpr (GT == GT_F32) {
            r[q] = __builtin_nontemporal_load(static_cast<const float *>(p) + a.e + q);
        } else {
            const uint16_t h =
                __builtin_nontemporal_load(static_cast<const uint16_t *>(p) + a.e + q);
            if constexpr (GT == GT_BF16)
                r[q] = __uint_as_float((uint32_t)h << 16);
            else
                r[q] = (float)__builtin_bit_cast(_Float16, h);
        }
    }
    return r;
}

// Elements past the chunk set to +0 (they must not enter a chunk's L1 norm).
__device__ __forceinline__ f4v inside(f4v v, At4) { return v; }
__device__ __forceinline__ f4v inside(f4v v, At1 a)
{
#pragma unroll
    for (int q = 0; q < 4; ++q)
        if (q >= a.nv) v[q] = 0.0f;
    return v;
}

// Sign nibble with the bits of elements past the chunk cleared (pad bits 0).
__device__ __forceinline__ uint32_t inside_bits(uint32_t nib, At4) { return nib; }
__device__ __forceinline__ uint32_t inside_bits(uint32_t nib, At1 a)
{
    return nib & ((1u << a.nv) - 1u);
}

// ---------------------------------------------------------------------------
// a1 (+a2): local step, one float4 per thread
// ---------------------------------------------------------------------------

// The chunk c and the offset e (a multiple of 4) in it of this thread's four
// elements; false when the thread has none.
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

// The momentum of elements e .. e+3 of chunk c after a deferred reconstruction:
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
template <int UIN, class A>
__device__ __forceinline__ f4v buffer_in(const float *u, A a, f4v m_old, const Scalars &s)
{
    if constexpr (UIN == U_MEM) {
        return ld(u, a);
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
// server copy; the other variants run one float4 per thread over the shard
// (whose length is a multiple of 4: every segment's is), so only U_ZERO has an
// unaligned form (AL = false).
template <bool VAR, int UIN, bool WU, int GT, bool AL>
__device__ __forceinline__ void local_body(const void *__restrict__ g, float *__restrict__ m,
                                           const float *x_src, float *x,
                                           float *__restrict__ v, float *__restrict__ u,
                                           const void *__restrict__ gbar, int64_t n4,
                                           const Scalars &s, const Chunks &ch, int64_t nchunks,
                                           int bpc, int lb, const SrvCopy &sm)
{
    static_assert(AL || UIN == U_ZERO, "only the chunk-grid variant has an unaligned form");
    At<AL> a;
    f4v mm;
    if constexpr (UIN == U_ZERO) {
        int64_t c;
        int e;
        if (!chunk_slot(ch, nchunks, bpc, lb, c, e)) return;
        a = at<AL>(ch.start[c] + e, ch.len[c] - e);
        mm = m_from_copy(sm, ch, c, e);
    } else {
        const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
        if (i >= n4) return;
        a = At4{i};
        mm = ld(m, a);
    }
    f4v gg = ldg<GT>(g, a), xx = ld(x_src, a), vv = ld(v, a);
    f4v uu = buffer_in<UIN>(u, a, mm, s);
    f4v gb;
    if (VAR) gb = ldg<GT>(gbar, a);
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        float mc = mm[c], xc = xx[c], uc = uu[c];
        local_elem(gg[c], mc, xc, vv[c], uc, s);
        mm[c] = mc;
        xx[c] = xc;
        uu[c] = uc;
    }
    st(m, a, mm);
    st(x, a, xx);
    if (WU) st(u, a, uu);
    if (VAR) {
#pragma unroll
        for (int c = 0; c < 4; ++c) vv[c] = var_elem(vv[c], gb[c], s);
        st(v, a, vv);
    }
}

// m = (bit ? S_c : -S_c) / Gamma from the server copy, over the chunk grid.
template <bool AL>
__device__ __forceinline__ void m_from_copy_body(float *__restrict__ m, const Chunks &ch,
                                                 int64_t nchunks, int bpc, int lb,
                                                 const SrvCopy &sm)
{
    int64_t c;
    int e;
    if (!chunk_slot(ch, nchunks, bpc, lb, c, e)) return;
    st(m, at<AL>(ch.start[c] + e, ch.len[c] - e), m_from_copy(sm, ch, c, e));
}

// ---------------------------------------------------------------------------
// chunk machinery
// ---------------------------------------------------------------------------

// One level of an xor butterfly across the lanes of a wave: both lanes of
// each pair (i, i ^ H) get op(value of the lower lane, value of the upper).
// The pairs are formed by lane permutations in the vector ALU (DPP inside
// 16-lane rows; the row-swap instructions across rows), not through the LDS.
// Every lane of the wave must be active.
template <int H, class Op>
__device__ __forceinline__ uint32_t butterfly(uint32_t x, Op op)
{
    static_assert(H == 1 || H == 2 || H == 4 || H == 8 || H == 16 || H == 32, "lane offset");
    const int v = (int)x;
    if constexpr (H <= 8) {
        // DPP controls: quad_perm [1,0,3,2] = i^1, [2,3,0,1] = i^2,
        // [3,2,1,0] = i^3; row_mirror = i^15 and row_half_mirror = i^7 in a row
        int y;
        if constexpr (H == 1) {
            y = __builtin_amdgcn_mov_dpp(v, 0xB1, 0xF, 0xF, false);
        } else if constexpr (H == 2) {
            y = __builtin_amdgcn_mov_dpp(v, 0x4E, 0xF, 0xF, false);
        } else if constexpr (H == 4) {  // i^3, then ^7
            y = __builtin_amdgcn_mov_dpp(__builtin_amdgcn_mov_dpp(v, 0x1B, 0xF, 0xF, false), 0x141,
                                         0xF, 0xF, false);
        } else {  // i^15, then ^7
            y = __builtin_amdgcn_mov_dpp(__builtin_amdgcn_mov_dpp(v, 0x140, 0xF, 0xF, false), 0x141,
                                         0xF, 0xF, false);
        }
        const uint32_t o = (uint32_t)y;
        return (threadIdx.x & H) ? op(o, x) : op(x, o);
    } else {
        // the swap returns {lower row or half in every lane, upper in every lane}
        const auto r = H == 16 ? __builtin_amdgcn_permlane16_swap(x, x, false, false)
                               : __builtin_amdgcn_permlane32_swap(x, x, false, false);
        return op((uint32_t)r[0], (uint32_t)r[1]);
    }
}

// op over aligned groups of N lanes (N a power of two, at most 64), the
// result in every lane of the group: the butterfly levels 1, 2, .., N/2.
template <int N, class Op>
__device__ __forceinline__ uint32_t lanes_reduce(uint32_t x, Op op)
{
    static_assert(N >= 1 && N <= 64 && (N & (N - 1)) == 0, "group size");
    if constexpr (N > 1) x = butterfly<1>(x, op);
    if constexpr (N > 2) x = butterfly<2>(x, op);
    if constexpr (N > 4) x = butterfly<4>(x, op);
    if constexpr (N > 8) x = butterfly<8>(x, op);
    if constexpr (N > 16) x = butterfly<16>(x, op);
    if constexpr (N > 32) x = butterfly<32>(x, op);
    return x;
}

// The cross-lane steps of the chunk machinery come in two forms.  DPP: lane
// permutations in the vector ALU (butterfly above), used by the server's
// compression.  Otherwise LDS-routed shuffles (__shfl_xor), used by the
// worker's compress kernel: there they measured faster, although the LDS
// form holds more registers.  Both add the same pairs in the same order.

// Sum over the lanes of a chunk that share a wave: an xor butterfly with
// rising offsets (the index-order pairwise tree over those lanes).
template <int L, bool DPP>
__device__ __forceinline__ float wave_tree(float x)
{
    constexpr int N = L < 64 ? L : 64;
    if constexpr (!DPP) {
#pragma unroll
        for (int o = 1; o < N; o <<= 1) x = x + __shfl_xor(x, o);
        return x;
    } else {
        const auto add = [](uint32_t a, uint32_t b) {
            return __float_as_uint(__uint_as_float(a) + __uint_as_float(b));
        };
        return __uint_as_float(lanes_reduce<N>(__float_as_uint(x), add));
    }
}

// OR over aligned groups of 8 lanes (fewer when L < 8).
template <int L, bool DPP>
__device__ __forceinline__ uint32_t wave_or8(uint32_t x)
{
    constexpr int N = L < 8 ? L : 8;
    if constexpr (!DPP) {
#pragma unroll
        for (int o = 1; o < N; o <<= 1) x |= (uint32_t)__shfl_xor((int)x, o);
        return x;
    } else {
        return lanes_reduce<N>(x, [](uint32_t a, uint32_t b) { return a | b; });
    }
}

// The chunk's pairwise L1 tree from each lane's per-block partial sums (the
// in-lane level).  Returns the total to every lane of the chunk.  Every
// thread of the workgroup must call it (it synchronises when L > 64).  `lds`
// holds (blockDim / 64) * V floats.
template <int L, int V, bool DPP>
__device__ __forceinline__ float chunk_tree(float (&part)[V], float *lds)
{
#pragma unroll
    for (int k = 0; k < V; ++k) part[k] = wave_tree<L, DPP>(part[k]);
    if constexpr (L <= 64) {
        // the chunk's lanes share a wave: the in-order tree over its blocks
#pragma unroll
        for (int h = 1; h < V; h <<= 1) {
#pragma unroll
            for (int k = 0; k + h < V; k += 2 * h) part[k] = part[k] + part[k + h];
        }
        return part[0];
    } else if constexpr (DPP) {
        // The wave totals of block k sit at k * NW + w (w: the chunk's wave),
        // at most 64 of them.  Lane j of every wave takes the one at j mod NP,
        // and the butterfly with rising offsets forms the tree over w (the low
        // index bits), then over k: one value per lane.
        constexpr int NW = L / 64;  // waves per chunk
        constexpr int NP = NW * V;  // wave totals per chunk
        static_assert(NP <= 64, "one wave holds the chunk's wave totals");
        const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
        const int base = (wave / NW) * NP;
        __syncthreads();  // lds may still be read by a previous call
        if (lane == 0) {
#pragma unroll
            for (int k = 0; k < V; ++k) lds[base + k * NW + wave % NW] = part[k];
        }
        __syncthreads();
        return wave_tree<NP, true>(lds[base + (lane & (NP - 1))]);
    } else {
        // every lane reads the chunk's NW * V wave totals and forms the tree
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
// signs (all 2*ceil(len/64) dwords of the chunk, pad bits 0) and the scale.
// AL: the chunk's elements start on a 16-byte boundary and len is a multiple
// of 4 (see At4 / At1).
// get_a(k) returns block k of a (from registers or from where the caller
// stashed it); part[k] = abs4 of it, formed by the caller.  DPP: the form of
// the cross-lane steps (see wave_tree).
template <int L, int V, bool AL, bool DPP, class GetA>
__device__ __forceinline__ void compress_chunk_from(const float (&part_in)[V], GetA get_a, int lc,
                                                    int len, bool active,
                                                    float *__restrict__ err, int64_t err_e0,
                                                    uint32_t *__restrict__ words32,
                                                    float *scale_out, float *lds)
{
    float part[V];
#pragma unroll
    for (int k = 0; k < V; ++k) part[k] = part_in[k];
    const float tot = chunk_tree<L, V, DPP>(part, lds);
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
            const At<AL> a = at<AL>(err_e0 + e, len - e);
            f4v d;
#pragma unroll
            for (int c = 0; c < 4; ++c) d[c] = ef_elem(ak[c], s);
            st(err, a, d);
            nib = inside_bits(sign4(ak), a);
        }
        const uint32_t dw = wave_or8<L, DPP>(nib << (4 * (lc & 7)));
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

// The server's compression of its average plus error, held in registers.
template <int L, int V, bool AL>
__device__ __forceinline__ void compress_chunk(f4v (&a)[V], int lc, int len, bool active,
                                               float *__restrict__ err, int64_t err_e0,
                                               uint32_t *__restrict__ words32, float *scale_out,
                                               float *lds)
{
    float part[V];
#pragma unroll
    for (int k = 0; k < V; ++k) part[k] = abs4(a[k]);
    compress_chunk_from<L, V, AL, true>(part, [&](int k) { return a[k]; }, lc, len, active, err,
                                        err_e0, words32, scale_out, lds);
}


// ---------------------------------------------------------------------------
// a3: worker compress + error feedback + pack (fused with the momentum and
// buffer lines when g != nullptr)
// ---------------------------------------------------------------------------

// UIN (with FUSED only; U_MEM otherwise): where u is (BufferIn).  GT: element
// type of g when FUSED, else of u (binary32 u, or the gradient itself under
// Algorithm 4).  `lds` holds 64 floats; `stash` L*V float4s when V > 1.
template <int L, int V, bool FUSED, int UIN, int GT, bool AL>
__device__ __forceinline__ void sync1_body(const void *__restrict__ g, const float *__restrict__ m,
                                           const void *__restrict__ u, float *__restrict__ err,
                                           const Chunks &ch, int64_t nchunks,
                                           uint32_t *__restrict__ packed32,
                                           float *__restrict__ scales, const Scalars &s,
                                           const SrvCopy &sm, float *lds, f4v *stash)
{
    // With several blocks per lane, a is parked in LDS across the chunk's
    // reduction instead of in registers: that keeps a 1024-lane chunk within
    // 64 registers, so two chunks share a CU.
    constexpr bool kStash = V > 1;
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
            const At<AL> p = at<AL>(e0 + e, len - e);
            const f4v dd = ld(err, p);
            f4v uu;
            if (FUSED) {
                const f4v gg = ldg<GT>(g, p);
                const f4v mm = UIN == U_ZERO ? m_from_copy(sm, ch, c, e) : ld(m, p);
                uu = buffer_in<UIN>(static_cast<const float *>(u), p, mm, s);
#pragma unroll
                for (int q = 0; q < 4; ++q) uu[q] = uu[q] + s.gamma * (s.b1 * mm[q] + s.c1 * gg[q]);
            } else {
                uu = ldg<GT>(u, p);
            }
#pragma unroll
            for (int q = 0; q < 4; ++q) ak[q] = uu[q] + dd[q];
            ak = inside(ak, p);
        }
        part[k] = abs4(ak);
        if constexpr (kStash)
            stash[k * L + lc] = ak;
        else
            a[k] = ak;
    }
    compress_chunk_from<L, V, AL, false>(
        part, [&](int k) { return kStash ? stash[k * L + lc] : a[kStash ? 0 : k]; }, lc, len,
        active, err, e0, packed32 + 2 * (active ? ch.word[c] : 0), scales + (active ? c : 0), lds);
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
template <bool VAR, bool DEFER, int GT, bool AL>
__device__ __forceinline__ void recon_body(const uint32_t *__restrict__ srv_packed32,
                                           const float *__restrict__ srv_scales, const Chunks &ch,
                                           int64_t nchunks, int bpc, int lb,
                                           float *__restrict__ m, float *__restrict__ x,
                                           float *__restrict__ v, float *__restrict__ u,
                                           float *__restrict__ anchor,
                                           const void *__restrict__ gbar, float gsum,
                                           const Scalars &s, const SrvCopy &sm)
{
    int64_t c;
    int e;
    if (!chunk_slot(ch, nchunks, bpc, lb, c, e)) return;
    const At<AL> a = at<AL>(ch.start[c] + e, ch.len[c] - e);
    const float sc = srv_scales[c];
    const int64_t wd = 2 * ch.word[c] + (e >> 5);
    const uint32_t dw = srv_packed32[wd];
    const uint32_t bits = dw >> (e & 31);
    if (DEFER) {
        // the copy the next step rebuilds m from (one thread per dword)
        if ((e & 31) == 0) sm.words32[wd] = dw;
        if (e == 0) sm.scales[c] = sc;
    }
    const f4v vv = ld(v, a), an = ld(anchor, a);
    f4v gb;
    if (VAR) gb = ldg<GT>(gbar, a);
    f4v mm, xx, nv;
    const float mq = sc / gsum;  // odd in sc, so one division serves both signs
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const float ub = ((bits >> q) & 1u) ? sc : -sc;
        mm[q] = ((bits >> q) & 1u) ? mq : -mq;
        xx[q] = an[q] - ub / sqrtf(vv[q] + s.eps);
        if (VAR) nv[q] = var_elem(vv[q], gb[q], s);
    }
    st(anchor, a, xx);
    if (!DEFER) {
        st(m, a, mm);
        st(x, a, xx);
        st(u, a, f4v{0.f, 0.f, 0.f, 0.f});
    }
    if (VAR) st(v, a, nv);
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

// t outside T_v: gbar = sigma * s of the server's packed words (v kept).
template <bool AL>
__device__ __forceinline__ void fv_apply_body(const uint32_t *__restrict__ srv_packed32,
                                              const float *__restrict__ srv_scales,
                                              const Chunks &ch, int64_t nchunks, int bpc, int lb,
                                              float *__restrict__ x, float *__restrict__ m,
                                              const float *__restrict__ v, const Scalars &s)
{
    int64_t c;
    int e;
    if (!chunk_slot(ch, nchunks, bpc, lb, c, e)) return;
    const At<AL> a = at<AL>(ch.start[c] + e, ch.len[c] - e);
    const float sc = srv_scales[c];
    const uint32_t bits = srv_packed32[2 * ch.word[c] + (e >> 5)] >> (e & 31);
    const f4v vv = ld(v, a);
    f4v xx = ld(x, a), mm = ld(m, a);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        float xc = xx[q], mc = mm[q], vc = vv[q];
        fv_elem(((bits >> q) & 1u) ? sc : -sc, xc, mc, vc, false, s);
        xx[q] = xc;
        mm[q] = mc;
    }
    st(x, a, xx);
    st(m, a, mm);
}

// ---------------------------------------------------------------------------
// kernel entry points of the chunk-mapped steps: <name> for aligned chunks,
// <name>_ua for the rest (the same body; see At4 / At1)
// ---------------------------------------------------------------------------

template <bool VAR, int UIN, bool WU, int GT>
__global__ __launch_bounds__(256) void k_local(const void *__restrict__ g, float *__restrict__ m,
                                               const float *x_src, float *x,
                                               float *__restrict__ v, float *__restrict__ u,
                                               const void *__restrict__ gbar, int64_t n4,
                                               Scalars s, Chunks ch, int64_t nchunks, int bpc,
                                               int lb, SrvCopy sm)
{
    local_body<VAR, UIN, WU, GT, true>(g, m, x_src, x, v, u, gbar, n4, s, ch, nchunks, bpc, lb,
                                       sm);
}

template <bool VAR, bool WU, int GT>
__global__ __launch_bounds__(256) void k_local_ua(const void *__restrict__ g,
                                                  float *__restrict__ m, const float *x_src,
                                                  float *x, float *__restrict__ v,
                                                  float *__restrict__ u,
                                                  const void *__restrict__ gbar, int64_t n4,
                                                  Scalars s, Chunks ch, int64_t nchunks, int bpc,
                                                  int lb, SrvCopy sm)
{
    local_body<VAR, U_ZERO, WU, GT, false>(g, m, x_src, x, v, u, gbar, n4, s, ch, nchunks, bpc,
                                           lb, sm);
}

__global__ __launch_bounds__(256) void k_m_from_copy(float *__restrict__ m, Chunks ch,
                                                     int64_t nchunks, int bpc, int lb,
                                                     SrvCopy sm);
__global__ __launch_bounds__(256) void k_m_from_copy_ua(float *__restrict__ m, Chunks ch,
                                                        int64_t nchunks, int bpc, int lb,
                                                        SrvCopy sm);

template <int L, int V, bool FUSED, int UIN, int GT>
__global__ __launch_bounds__(L > 256 ? L : 256, V > 1 ? 8 : 1) void k_sync1(
    const void *__restrict__ g, const float *__restrict__ m, const void *__restrict__ u,
    float *__restrict__ err, Chunks ch, int64_t nchunks, uint32_t *__restrict__ packed32,
    float *__restrict__ scales, Scalars s, SrvCopy sm)
{
    __shared__ float lds[64];
    __shared__ f4v stash[V > 1 ? L * V : 1];
    sync1_body<L, V, FUSED, UIN, GT, true>(g, m, u, err, ch, nchunks, packed32, scales, s, sm,
                                           lds, stash);
}

template <int L, int V, bool FUSED, int UIN, int GT>
__global__ __launch_bounds__(L > 256 ? L : 256, V > 1 ? 8 : 1) void k_sync1_ua(
    const void *__restrict__ g, const float *__restrict__ m, const void *__restrict__ u,
    float *__restrict__ err, Chunks ch, int64_t nchunks, uint32_t *__restrict__ packed32,
    float *__restrict__ scales, Scalars s, SrvCopy sm)
{
    __shared__ float lds[64];
    __shared__ f4v stash[V > 1 ? L * V : 1];
    sync1_body<L, V, FUSED, UIN, GT, false>(g, m, u, err, ch, nchunks, packed32, scales, s, sm,
                                            lds, stash);
}

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
    recon_body<VAR, DEFER, GT, true>(srv_packed32, srv_scales, ch, nchunks, bpc, lb, m, x, v, u,
                                     anchor, gbar, gsum, s, sm);
}

template <bool VAR, bool DEFER, int GT>
__global__ __launch_bounds__(256) void k_recon_ua(const uint32_t *__restrict__ srv_packed32,
                                                  const float *__restrict__ srv_scales,
                                                  Chunks ch, int64_t nchunks, int bpc, int lb,
                                                  float *__restrict__ m, float *__restrict__ x,
                                                  float *__restrict__ v, float *__restrict__ u,
                                                  float *__restrict__ anchor,
                                                  const void *__restrict__ gbar, float gsum,
                                                  Scalars s, SrvCopy sm)
{
    recon_body<VAR, DEFER, GT, false>(srv_packed32, srv_scales, ch, nchunks, bpc, lb, m, x, v,
                                      u, anchor, gbar, gsum, s, sm);
}

__global__ __launch_bounds__(256) void k_fv_apply(const uint32_t *__restrict__ srv_packed32,
                                                  const float *__restrict__ srv_scales, Chunks ch,
                                                  int64_t nchunks, int bpc, int lb,
                                                  float *__restrict__ x, float *__restrict__ m,
                                                  const float *__restrict__ v, Scalars s);
__global__ __launch_bounds__(256) void k_fv_apply_ua(const uint32_t *__restrict__ srv_packed32,
                                                     const float *__restrict__ srv_scales,
                                                     Chunks ch, int64_t nchunks, int bpc, int lb,
                                                     float *__restrict__ x, float *__restrict__ m,
                                                     const float *__restrict__ v, Scalars s);

// ---------------------------------------------------------------------------
// launch helpers
// ---------------------------------------------------------------------------

static inline int next_pow2(int v)
{
    int p = 1;
    while (p < v) p <<= 1;
    return p;
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

// The local step right after a deferred reconstruction (U_ZERO), over the
// chunk grid: k_local<VAR, U_ZERO, WU, GT> or its unaligned form.
template <bool AL>
static hipError_t launch_local_zero_t(bool var, bool write_u, const void *g, float *m,
                                      const float *x_src, float *x, float *v, float *u,
                                      const void *gbar, int64_t n4, const Scalars &s, int gt,
                                      const Chunks &ch, int64_t nchunks, int chunk,
                                      const SrvCopy &sm, hipStream_t st)
{
    int bpc = 1, lb = 1;
    const int64_t blocks = chunk_slots(chunk, nchunks, bpc, lb);
    if (blocks == 0) return hipSuccess;
    const dim3 grid((unsigned)blocks), block(256);
    return with_grad_type(gt, [&](auto T) {
        constexpr int GT = decltype(T)::value;
        auto go = [&](auto kernel) {
            hipLaunchKernelGGL(kernel, grid, block, 0, st, g, m, x_src, x, v, u, gbar, n4, s, ch,
                               nchunks, bpc, lb, sm);
            return hipGetLastError();
        };
        if constexpr (AL) {
            if (var) return write_u ? go(k_local<true, U_ZERO, true, GT>)
                                    : go(k_local<true, U_ZERO, false, GT>);
            return write_u ? go(k_local<false, U_ZERO, true, GT>)
                           : go(k_local<false, U_ZERO, false, GT>);
        } else {
            if (var) return write_u ? go(k_local_ua<true, true, GT>)
                                    : go(k_local_ua<true, false, GT>);
            return write_u ? go(k_local_ua<false, true, GT>) : go(k_local_ua<false, false, GT>);
        }
    });
}

template <bool AL>
static hipError_t launch_m_from_copy_t(float *m, const Chunks &ch, int64_t nchunks, int chunk,
                                       const SrvCopy &sm, hipStream_t st)
{
    if (nchunks == 0) return hipSuccess;
    int bpc, lb;
    const int64_t blocks = chunk_slots(chunk, nchunks, bpc, lb);
    hipLaunchKernelGGL(AL ? k_m_from_copy : k_m_from_copy_ua, dim3((unsigned)blocks), dim3(256),
                       0, st, m, ch, nchunks, bpc, lb, sm);
    return hipGetLastError();
}

template <bool AL>
static hipError_t launch_sync1_t(Geometry geo, bool fused, int u_in, const void *g,
                                 const float *m, const void *u, float *err, const Chunks &ch,
                                 int64_t nchunks, uint64_t *packed, float *scales,
                                 const Scalars &s, int gt, int ut, const SrvCopy &sm,
                                 hipStream_t st)
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
            if constexpr (AL) {
                if (!fused) return go(k_sync1<L, V, false, U_MEM, GT>);
                switch (u_in) {
                case U_MEM: return go(k_sync1<L, V, true, U_MEM, GT>);
                case U_ZERO: return go(k_sync1<L, V, true, U_ZERO, GT>);
                case U_GM: return go(k_sync1<L, V, true, U_GM, GT>);
                default: return hipErrorInvalidValue;
                }
            } else {
                if (!fused) return go(k_sync1_ua<L, V, false, U_MEM, GT>);
                switch (u_in) {
                case U_MEM: return go(k_sync1_ua<L, V, true, U_MEM, GT>);
                case U_ZERO: return go(k_sync1_ua<L, V, true, U_ZERO, GT>);
                case U_GM: return go(k_sync1_ua<L, V, true, U_GM, GT>);
                default: return hipErrorInvalidValue;
                }
            }
        });
    });
}

template <bool AL>
static hipError_t launch_fv_apply_t(const uint64_t *srv_packed, const float *srv_scales,
                                    const Chunks &ch, int64_t nchunks, float *x, float *m,
                                    const float *v, const Scalars &s, int chunk, hipStream_t st)
{
    if (nchunks == 0) return hipSuccess;
    int bpc, lb;
    const int64_t grid = chunk_slots(chunk, nchunks, bpc, lb);
    hipLaunchKernelGGL(AL ? k_fv_apply : k_fv_apply_ua, dim3((unsigned)grid), dim3(256), 0, st,
                       reinterpret_cast<const uint32_t *>(srv_packed), srv_scales, ch, nchunks,
                       bpc, lb, x, m, v, s);
    return hipGetLastError();
}

template <bool AL>
static hipError_t launch_recon_t(bool var, bool defer, const uint64_t *srv_packed,
                                 const float *srv_scales, const Chunks &ch, int64_t nchunks,
                                 float *m, float *x, float *v, float *u, float *anchor,
                                 const void *gbar, float gsum, const Scalars &s, int gt,
                                 int chunk, const SrvCopy &sm, hipStream_t st)
{
    if (nchunks == 0) return hipSuccess;
    int bpc, lb;
    const int64_t grid = chunk_slots(chunk, nchunks, bpc, lb);
    const uint32_t *p32 = reinterpret_cast<const uint32_t *>(srv_packed);
    const dim3 g3((unsigned)grid), b3(256);
    return with_grad_type(gt, [&](auto T) {
        constexpr int GT = decltype(T)::value;
        auto go = [&](auto kernel) {
            hipLaunchKernelGGL(kernel, g3, b3, 0, st, p32, srv_scales, ch, nchunks, bpc, lb, m, x,
                               v, u, anchor, gbar, gsum, s, sm);
            return hipGetLastError();
        };
        if constexpr (AL) {
            if (var) return defer ? go(k_recon<true, true, GT>) : go(k_recon<true, false, GT>);
            return defer ? go(k_recon<false, true, GT>) : go(k_recon<false, false, GT>);
        } else {
            if (var) return defer ? go(k_recon_ua<true, true, GT>) : go(k_recon_ua<true, false, GT>);
            return defer ? go(k_recon_ua<false, true, GT>) : go(k_recon_ua<false, false, GT>);
        }
    });
}

}  // namespace zo
