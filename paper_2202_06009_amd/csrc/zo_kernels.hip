// zo_kernels.hip -- gfx950 kernels of the 0/1 Adam hot path: the elementwise
// steps, the worker compress, the reconstruction and their launchers (the
// server is in zo_server.hip, the unaligned forms of the chunk kernels in
// zo_kernels_ua.hip, the code they share in zo_device.h).
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
#include "zo_device.h"

namespace zo {

// ---------------------------------------------------------------------------
// a2 standalone, Algorithm 4's full-precision step, the buffer reset
// ---------------------------------------------------------------------------

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


// dst = +0, one float4 per thread (u after a deferred reset).
__global__ __launch_bounds__(256) void k_zero(float *__restrict__ dst, int64_t n4)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n4) return;
    stnt(dst, i, f4v{0.f, 0.f, 0.f, 0.f});
}
// Entry points of chunk-grid kernels whose bodies are in zo_device.h (their
// unaligned forms are in zo_kernels_ua.hip).
__global__ __launch_bounds__(256) void k_m_from_copy(float *__restrict__ m, Chunks ch,
                                                     int64_t nchunks, int bpc, int lb,
                                                     SrvCopy sm)
{
    m_from_copy_body<true>(m, ch, nchunks, bpc, lb, sm);
}

__global__ __launch_bounds__(256) void k_fv_apply(const uint32_t *__restrict__ srv_packed32,
                                                  const float *__restrict__ srv_scales, Chunks ch,
                                                  int64_t nchunks, int bpc, int lb,
                                                  float *__restrict__ x, float *__restrict__ m,
                                                  const float *__restrict__ v, Scalars s)
{
    fv_apply_body<true>(srv_packed32, srv_scales, ch, nchunks, bpc, lb, x, m, v, s);
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
// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------

// Lanes per chunk and blocks per lane of the compress kernels: one float4 per
// lane and block, up to 1024 lanes (16 waves) per chunk.
Geometry geometry_for(int chunk)
{
    const int lanes = (chunk + 3) / 4;
    if (lanes <= 256) return Geometry{next_pow2(lanes), 1};
    const int L = next_pow2(lanes) < 1024 ? next_pow2(lanes) : 1024;
    return Geometry{L, next_pow2((lanes + L - 1) / L)};
}

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
                        int chunk, bool al, const SrvCopy &sm, hipStream_t st)
{
    const int64_t n4 = n / 4;
    if (n4 == 0) return hipSuccess;
    if (!write_u && u_in != U_ZERO) return hipErrorInvalidValue;
    // U_ZERO: the chunk grid; otherwise one float4 per thread
    if (u_in == U_ZERO) {
        if (al)
            return launch_local_zero_t<true>(var, write_u, g, m, x_src, x, v, u, gbar, n4, s, gt,
                                             ch, nchunks, chunk, sm, st);
        return launch_local_zero_ua(var, write_u, g, m, x_src, x, v, u, gbar, n4, s, gt, ch,
                                    nchunks, chunk, sm, st);
    }
    const dim3 grid(grid_for(n4, 256)), block(256);
    return with_grad_type(gt, [&](auto T) {
        constexpr int GT = decltype(T)::value;
        auto go = [&](auto kernel) {
            hipLaunchKernelGGL(kernel, grid, block, 0, st, g, m, x_src, x, v, u, gbar, n4, s, ch,
                               nchunks, 1, 1, sm);
            return hipGetLastError();
        };
        switch (u_in) {
        case U_MEM: return var ? go(k_local<true, U_MEM, true, GT>)
                               : go(k_local<false, U_MEM, true, GT>);
        case U_GM: return var ? go(k_local<true, U_GM, true, GT>)
                              : go(k_local<false, U_GM, true, GT>);
        default: return hipErrorInvalidValue;
        }
    });
}

hipError_t launch_m_from_copy(float *m, const Chunks &ch, int64_t nchunks, int chunk, bool al,
                              const SrvCopy &sm, hipStream_t st)
{
    return al ? launch_m_from_copy_t<true>(m, ch, nchunks, chunk, sm, st)
              : launch_m_from_copy_ua(m, ch, nchunks, chunk, sm, st);
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
                        bool al, const SrvCopy &sm, hipStream_t st)
{
    if (al)
        return launch_sync1_t<true>(geo, fused, u_in, g, m, u, err, ch, nchunks, packed, scales,
                                    s, gt, ut, sm, st);
    return launch_sync1_ua(geo, fused, u_in, g, m, u, err, ch, nchunks, packed, scales, s, gt, ut,
                           sm, st);
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
                           int chunk, bool al, hipStream_t st)
{
    return al ? launch_fv_apply_t<true>(srv_packed, srv_scales, ch, nchunks, x, m, v, s, chunk, st)
              : launch_fv_apply_ua(srv_packed, srv_scales, ch, nchunks, x, m, v, s, chunk, st);
}

hipError_t launch_recon(bool var, bool defer, const uint64_t *srv_packed,
                        const float *srv_scales, const Chunks &ch, int64_t nchunks, float *m,
                        float *x, float *v, float *u, float *anchor, const void *gbar,
                        float gsum, const Scalars &s, int gt, int chunk, bool al,
                        const SrvCopy &sm, hipStream_t st)
{
    if (al)
        return launch_recon_t<true>(var, defer, srv_packed, srv_scales, ch, nchunks, m, x, v, u,
                                    anchor, gbar, gsum, s, gt, chunk, sm, st);
    return launch_recon_ua(var, defer, srv_packed, srv_scales, ch, nchunks, m, x, v, u, anchor,
                           gbar, gsum, s, gt, chunk, sm, st);
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
