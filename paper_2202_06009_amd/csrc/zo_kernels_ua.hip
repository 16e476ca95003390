// zo_kernels_ua.hip -- the chunk kernels of the 0/1 Adam hot path for chunk
// lengths that are not a multiple of 4: a chunk then need not start on a
// 16-byte boundary and may end inside a float4, so each lane reads and writes
// its four elements one by one and masks those past the chunk (At1 in
// zo_device.h).  The arithmetic, the lane layout, the L1 tree and the packing
// are the aligned kernels' own code (the same templates), so the results are
// the same functions of the inputs.
#include "zo_device.h"

namespace zo {

__global__ __launch_bounds__(256) void k_m_from_copy_ua(float *__restrict__ m, Chunks ch,
                                                        int64_t nchunks, int bpc, int lb,
                                                        SrvCopy sm)
{
    m_from_copy_body<false>(m, ch, nchunks, bpc, lb, sm);
}

__global__ __launch_bounds__(256) void k_fv_apply_ua(const uint32_t *__restrict__ srv_packed32,
                                                     const float *__restrict__ srv_scales,
                                                     Chunks ch, int64_t nchunks, int bpc, int lb,
                                                     float *__restrict__ x, float *__restrict__ m,
                                                     const float *__restrict__ v, Scalars s)
{
    fv_apply_body<false>(srv_packed32, srv_scales, ch, nchunks, bpc, lb, x, m, v, s);
}

hipError_t launch_local_zero_ua(bool var, bool write_u, const void *g, float *m,
                                const float *x_src, float *x, float *v, float *u,
                                const void *gbar, int64_t n4, const Scalars &s, int gt,
                                const Chunks &ch, int64_t nchunks, int chunk, const SrvCopy &sm,
                                hipStream_t st)
{
    return launch_local_zero_t<false>(var, write_u, g, m, x_src, x, v, u, gbar, n4, s, gt, ch,
                                      nchunks, chunk, sm, st);
}

hipError_t launch_m_from_copy_ua(float *m, const Chunks &ch, int64_t nchunks, int chunk,
                                 const SrvCopy &sm, hipStream_t st)
{
    return launch_m_from_copy_t<false>(m, ch, nchunks, chunk, sm, st);
}

hipError_t launch_sync1_ua(Geometry geo, bool fused, int u_in, const void *g, const float *m,
                           const void *u, float *err, const Chunks &ch, int64_t nchunks,
                           uint64_t *packed, float *scales, const Scalars &s, int gt, int ut,
                           const SrvCopy &sm, hipStream_t st)
{
    return launch_sync1_t<false>(geo, fused, u_in, g, m, u, err, ch, nchunks, packed, scales, s,
                                 gt, ut, sm, st);
}

hipError_t launch_fv_apply_ua(const uint64_t *srv_packed, const float *srv_scales,
                              const Chunks &ch, int64_t nchunks, float *x, float *m,
                              const float *v, const Scalars &s, int chunk, hipStream_t st)
{
    return launch_fv_apply_t<false>(srv_packed, srv_scales, ch, nchunks, x, m, v, s, chunk, st);
}

hipError_t launch_recon_ua(bool var, bool defer, const uint64_t *srv_packed,
                           const float *srv_scales, const Chunks &ch, int64_t nchunks, float *m,
                           float *x, float *v, float *u, float *anchor, const void *gbar,
                           float gsum, const Scalars &s, int gt, int chunk, const SrvCopy &sm,
                           hipStream_t st)
{
    return launch_recon_t<false>(var, defer, srv_packed, srv_scales, ch, nchunks, m, x, v, u,
                                 anchor, gbar, gsum, s, gt, chunk, sm, st);
}

}  // namespace zo
