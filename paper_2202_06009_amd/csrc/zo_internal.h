// zo_internal.h -- types shared by the host library and the kernel launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace zo {

// Binary32 scalars of one call; c1 = 1 - beta1 and c2 = 1 - beta2 are formed
// in binary32 on the host once, so every kernel uses the same constants.
struct Scalars {
    float b1, c1, b2, c2, eps, gamma;
    float gamma_u;  // U_GM: the buffer is +0 + gamma_u * m (see BufferIn)
};

// Where a kernel finds the buffer u (and, after a deferred reconstruction, the
// momentum).  U_MEM: u and m in memory.  U_ZERO: the state a deferred
// reconstruction leaves: u = +0, and m = (sign bit ? S_c : -S_c) / gamma_m from
// the library's copy of that server output (SrvCopy).  U_GM: u = +0 + gamma_u
// * m with m in memory, the momentum before this step (the only local step
// since the reset ran with gamma_u and wrote m; binary32, so the product is
// the value it added).
enum BufferIn { U_MEM = 0, U_ZERO = 1, U_GM = 2 };

// The library's copy of the last server output in deferred mode (packed sign
// words indexed like the shard's, one scale per chunk) and the learning-rate
// sum Gamma it was divided by.
struct SrvCopy {
    uint32_t *words32;
    float *scales;
    float gamma_m;
};

// Grid of the chunk-mapped elementwise kernels: bpc 256-thread workgroups per
// chunk of more than 1024 elements, else several chunks of lb lanes per
// workgroup.  Returns the workgroup count.
int64_t chunk_slots(int chunk, int64_t nchunks, int &bpc, int &lb);

// Device chunk table: start element, length, first packed word.
struct Chunks {
    const int64_t *start;
    const int32_t *len;
    const int64_t *word;
};

// Mapping of one chunk onto a workgroup: L lanes per chunk (a power of two
// <= 1024; several chunks share a 256-thread workgroup when L < 256), V blocks
// of 4L elements per lane (1, 2 or 4; > 1 only when L = 1024).
// 4 * L * V >= the configured chunk length.
struct Geometry {
    int L, V;
};

Geometry geometry_for(int chunk);

// Element type of the gradient inputs g and gbar (zo_config.grad_dtype).
enum GradType { GT_F32 = 0, GT_F16 = 1, GT_BF16 = 2 };

// Server-average algorithm.
enum SrvAlgo { SRV_AUTO = 0, SRV_PLAIN = 1 };

// `al` (every launcher of a chunk kernel): every chunk length is a multiple of
// 4, so every chunk starts and ends on a 16-byte boundary and its lanes use
// float4 accesses; otherwise the unaligned forms (zo_kernels_ua.hip).

// u_in: where u is (BufferIn; U_ZERO also takes m from `sm`, over the chunk
// grid); write_u: false only with U_ZERO, leaving u = gamma * m implicit;
// x_src may equal x.
hipError_t launch_local(bool var, int u_in, bool write_u, const void *g, float *m,
                        const float *x_src, float *x, float *v, float *u, const void *gbar,
                        int64_t n, const Scalars &s, int gt, const Chunks &ch, int64_t nchunks,
                        int chunk, bool al, const SrvCopy &sm, hipStream_t st);
// m = (bit ? S_c : -S_c) / gamma_m from the server copy, over the shard.
hipError_t launch_m_from_copy(float *m, const Chunks &ch, int64_t nchunks, int chunk, bool al,
                              const SrvCopy &sm, hipStream_t st);
// u = +0 + gamma_u * m (writes out an implicit U_GM buffer).
hipError_t launch_u_from_m(float *u, const float *m, int64_t n, float gamma_u, hipStream_t st);
hipError_t launch_zero(float *dst, int64_t n, hipStream_t st);
hipError_t launch_var(float *v, const void *gbar, int64_t n, const Scalars &s, int gt,
                      hipStream_t st);
// u_in (fused only): where u is (BufferIn).  gt: element type of g (fused);
// ut: of u, the compressed source when not fused (binary32 u, or the
// gradient under Algorithm 4).
hipError_t launch_sync1(Geometry geo, bool fused, int u_in, const void *g, const float *m,
                        const void *u, float *err, const Chunks &ch, int64_t nchunks,
                        uint64_t *packed, float *scales, const Scalars &s, int gt, int ut,
                        bool al, const SrvCopy &sm, hipStream_t st);
hipError_t launch_srv(Geometry geo, int algo, const uint64_t *packed, const float *scales, int W,
                      int64_t wstride, int64_t cstride, const Chunks &ch, int64_t c0,
                      int64_t nch, int64_t word0, int64_t elem0, float *srv_err,
                      uint64_t *srv_packed, float *srv_scales, float *avg, uint8_t *flags,
                      int chunk, bool al, hipStream_t st);
// defer: write the anchor and `sm` only (the model stays in the anchor, u = 0
// and m = the server average / Gamma implicit).
hipError_t launch_recon(bool var, bool defer, const uint64_t *srv_packed,
                        const float *srv_scales, const Chunks &ch, int64_t nchunks, float *m,
                        float *x, float *v, float *u, float *anchor, const void *gbar,
                        float gsum, const Scalars &s, int gt, int chunk, bool al,
                        const SrvCopy &sm, hipStream_t st);
// Algorithm 4: the full-precision step (t in T_v) and the step from the
// server's compressed average (t outside T_v).
hipError_t launch_fv_full(const void *gbar, float *x, float *m, float *v, int64_t n,
                          const Scalars &s, int gt, hipStream_t st);
hipError_t launch_fv_apply(const uint64_t *srv_packed, const float *srv_scales, const Chunks &ch,
                           int64_t nchunks, float *x, float *m, const float *v, const Scalars &s,
                           int chunk, bool al, hipStream_t st);
hipError_t launch_copy(const float *src, float *dst, int64_t n, bool nt, hipStream_t st);

// Streams of the HBM-mix diagnostic: up to 6 read and 4 write arrays.
struct StreamPtrs {
    const float *src[6];
    float *dst[5];
};
hipError_t launch_stream(int R, int S, const StreamPtrs &p, int64_t n, hipStream_t st);
hipError_t launch_srv_pattern(int chunk, const uint64_t *packed, int W, int64_t wstride,
                              const Chunks &ch, int64_t c0, int64_t nch, int64_t word0,
                              int64_t elem0, float *srv_err, hipStream_t st);
hipError_t launch_divsqrt(const float *a, const float *b, float *q, float *r, int64_t n,
                          hipStream_t st);

// The unaligned forms of the chunk launchers (zo_kernels_ua.hip), called by
// the launchers above when `al` is false.
hipError_t launch_local_zero_ua(bool var, bool write_u, const void *g, float *m,
                                const float *x_src, float *x, float *v, float *u,
                                const void *gbar, int64_t n4, const Scalars &s, int gt,
                                const Chunks &ch, int64_t nchunks, int chunk, const SrvCopy &sm,
                                hipStream_t st);
hipError_t launch_m_from_copy_ua(float *m, const Chunks &ch, int64_t nchunks, int chunk,
                                 const SrvCopy &sm, hipStream_t st);
hipError_t launch_sync1_ua(Geometry geo, bool fused, int u_in, const void *g, const float *m,
                           const void *u, float *err, const Chunks &ch, int64_t nchunks,
                           uint64_t *packed, float *scales, const Scalars &s, int gt, int ut,
                           const SrvCopy &sm, hipStream_t st);
hipError_t launch_fv_apply_ua(const uint64_t *srv_packed, const float *srv_scales,
                              const Chunks &ch, int64_t nchunks, float *x, float *m,
                              const float *v, const Scalars &s, int chunk, hipStream_t st);
hipError_t launch_recon_ua(bool var, bool defer, const uint64_t *srv_packed,
                           const float *srv_scales, const Chunks &ch, int64_t nchunks, float *m,
                           float *x, float *v, float *u, float *anchor, const void *gbar,
                           float gsum, const Scalars &s, int gt, int chunk, const SrvCopy &sm,
                           hipStream_t st);

}  // namespace zo
