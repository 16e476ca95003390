// zo_server.hip -- the server half of Algorithm 2 on gfx950: unpack the W
// workers' packed signs, average them exactly, add the server error, compress
// the result with Equation 3 per chunk and pack it (k_srv_lut with subset-sum
// lookup tables, k_srv_plain otherwise), plus the diagnostic of the server's
// memory accesses.  Shared device code is in zo_device.h.
#include "zo_device.h"

namespace zo {

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
    lo = (int)lanes_reduce<LW>((uint32_t)lo, [](uint32_t a, uint32_t b) {
        return (uint32_t)min((int)a, (int)b);
    });
    hi = (int)lanes_reduce<LW>((uint32_t)hi, [](uint32_t a, uint32_t b) {
        return (uint32_t)max((int)a, (int)b);
    });
    bad = (int)lanes_reduce<LW>((uint32_t)bad, [](uint32_t a, uint32_t b) { return a | b; });
    int lg = 0;
    while ((1 << lg) < W) ++lg;
    if (hi < lo) return (uint32_t)bad;  // every scale is zero
    return (uint32_t)(bad || (hi + 1 + lg - lo > 53));
}

// Plain server: per element, per worker, select +-S_w and add in binary64.
// Kept for worker counts whose lookup tables do not fit in LDS.
// AL: aligned chunks (see At4 / At1); the only server form for chunk lengths
// that are not a multiple of 4.
template <int L, int V, bool AL>
__device__ __forceinline__ void srv_plain_body(
    const uint32_t *__restrict__ packed32, const float *__restrict__ scales, int W,
    int64_t wstride, int64_t cstride, const Chunks &ch, int64_t c0, int64_t nch, int64_t word0,
    int64_t elem0, float *__restrict__ srv_err, uint32_t *__restrict__ srv_packed32,
    float *__restrict__ srv_scales, float *__restrict__ avg_out, uint8_t *__restrict__ flags,
    double inv_w, int w_pow2, float *lds)
{
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
            const At<AL> p = at<AL>(el + e, len - e);
            if (avg_out) st(avg_out, p, av);
            const f4v d = ld(srv_err, p);
            // formed in a local vector: masking b[k] in place after writing its
            // elements made this compiler drop the block's loads and adds
            f4v bk;
#pragma unroll
            for (int q = 0; q < 4; ++q) bk[q] = av[q] + d[q];
            b[k] = inside(bk, p);
        }
    }
    compress_chunk<L, V, AL>(b, lc, len, active, srv_err, el,
                             srv_packed32 + 2 * (active ? ch.word[c] : 0), srv_scales + c, lds);
    // sticky: a flag once set stays set until the handle is recreated
    const uint32_t f = inexact_flag<L>(scales + (active ? cr : 0), cstride, W, lc);
    if (active && lc == 0 && f) flags[cr] = 1;
}

template <int L, int V>
__global__ __launch_bounds__(L > 256 ? L : 256) void k_srv_plain(
    const uint32_t *__restrict__ packed32, const float *__restrict__ scales, int W,
    int64_t wstride, int64_t cstride, Chunks ch, int64_t c0, int64_t nch, int64_t word0,
    int64_t elem0, float *__restrict__ srv_err, uint32_t *__restrict__ srv_packed32,
    float *__restrict__ srv_scales, float *__restrict__ avg_out, uint8_t *__restrict__ flags,
    double inv_w, int w_pow2)
{
    __shared__ float lds[64];
    srv_plain_body<L, V, true>(packed32, scales, W, wstride, cstride, ch, c0, nch, word0, elem0,
                               srv_err, srv_packed32, srv_scales, avg_out, flags, inv_w, w_pow2,
                               lds);
}

template <int L, int V>
__global__ __launch_bounds__(L > 256 ? L : 256) void k_srv_plain_ua(
    const uint32_t *__restrict__ packed32, const float *__restrict__ scales, int W,
    int64_t wstride, int64_t cstride, Chunks ch, int64_t c0, int64_t nch, int64_t word0,
    int64_t elem0, float *__restrict__ srv_err, uint32_t *__restrict__ srv_packed32,
    float *__restrict__ srv_scales, float *__restrict__ avg_out, uint8_t *__restrict__ flags,
    double inv_w, int w_pow2)
{
    __shared__ float lds[64];
    srv_plain_body<L, V, false>(packed32, scales, W, wstride, cstride, ch, c0, nch, word0, elem0,
                                srv_err, srv_packed32, srv_scales, avg_out, flags, inv_w, w_pow2,
                                lds);
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
    compress_chunk<LD, 8, true>(bv, lc, len, active, srv_err, el,
                                srv_packed32 + 2 * (active ? ch.word[c] : 0), srv_scales + c,
                                tree);
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
                      int chunk, bool al, hipStream_t st)
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
    // the lookup tables serve aligned chunks only
    const bool lut = al && algo != SRV_PLAIN && sg.V == 1 && G <= 16 && lds <= kSrvLdsMax;
    if (!lut) {
        return with_geometry(geo, [&](auto Lc, auto Vc) {
            constexpr int L = decltype(Lc)::value, V = decltype(Vc)::value;
            auto go = [&](auto kernel) {
                hipLaunchKernelGGL(kernel, dim3(grid_for(nch, chunks_per_block<L>())),
                                   dim3(chunk_block<L>()), 0, st,
                                   reinterpret_cast<const uint32_t *>(packed), scales, W, wstride,
                                   cstride, ch, c0, nch, word0, elem0, srv_err,
                                   reinterpret_cast<uint32_t *>(srv_packed), srv_scales, avg,
                                   flags, inv_w, pow2 ? 1 : 0);
                return hipGetLastError();
            };
            return al ? go(k_srv_plain<L, V>) : go(k_srv_plain_ua<L, V>);
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

}  // namespace zo
