// synth.hip -- seeded synthetic inputs for the 0/1 Adam tests and benchmark.
//
// Holds none of the optimizer's arithmetic.  Every value is a pure function of
// (seed, stream, step, index), computed with integer operations and at most two
// IEEE binary32 multiplies, so the host fill and the device fill give the same
// bits: the oracle (host) and the HIP library (device) see identical inputs
// without copying full shards between them.
//
// Hash: the SplitMix64 output function (Steele, Lea and Flood, "Fast
// splittable pseudorandom number generators", OOPSLA 2014) applied to
// key + (index + 1) * golden-gamma, i.e. the index-th output of a SplitMix64
// stream whose state starts at `key`.
//
// Approximate normal: Irwin-Hall sum of the four 16-bit lanes of one hash,
// centred (mean 4 * 32767.5 = 131070) and scaled by sigma / sqrt(4 * var)
// where var = (65536^2 - 1) / 12 is the variance of one uniform 16-bit lane.
// The integer is exact in binary32 (|z| < 2^24), so one multiply rounds.
// Outliers: a second hash selects an element with probability per_mille/1000,
// whose value is then multiplied by `factor`.
#include <hip/hip_runtime.h>
#include <stdint.h>

#define ZS_GOLDEN 0x9E3779B97F4A7C15ull
#define ZS_OUTLIER_SALT 0xD1B54A32D192ED03ull

__host__ __device__ static inline uint64_t zs_mix(uint64_t z)
{
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

__host__ __device__ static inline uint64_t zs_hash(uint64_t key, uint64_t idx)
{
    return zs_mix(key + (idx + 1u) * ZS_GOLDEN);
}

__host__ __device__ static inline float zs_normal(uint64_t key, uint64_t idx, float ksigma,
                                                  uint32_t per_mille, float factor)
{
    uint64_t h = zs_hash(key, idx);
    int32_t z = (int32_t)(h & 0xFFFFu) + (int32_t)((h >> 16) & 0xFFFFu) +
                (int32_t)((h >> 32) & 0xFFFFu) + (int32_t)((h >> 48) & 0xFFFFu) - 131070;
    float val = (float)z * ksigma;
    if (per_mille) {
        uint64_t h2 = zs_mix(h ^ ZS_OUTLIER_SALT);
        if ((uint32_t)(h2 % 1000u) < per_mille) val = val * factor;
    }
    return val;
}

__host__ __device__ static inline float zs_scale(uint64_t key, uint64_t idx, float base)
{
    uint64_t h = zs_hash(key, idx);
    float f = 0.5f + (float)(uint32_t)(h >> 40) * 0x1p-24f;  // [0.5, 1.5)
    return base * f;
}

extern "C" {

// Key of one (seed, stream, step) triple.
uint64_t zs_key(uint64_t seed, uint32_t stream, int64_t step)
{
    uint64_t k = zs_mix(seed + ZS_GOLDEN);
    k = zs_mix(k ^ ((uint64_t)stream * 0xA0761D6478BD642Full));
    k = zs_mix(k ^ ((uint64_t)step * 0xE7037ED1A0B428DBull));
    return k;
}

// ---------------------------------------------------------------- host fills
void zs_fill_normal_host(float *out, int64_t n, int64_t idx0, uint64_t key, float ksigma,
                         uint32_t per_mille, float factor)
{
    for (int64_t i = 0; i < n; ++i)
        out[i] = zs_normal(key, (uint64_t)(idx0 + i), ksigma, per_mille, factor);
}

void zs_fill_bits_host(uint64_t *out, int64_t nwords, int64_t word0, uint64_t key)
{
    for (int64_t i = 0; i < nwords; ++i) out[i] = zs_hash(key, (uint64_t)(word0 + i));
}

void zs_fill_scales_host(float *out, int64_t n, int64_t idx0, uint64_t key, float base)
{
    for (int64_t i = 0; i < n; ++i) out[i] = zs_scale(key, (uint64_t)(idx0 + i), base);
}

// The same fills over several index ranges [idx0[r], idx0[r] + len[r]), written
// back to back into `out` (one call for a sample of scattered chunks).
void zs_fill_normal_host_ranges(float *out, int64_t nranges, const int64_t *idx0,
                                const int64_t *len, uint64_t key, float ksigma,
                                uint32_t per_mille, float factor)
{
    for (int64_t r = 0; r < nranges; ++r) {
        zs_fill_normal_host(out, len[r], idx0[r], key, ksigma, per_mille, factor);
        out += len[r];
    }
}

void zs_fill_bits_host_ranges(uint64_t *out, int64_t nranges, const int64_t *word0,
                              const int64_t *nwords, uint64_t key)
{
    for (int64_t r = 0; r < nranges; ++r) {
        zs_fill_bits_host(out, nwords[r], word0[r], key);
        out += nwords[r];
    }
}

void zs_fill_scales_host_ranges(float *out, int64_t nranges, const int64_t *idx0,
                                const int64_t *len, uint64_t key, float base)
{
    for (int64_t r = 0; r < nranges; ++r) {
        zs_fill_scales_host(out, len[r], idx0[r], key, base);
        out += len[r];
    }
}

}  // extern "C"

// -------------------------------------------------------------- device fills
__global__ void zs_normal_kernel(float *out, int64_t n, int64_t idx0, uint64_t key, float ksigma,
                                 uint32_t per_mille, float factor)
{
    int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
        out[i] = zs_normal(key, (uint64_t)(idx0 + i), ksigma, per_mille, factor);
}

__global__ void zs_bits_kernel(uint64_t *out, int64_t nwords, int64_t word0, uint64_t key)
{
    int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nwords; i += stride)
        out[i] = zs_hash(key, (uint64_t)(word0 + i));
}

__global__ void zs_scales_kernel(float *out, int64_t n, int64_t idx0, uint64_t key, float base)
{
    int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
        out[i] = zs_scale(key, (uint64_t)(idx0 + i), base);
}

static unsigned zs_grid(int64_t n)
{
    int64_t blocks = (n + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    if (blocks < 1) blocks = 1;
    return (unsigned)blocks;
}

extern "C" {

// Device fills: asynchronous on `stream`; return a hipError_t value.
int zs_fill_normal_dev(float *out, int64_t n, int64_t idx0, uint64_t key, float ksigma,
                       uint32_t per_mille, float factor, hipStream_t stream)
{
    if (n <= 0) return 0;
    hipLaunchKernelGGL(zs_normal_kernel, dim3(zs_grid(n)), dim3(256), 0, stream, out, n, idx0,
                       key, ksigma, per_mille, factor);
    return (int)hipGetLastError();
}

int zs_fill_bits_dev(uint64_t *out, int64_t nwords, int64_t word0, uint64_t key, hipStream_t stream)
{
    if (nwords <= 0) return 0;
    hipLaunchKernelGGL(zs_bits_kernel, dim3(zs_grid(nwords)), dim3(256), 0, stream, out, nwords,
                       word0, key);
    return (int)hipGetLastError();
}

int zs_fill_scales_dev(float *out, int64_t n, int64_t idx0, uint64_t key, float base,
                       hipStream_t stream)
{
    if (n <= 0) return 0;
    hipLaunchKernelGGL(zs_scales_kernel, dim3(zs_grid(n)), dim3(256), 0, stream, out, n, idx0,
                       key, base);
    return (int)hipGetLastError();
}

}  // extern "C"
