// zo_adam.cpp -- host side of the 0/1 Adam C ABI (include/zo_adam.h).
//
// Validates every call before launching anything, keeps the step state
// machine of Algorithm 1 (which lines of step t have run), accumulates the
// learning-rate sum Gamma of the current interval in binary32, and launches
// exactly one kernel per hot-path call on the handle's stream.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <vector>

#include "zo_adam.h"
#include "zo_internal.h"

namespace {

enum Phase {
    PH_IDLE = 0,        // expecting the first call of step t
    PH_LOCAL_SYNC = 1,  // zo_local_step ran at a sync step; compress (g = NULL) next
    PH_COMPRESSED = 2,  // worker half of Algorithm 2 done
    PH_AVERAGED = 3,    // server half done
    PH_VAR_PENDING = 4  // only the variance line of step t is left
};

constexpr int32_t kMaxChunk = 16384;
constexpr int32_t kMaxWorld = 1 << 16;

inline bool aligned(const void *p, uintptr_t a) { return ((uintptr_t)p & (a - 1)) == 0; }

bool strictly_increasing(const int64_t *v, int32_t n)
{
    for (int32_t i = 0; i < n; ++i) {
        if (v[i] < 0) return false;
        if (i && v[i] <= v[i - 1]) return false;
    }
    return true;
}

int check_segments(int32_t nseg, const int64_t *seg_off, int32_t chunk)
{
    if (nseg < 1 || !seg_off) return ZO_EINVAL;
    if (chunk < 1 || chunk > kMaxChunk) return ZO_EINVAL;
    if (seg_off[0] != 0) return ZO_EINVAL;
    for (int32_t s = 0; s < nseg; ++s)
        if (seg_off[s + 1] < seg_off[s]) return ZO_EINVAL;
    for (int32_t s = 0; s <= nseg; ++s)
        if (seg_off[s] % 4) return ZO_EALIGN;
    return ZO_OK;
}

}  // namespace

struct zo_adam {
    zo::Scalars sc{};
    int32_t world = 1, chunk = 4;
    bool al = true;  // chunk % 4 == 0: every chunk starts and ends on a float4
    int64_t n = 0, nchunks = 0, nwords = 0;
    std::vector<int64_t> hstart, hword;
    std::vector<int32_t> hlen;
    void *dtable = nullptr;
    uint8_t *dflags = nullptr;
    zo::Chunks ch{};
    zo::Geometry geo{};
    int64_t c0 = 0, c1 = 0, w0 = 0, w1 = 0, e0 = 0, e1 = 0;
    zo_state st{};
    hipStream_t stream = nullptr;
    std::vector<int64_t> tv, tu;
    int64_t t = 0;
    int phase = PH_IDLE;
    float gamma_sum = 0.0f;
    int srv_algo = zo::SRV_AUTO;
    // Deferred sync writes: the reconstruction leaves the new model only in
    // the anchor (x_in_anchor) and u = +0 implicit (u_in = U_ZERO); the first
    // local step after it writes x but leaves u = +0 + gamma m implicit too
    // (U_GM, gamma_u = its gamma), the next one writes u (or zo_materialize).
    bool defer = false, x_in_anchor = false;
    int u_in = zo::U_MEM;
    float gamma_u = 0.0f;
    // deferred mode: the copy of the last server output the momentum is
    // rebuilt from while u_in == U_ZERO (allocated with the chunk table)
    zo::SrvCopy sm{};
    // Algorithm 4 instead of Algorithm 1; fv_gamma = gamma_t of the step whose
    // compressed average zo_sync_update applies.
    bool fv = false;
    float fv_gamma = 0.0f;
    int gt = zo::GT_F32;          // element type of g and gbar
    uintptr_t galign = 16;        // their alignment: one float4 of elements
    char hip_err[192] = {0};

    // the schedules T_v and T_u: the vectors above, or a static slot's arrays
    const int64_t *tvp = nullptr, *tup = nullptr;
    int64_t ntv = 0, ntu = 0;
    // zo_adam_init_static: the device whose static slot holds this handle
    // (its chunk table, flags and server copy are in that device's scratch
    // array; no host chunk table is kept); -1 for zo_adam_init
    int slot = -1;

    bool in_tv(int64_t s) const { return std::binary_search(tvp, tvp + ntv, s); }
    bool in_tu(int64_t s) const { return std::binary_search(tup, tup + ntu, s); }

    int hip_fail(hipError_t e)
    {
        std::snprintf(hip_err, sizeof hip_err, "%s: %s", hipGetErrorName(e), hipGetErrorString(e));
        return ZO_EHIP;
    }

    // Step t is complete: advance.
    void finish_step()
    {
        phase = PH_IDLE;
        ++t;
    }
};

extern "C" {

int64_t zo_plan_num_chunks(int32_t nseg, const int64_t *seg_off, int32_t chunk)
{
    int rc = check_segments(nseg, seg_off, chunk);
    if (rc) return rc;
    int64_t total = 0;
    for (int32_t s = 0; s < nseg; ++s) total += (seg_off[s + 1] - seg_off[s] + chunk - 1) / chunk;
    return total;
}

int64_t zo_plan_chunks(int32_t nseg, const int64_t *seg_off, int32_t chunk, int64_t *start,
                       int64_t *len, int64_t *word)
{
    int rc = check_segments(nseg, seg_off, chunk);
    if (rc) return rc;
    int64_t c = 0, w = 0;
    for (int32_t s = 0; s < nseg; ++s) {
        const int64_t end = seg_off[s + 1];
        for (int64_t pos = seg_off[s]; pos < end; pos += chunk, ++c) {
            const int64_t l = std::min<int64_t>(chunk, end - pos);
            if (start) start[c] = pos;
            if (len) len[c] = l;
            if (word) word[c] = w;
            w += (l + 63) / 64;
        }
    }
    return w;
}

int zo_config_check(const zo_config *cfg)
{
    if (!cfg) return ZO_EINVAL;
    const float b1 = cfg->beta1, b2 = cfg->beta2, e = cfg->eps;
    if (!(b1 >= 0.0f && b1 < 1.0f) || !(b2 >= 0.0f && b2 < 1.0f)) return ZO_EINVAL;
    if (!(e >= 0.0f) || !std::isfinite(e)) return ZO_EINVAL;
    if (cfg->world < 1 || cfg->world > kMaxWorld) return ZO_EINVAL;
    if (cfg->n < 0) return ZO_EINVAL;
    int rc = check_segments(cfg->nseg, cfg->seg_off, cfg->chunk);
    if (rc) return rc;
    if (cfg->seg_off[cfg->nseg] != cfg->n) return ZO_EINVAL;
    if (cfg->ntv < 0 || cfg->ntu < 0) return ZO_EINVAL;
    if (cfg->ntv && (!cfg->tv || !strictly_increasing(cfg->tv, cfg->ntv))) return ZO_EINVAL;
    if (cfg->ntu && (!cfg->tu || !strictly_increasing(cfg->tu, cfg->ntu))) return ZO_EINVAL;
    if (cfg->algorithm != ZO_ALG_ZERO_ONE_ADAM && cfg->algorithm != ZO_ALG_FROZEN_VARIANCE)
        return ZO_EINVAL;
    if (cfg->algorithm == ZO_ALG_FROZEN_VARIANCE && (cfg->ntu != 0 || cfg->defer_sync_writes))
        return ZO_EINVAL;
    if (cfg->grad_dtype != ZO_DTYPE_F32 && cfg->grad_dtype != ZO_DTYPE_F16 &&
        cfg->grad_dtype != ZO_DTYPE_BF16)
        return ZO_EINVAL;
    const int64_t nch = zo_plan_num_chunks(cfg->nseg, cfg->seg_off, cfg->chunk);
    const int64_t end = cfg->srv_chunk_end < 0 ? nch : cfg->srv_chunk_end;
    if (cfg->srv_chunk_begin < 0 || cfg->srv_chunk_begin > end || end > nch) return ZO_EINVAL;
    return ZO_OK;
}

}  // extern "C"

namespace {

// The state pointers zo_adam_init requires (Algorithm 4 has no buffer u and
// no anchor), each 16-byte aligned.
int check_state(const zo_config *cfg, const zo_state *st)
{
    if (!st) return ZO_EINVAL;
    const bool fv = cfg->algorithm == ZO_ALG_FROZEN_VARIANCE;
    const float *ptrs[] = {st->x, st->m, st->v, st->err, st->srv_err, st->u, st->anchor};
    for (int i = 0; i < 7; ++i) {
        const bool needed = i < 5 || !fv;
        if (cfg->n > 0 && needed && !ptrs[i]) return ZO_EINVAL;
        if (!aligned(ptrs[i], 16)) return ZO_EALIGN;
    }
    return ZO_OK;
}

// Every field of a handle that comes from the configuration, except the
// schedules and the chunk table (no allocation).
void set_fields(zo_adam *h, const zo_config *cfg, const zo_state *st, hipStream_t stream)
{
    h->sc.b1 = cfg->beta1;
    h->sc.b2 = cfg->beta2;
    h->sc.eps = cfg->eps;
    h->sc.c1 = 1.0f - cfg->beta1;
    h->sc.c2 = 1.0f - cfg->beta2;
    h->world = cfg->world;
    h->chunk = cfg->chunk;
    h->al = cfg->chunk % 4 == 0;
    h->n = cfg->n;
    h->geo = zo::geometry_for(cfg->chunk);
    h->st = *st;
    h->stream = stream;
    h->defer = cfg->defer_sync_writes != 0;
    h->fv = cfg->algorithm == ZO_ALG_FROZEN_VARIANCE;
    h->gt = cfg->grad_dtype == ZO_DTYPE_F16 ? zo::GT_F16
            : cfg->grad_dtype == ZO_DTYPE_BF16 ? zo::GT_BF16 : zo::GT_F32;
    h->galign = h->gt == zo::GT_F32 ? 16 : 8;
    h->nchunks = zo_plan_num_chunks(cfg->nseg, cfg->seg_off, cfg->chunk);
    h->c0 = cfg->srv_chunk_begin;
    h->c1 = cfg->srv_chunk_end < 0 ? h->nchunks : cfg->srv_chunk_end;
}

// Bytes of the device block a handle uses: the chunk table (start, word,
// length), one exactness flag per server chunk and, with deferred sync
// writes, the copy of the server's packed words and scales at copy_off.
size_t device_block(const zo_adam *h, size_t &copy_off)
{
    const size_t nb = (size_t)h->nchunks;
    copy_off = (nb * (8 + 8 + 4) + (size_t)(h->c1 - h->c0) + 64 + 255) & ~(size_t)255;
    const size_t copy_bytes = h->defer ? (size_t)h->nwords * 8 + nb * 4 : 0;
    return nb ? copy_off + copy_bytes : 0;
}

// Point the handle's device views into the block at `base`.
void place_block(zo_adam *h, char *base, size_t copy_off)
{
    const size_t nb = (size_t)h->nchunks;
    h->ch.start = (const int64_t *)base;
    h->ch.word = (const int64_t *)(base + nb * 8);
    h->ch.len = (const int32_t *)(base + nb * 16);
    h->dflags = (uint8_t *)(base + nb * 20);
    if (h->defer) {
        h->sm.words32 = (uint32_t *)(base + copy_off);
        h->sm.scales = (float *)(base + copy_off + (size_t)h->nwords * 8);
    }
}

// The Require line of Algorithm 1 on the device: m = v = u = 0; errors start
// at 0 (Algorithm 2); the anchor x_{t'} with t' = 0 is x_0; flags cleared.
hipError_t start_state(zo_adam *h, hipStream_t stream)
{
    const zo_state *st = &h->st;
    if (h->nchunks > 0) {
        hipError_t e = hipMemsetAsync(h->dflags, 0, (size_t)(h->c1 - h->c0) + 1, stream);
        if (e != hipSuccess) return e;
    }
    if (h->n == 0) return hipSuccess;
    const size_t fb = (size_t)h->n * sizeof(float);
    const bool fv = h->fv;
    hipError_t es[6] = {
        hipMemsetAsync(st->m, 0, fb, stream), hipMemsetAsync(st->v, 0, fb, stream),
        fv ? hipSuccess : hipMemsetAsync(st->u, 0, fb, stream),
        hipMemsetAsync(st->err, 0, fb, stream),
        h->e1 > h->e0 ? hipMemsetAsync(st->srv_err, 0, (size_t)(h->e1 - h->e0) * 4, stream)
                      : hipSuccess,
        fv ? hipSuccess : hipMemcpyAsync(st->anchor, st->x, fb, hipMemcpyDeviceToDevice, stream)};
    for (hipError_t e : es)
        if (e != hipSuccess) return e;
    return hipSuccess;
}

// ---- handles that allocate nothing (zo_adam_init_static) ------------------
//
// One handle per device at a time.  Its chunk table, flags and (deferred sync
// writes) server copy live in `scratch`, a static device array of
// kScratchBytes that every GPU the library runs on holds until the process
// ends; the handle and its schedules live in a static host slot of that
// device.  Nothing is allocated on the host or the device.
constexpr size_t kScratchBytes = (size_t)4 << 20;
constexpr int kMaxDevices = 16;
constexpr int64_t kStaticMaxSched = 65536;
constexpr int64_t kStage = 4096;  // chunk table entries uploaded per batch

static __device__ __align__(256) uint8_t scratch[kScratchBytes];

struct StaticSlot {
    zo_adam h;
    int64_t tv[kStaticMaxSched], tu[kStaticMaxSched];
    char *dev = nullptr;  // this device's address of `scratch`
    bool live = false;
};
StaticSlot g_slots[kMaxDevices];
std::mutex g_slots_mu;                 // guards the slots and the staging arrays
int64_t g_stage_start[kStage], g_stage_word[kStage];
int32_t g_stage_len[kStage];

// Upload the chunk table of h (planned as zo_plan_chunks plans it) into its
// device block in batches through the static staging arrays, and set the
// server range's element and word bounds.  Called with g_slots_mu held.
hipError_t upload_table(zo_adam *h, const zo_config *cfg, hipStream_t stream)
{
    const size_t nb = (size_t)h->nchunks;
    char *base = (char *)h->ch.start;
    int64_t c = 0, w = 0, filled = 0, first = 0;
    h->e0 = h->e1 = h->w0 = h->w1 = 0;
    auto flush = [&]() -> hipError_t {
        if (filled == 0) return hipSuccess;
        hipError_t e = hipMemcpyAsync(base + (size_t)first * 8, g_stage_start, (size_t)filled * 8,
                                      hipMemcpyHostToDevice, stream);
        if (e == hipSuccess)
            e = hipMemcpyAsync(base + nb * 8 + (size_t)first * 8, g_stage_word,
                               (size_t)filled * 8, hipMemcpyHostToDevice, stream);
        if (e == hipSuccess)
            e = hipMemcpyAsync(base + nb * 16 + (size_t)first * 4, g_stage_len, (size_t)filled * 4,
                               hipMemcpyHostToDevice, stream);
        if (e == hipSuccess) e = hipStreamSynchronize(stream);  // the staging is reused
        first += filled;
        filled = 0;
        return e;
    };
    for (int32_t sg = 0; sg < cfg->nseg; ++sg) {
        const int64_t end = cfg->seg_off[sg + 1];
        for (int64_t pos = cfg->seg_off[sg]; pos < end; pos += cfg->chunk, ++c) {
            const int64_t l = std::min<int64_t>(cfg->chunk, end - pos);
            if (c == h->c0) {
                h->e0 = pos;
                h->w0 = w;
            }
            if (c == h->c1 - 1) {
                h->e1 = pos + l;
                h->w1 = w + (l + 63) / 64;
            }
            g_stage_start[filled] = pos;
            g_stage_word[filled] = w;
            g_stage_len[filled] = (int32_t)l;
            w += (l + 63) / 64;
            if (++filled == kStage) {
                hipError_t e = flush();
                if (e != hipSuccess) return e;
            }
        }
    }
    h->nwords = w;
    return flush();
}

}  // namespace

extern "C" {

int zo_adam_init(zo_adam **out, const zo_config *cfg, const zo_state *st, hipStream_t stream)
{
    if (!out) return ZO_EINVAL;
    *out = nullptr;
    int rc = zo_config_check(cfg);
    if (rc) return rc;
    rc = check_state(cfg, st);
    if (rc) return rc;

    zo_adam *h = new (std::nothrow) zo_adam();
    if (!h) return ZO_ENOMEM;
    set_fields(h, cfg, st, stream);
    std::vector<int64_t> len64;
    try {
        h->tv.assign(cfg->tv, cfg->tv + cfg->ntv);
        h->tu.assign(cfg->tu, cfg->tu + cfg->ntu);
        h->hstart.resize(h->nchunks);
        h->hword.resize(h->nchunks);
        h->hlen.resize(h->nchunks);
        len64.resize(h->nchunks);
    } catch (...) {
        delete h;
        return ZO_ENOMEM;
    }
    h->tvp = h->tv.data();
    h->tup = h->tu.data();
    h->ntv = cfg->ntv;
    h->ntu = cfg->ntu;
    h->nwords = zo_plan_chunks(cfg->nseg, cfg->seg_off, cfg->chunk, h->hstart.data(),
                               len64.data(), h->hword.data());
    for (int64_t c = 0; c < h->nchunks; ++c) h->hlen[c] = (int32_t)len64[c];
    if (h->c1 > h->c0) {
        h->e0 = h->hstart[h->c0];
        h->e1 = h->hstart[h->c1 - 1] + h->hlen[h->c1 - 1];
        h->w0 = h->hword[h->c0];
        h->w1 = h->hword[h->c1 - 1] + (h->hlen[h->c1 - 1] + 63) / 64;
    } else {
        h->e0 = h->e1 = h->w0 = h->w1 = 0;
    }

    // Device chunk table + per-chunk exactness flags (+ in deferred mode the
    // server-output copy: packed words and scales): the only allocations.
    const size_t nb = (size_t)h->nchunks;
    size_t copy_off = 0;
    const size_t bytes = device_block(h, copy_off);
    if (nb) {
        hipError_t e = hipMalloc(&h->dtable, bytes);
        if (e != hipSuccess) {
            (void)hipGetLastError();
            delete h;
            return e == hipErrorOutOfMemory ? ZO_ENOMEM : ZO_EHIP;
        }
        char *base = (char *)h->dtable;
        place_block(h, base, copy_off);
        hipError_t e1 = hipMemcpyAsync(base, h->hstart.data(), nb * 8, hipMemcpyHostToDevice,
                                       stream);
        hipError_t e2 = hipMemcpyAsync(base + nb * 8, h->hword.data(), nb * 8,
                                       hipMemcpyHostToDevice, stream);
        hipError_t e3 = hipMemcpyAsync(base + nb * 16, h->hlen.data(), nb * 4,
                                       hipMemcpyHostToDevice, stream);
        if (e1 || e2 || e3) {
            rc = h->hip_fail(e1 ? e1 : e2 ? e2 : e3);
            (void)hipStreamSynchronize(stream);
            (void)hipFree(h->dtable);
            delete h;
            return rc;
        }
    }
    hipError_t e = start_state(h, stream);
    if (e != hipSuccess) {
        rc = h->hip_fail(e);
        (void)hipStreamSynchronize(stream);
        if (h->dtable) (void)hipFree(h->dtable);
        delete h;
        return rc;
    }
    *out = h;
    return ZO_OK;
}

int zo_adam_init_static(zo_adam **out, const zo_config *cfg, const zo_state *st,
                        hipStream_t stream)
{
    if (!out) return ZO_EINVAL;
    *out = nullptr;
    int rc = zo_config_check(cfg);
    if (rc) return rc;
    rc = check_state(cfg, st);
    if (rc) return rc;
    if (cfg->ntv > kStaticMaxSched || cfg->ntu > kStaticMaxSched) return ZO_ESCRATCH;
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return ZO_EHIP;

    std::lock_guard<std::mutex> lock(g_slots_mu);
    StaticSlot &slot = g_slots[dev];
    if (slot.live) return ZO_ESTATE;  // one handle per device at a time
    if (!slot.dev) {
        // set-up, once per device with that device current: the device
        // address of this device's copy of `scratch` (the host-side name is
        // not a device address)
        void *p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
            (void)hipGetLastError();
            return ZO_EHIP;
        }
        slot.dev = (char *)p;
    }
    zo_adam *h = &slot.h;
    *h = zo_adam();  // a fresh handle: empty vectors, nothing allocated
    set_fields(h, cfg, st, stream);
    std::copy(cfg->tv, cfg->tv + cfg->ntv, slot.tv);
    std::copy(cfg->tu, cfg->tu + cfg->ntu, slot.tu);
    h->tvp = slot.tv;
    h->tup = slot.tu;
    h->ntv = cfg->ntv;
    h->ntu = cfg->ntu;
    h->slot = dev;
    // the word count, for the block's size (a pass over the chunks)
    int64_t words = 0;
    for (int32_t sg = 0; sg < cfg->nseg; ++sg)
        for (int64_t pos = cfg->seg_off[sg]; pos < cfg->seg_off[sg + 1]; pos += cfg->chunk)
            words += (std::min<int64_t>(cfg->chunk, cfg->seg_off[sg + 1] - pos) + 63) / 64;
    h->nwords = words;
    size_t copy_off = 0;
    if (device_block(h, copy_off) > kScratchBytes) return ZO_ESCRATCH;
    place_block(h, slot.dev, copy_off);
    hipError_t e = h->nchunks > 0 ? upload_table(h, cfg, stream) : hipSuccess;
    if (e == hipSuccess) e = start_state(h, stream);
    if (e != hipSuccess) {
        rc = h->hip_fail(e);
        (void)hipStreamSynchronize(stream);
        return rc;
    }
    slot.live = true;
    *out = h;
    return ZO_OK;
}

int zo_adam_destroy(zo_adam *h)
{
    if (!h) return ZO_EINVAL;
    int rc = ZO_OK;
    hipError_t e = hipStreamSynchronize(h->stream);
    if (e != hipSuccess) rc = h->hip_fail(e);
    if (h->slot >= 0) {
        // a static handle: its slot becomes free (nothing to free)
        std::lock_guard<std::mutex> lock(g_slots_mu);
        g_slots[h->slot].live = false;
        return rc;
    }
    if (h->dtable) {
        e = hipFree(h->dtable);
        if (e != hipSuccess && rc == ZO_OK) rc = ZO_EHIP;
    }
    delete h;
    return rc;
}

int zo_set_stream(zo_adam *h, hipStream_t stream)
{
    if (!h) return ZO_EINVAL;
    h->stream = stream;
    return ZO_OK;
}

static bool bad_gamma(float g) { return !(g > 0.0f) || !std::isfinite(g); }

int zo_local_step(zo_adam *h, int64_t t, float gamma, const void *g, const void *gbar)
{
    if (!h || h->fv) return ZO_EINVAL;
    if (h->n > 0 && !g) return ZO_EINVAL;
    if (bad_gamma(gamma)) return ZO_EINVAL;
    if (!aligned(g, h->galign) || !aligned(gbar, h->galign)) return ZO_EALIGN;
    if (h->phase != PH_IDLE || t != h->t) return ZO_ESTATE;
    const bool tu = h->in_tu(t), tv = h->in_tv(t);
    if (gbar && (!tv || tu)) return ZO_EINVAL;
    zo::Scalars s = h->sc;
    s.gamma = gamma;
    const float *x_src = h->x_in_anchor ? h->st.anchor : h->st.x;
    // u stays implicit after the first local step since a deferred reset,
    // unless a compress of u itself (the unfused sync) follows
    const bool write_u = !(h->u_in == zo::U_ZERO && !tu);
    s.gamma_u = h->gamma_u;
    hipError_t e = zo::launch_local(gbar != nullptr, h->u_in, write_u, g, h->st.m, x_src,
                                    h->st.x, h->st.v, h->st.u, gbar, h->n, s, h->gt, h->ch,
                                    h->nchunks, h->chunk, h->al, h->sm, h->stream);
    if (e != hipSuccess) return h->hip_fail(e);
    h->x_in_anchor = false;
    if (write_u) {
        h->u_in = zo::U_MEM;
    } else {
        h->u_in = zo::U_GM;
        h->gamma_u = gamma;
    }
    h->gamma_sum = h->gamma_sum + gamma;
    if (tu)
        h->phase = PH_LOCAL_SYNC;
    else if (tv && !gbar)
        h->phase = PH_VAR_PENDING;
    else
        h->finish_step();
    return ZO_OK;
}

int zo_compress_pack_ef(zo_adam *h, int64_t t, float gamma, const void *g, uint64_t *packed0,
                        float *scales0)
{
    if (!h) return ZO_EINVAL;
    if (h->nchunks > 0 && (!packed0 || !scales0)) return ZO_EINVAL;
    if (!aligned(g, h->galign)) return ZO_EALIGN;
    if (!aligned(packed0, 8) || !aligned(scales0, 4)) return ZO_EALIGN;
    if (h->fv) {
        // Algorithm 4, t outside T_v: compress the gradient itself (a = g + delta)
        if (h->n > 0 && !g) return ZO_EINVAL;
        if (bad_gamma(gamma)) return ZO_EINVAL;
        if (t != h->t || h->phase != PH_IDLE || h->in_tv(t)) return ZO_ESTATE;
        zo::Scalars s = h->sc;
        hipError_t e = zo::launch_sync1(h->geo, false, zo::U_MEM, nullptr, nullptr, g, h->st.err,
                                        h->ch, h->nchunks, packed0, scales0, s, zo::GT_F32,
                                        h->gt, h->al, h->sm, h->stream);
        if (e != hipSuccess) return h->hip_fail(e);
        h->fv_gamma = gamma;
        h->phase = PH_COMPRESSED;
        return ZO_OK;
    }
    if (t != h->t || !h->in_tu(t)) return ZO_ESTATE;
    const bool fused = g != nullptr;
    if (fused) {
        if (h->phase != PH_IDLE) return ZO_ESTATE;
        if (bad_gamma(gamma)) return ZO_EINVAL;
    } else if (h->phase != PH_LOCAL_SYNC) {
        return ZO_ESTATE;
    }
    zo::Scalars s = h->sc;
    s.gamma = fused ? gamma : 0.0f;
    s.gamma_u = h->gamma_u;
    // (after zo_local_step at this step u has been written: U_MEM on the
    // unfused path)
    hipError_t e = zo::launch_sync1(h->geo, fused, fused ? h->u_in : zo::U_MEM, g, h->st.m,
                                    h->st.u, h->st.err, h->ch, h->nchunks, packed0, scales0, s,
                                    h->gt, zo::GT_F32, h->al, h->sm, h->stream);
    if (e != hipSuccess) return h->hip_fail(e);
    if (fused) h->gamma_sum = h->gamma_sum + gamma;
    h->phase = PH_COMPRESSED;
    return ZO_OK;
}

int zo_unpack_average(zo_adam *h, int64_t t, const uint64_t *packed, const float *scales,
                      uint64_t *srv_packed, float *srv_scales, float *avg_debug)
{
    if (!h) return ZO_EINVAL;
    const int64_t nch = h->c1 - h->c0;
    if (nch > 0 && (!packed || !scales || !srv_packed || !srv_scales)) return ZO_EINVAL;
    if (!aligned(packed, 8) || !aligned(srv_packed, 8) || !aligned(scales, 4) ||
        !aligned(srv_scales, 4) || !aligned(avg_debug, 16))
        return ZO_EALIGN;
    if (t != h->t || h->phase != PH_COMPRESSED) return ZO_ESTATE;
    hipError_t e = zo::launch_srv(h->geo, h->srv_algo, packed, scales, h->world, h->w1 - h->w0,
                                  nch, h->ch, h->c0, nch, h->w0, h->e0, h->st.srv_err,
                                  srv_packed, srv_scales, avg_debug, h->dflags, h->chunk,
                                  h->al, h->stream);
    if (e != hipSuccess) return h->hip_fail(e);
    h->phase = PH_AVERAGED;
    return ZO_OK;
}

int zo_sync_update(zo_adam *h, int64_t t, const uint64_t *srv_packed, const float *srv_scales,
                   const void *gbar)
{
    if (!h) return ZO_EINVAL;
    if (h->nchunks > 0 && (!srv_packed || !srv_scales)) return ZO_EINVAL;
    if (!aligned(srv_packed, 8) || !aligned(srv_scales, 4) || !aligned(gbar, h->galign))
        return ZO_EALIGN;
    if (t != h->t || h->phase != PH_AVERAGED) return ZO_ESTATE;
    if (h->fv) {
        if (gbar) return ZO_EINVAL;
        zo::Scalars s = h->sc;
        s.gamma = h->fv_gamma;
        hipError_t e = zo::launch_fv_apply(srv_packed, srv_scales, h->ch, h->nchunks, h->st.x,
                                           h->st.m, h->st.v, s, h->chunk, h->al, h->stream);
        if (e != hipSuccess) return h->hip_fail(e);
        h->finish_step();
        return ZO_OK;
    }
    const bool tv = h->in_tv(t);
    if (gbar && !tv) return ZO_EINVAL;
    // the deferred kernel reads the anchor, which holds x_{t'} in both cases
    zo::SrvCopy sm = h->sm;
    sm.gamma_m = h->gamma_sum;
    hipError_t e = zo::launch_recon(gbar != nullptr, h->defer, srv_packed, srv_scales, h->ch,
                                    h->nchunks, h->st.m, h->st.x, h->st.v, h->st.u,
                                    h->st.anchor, gbar, h->gamma_sum, h->sc, h->gt, h->chunk,
                                    h->al, sm, h->stream);
    if (e != hipSuccess) return h->hip_fail(e);
    if (h->defer) {
        h->x_in_anchor = true;
        h->u_in = zo::U_ZERO;
        h->sm.gamma_m = h->gamma_sum;
    }
    h->gamma_sum = 0.0f;
    if (tv && !gbar)
        h->phase = PH_VAR_PENDING;
    else
        h->finish_step();
    return ZO_OK;
}

int zo_fullprec_step(zo_adam *h, int64_t t, float gamma, const void *gbar)
{
    if (!h || !h->fv) return ZO_EINVAL;
    if (h->n > 0 && !gbar) return ZO_EINVAL;
    if (bad_gamma(gamma)) return ZO_EINVAL;
    if (!aligned(gbar, h->galign)) return ZO_EALIGN;
    if (t != h->t || h->phase != PH_IDLE || !h->in_tv(t)) return ZO_ESTATE;
    zo::Scalars s = h->sc;
    s.gamma = gamma;
    hipError_t e = zo::launch_fv_full(gbar, h->st.x, h->st.m, h->st.v, h->n, s, h->gt, h->stream);
    if (e != hipSuccess) return h->hip_fail(e);
    h->finish_step();
    return ZO_OK;
}

int zo_variance_update(zo_adam *h, int64_t t, const void *gbar)
{
    if (!h || h->fv) return ZO_EINVAL;
    if (h->n > 0 && !gbar) return ZO_EINVAL;
    if (!aligned(gbar, h->galign)) return ZO_EALIGN;
    if (t != h->t || h->phase != PH_VAR_PENDING) return ZO_ESTATE;
    hipError_t e = zo::launch_var(h->st.v, gbar, h->n, h->sc, h->gt, h->stream);
    if (e != hipSuccess) return h->hip_fail(e);
    h->finish_step();
    return ZO_OK;
}

int zo_state_location(const zo_adam *h, float **x_now, int32_t *u_mode, float *u_gamma)
{
    if (!h) return ZO_EINVAL;
    if (x_now) *x_now = h->x_in_anchor ? h->st.anchor : h->st.x;
    if (u_mode) *u_mode = h->u_in;
    if (u_gamma) *u_gamma = h->u_in == zo::U_GM ? h->gamma_u : 0.0f;
    return ZO_OK;
}

int zo_read_state(zo_adam *h, int32_t which, float *out)
{
    if (!h) return ZO_EINVAL;
    if (which != ZO_STATE_X && which != ZO_STATE_M && which != ZO_STATE_U) return ZO_EINVAL;
    if (which == ZO_STATE_U && h->fv) return ZO_EINVAL;
    if (h->n > 0 && !out) return ZO_EINVAL;
    if (!aligned(out, 16)) return ZO_EALIGN;
    if (h->phase != PH_IDLE) return ZO_ESTATE;
    hipError_t e = hipSuccess;
    if (which == ZO_STATE_X) {
        e = zo::launch_copy(h->x_in_anchor ? h->st.anchor : h->st.x, out, h->n, true, h->stream);
    } else if (which == ZO_STATE_M) {
        e = h->u_in == zo::U_ZERO
                ? zo::launch_m_from_copy(out, h->ch, h->nchunks, h->chunk, h->al, h->sm,
                                         h->stream)
                : zo::launch_copy(h->st.m, out, h->n, true, h->stream);
    } else if (h->u_in == zo::U_ZERO) {
        e = zo::launch_zero(out, h->n, h->stream);
    } else if (h->u_in == zo::U_GM) {
        e = zo::launch_u_from_m(out, h->st.m, h->n, h->gamma_u, h->stream);
    } else {
        e = zo::launch_copy(h->st.u, out, h->n, true, h->stream);
    }
    return e == hipSuccess ? ZO_OK : h->hip_fail(e);
}

int zo_materialize(zo_adam *h)
{
    if (!h || h->fv) return ZO_EINVAL;
    if (h->phase != PH_IDLE) return ZO_ESTATE;
    if (h->x_in_anchor && h->n > 0) {
        hipError_t e = zo::launch_copy(h->st.anchor, h->st.x, h->n, true, h->stream);
        if (e != hipSuccess) return h->hip_fail(e);
    }
    h->x_in_anchor = false;
    if (h->u_in == zo::U_ZERO) {
        hipError_t e = zo::launch_zero(h->st.u, h->n, h->stream);
        if (e == hipSuccess)
            e = zo::launch_m_from_copy(h->st.m, h->ch, h->nchunks, h->chunk, h->al, h->sm,
                                       h->stream);
        if (e != hipSuccess) return h->hip_fail(e);
    } else if (h->u_in == zo::U_GM) {
        hipError_t e = zo::launch_u_from_m(h->st.u, h->st.m, h->n, h->gamma_u, h->stream);
        if (e != hipSuccess) return h->hip_fail(e);
    }
    h->u_in = zo::U_MEM;
    return ZO_OK;
}

int64_t zo_num_chunks(const zo_adam *h) { return h ? h->nchunks : ZO_EINVAL; }
int64_t zo_packed_words(const zo_adam *h) { return h ? h->nwords : ZO_EINVAL; }
float zo_gamma_sum(const zo_adam *h) { return h ? h->gamma_sum : 0.0f; }
int64_t zo_next_step(const zo_adam *h) { return h ? h->t : ZO_EINVAL; }

int zo_server_range(const zo_adam *h, int64_t *chunk0, int64_t *nchunks, int64_t *word0,
                    int64_t *nwords, int64_t *elem0, int64_t *nelems)
{
    if (!h) return ZO_EINVAL;
    if (chunk0) *chunk0 = h->c0;
    if (nchunks) *nchunks = h->c1 - h->c0;
    if (word0) *word0 = h->w0;
    if (nwords) *nwords = h->w1 - h->w0;
    if (elem0) *elem0 = h->e0;
    if (nelems) *nelems = h->e1 - h->e0;
    return ZO_OK;
}

int zo_chunk_table(const zo_adam *h, int64_t *start, int64_t *len, int64_t *word)
{
    if (!h) return ZO_EINVAL;
    if (h->slot >= 0) {
        // a static handle keeps its table on the device only
        const size_t nb = (size_t)h->nchunks;
        hipError_t e = hipStreamSynchronize(h->stream);
        if (e == hipSuccess && start && nb)
            e = hipMemcpy(start, h->ch.start, nb * 8, hipMemcpyDeviceToHost);
        if (e == hipSuccess && word && nb)
            e = hipMemcpy(word, h->ch.word, nb * 8, hipMemcpyDeviceToHost);
        if (e == hipSuccess && len && nb) {
            // int32 on the device: widen in place from the array's tail
            int32_t *l32 = reinterpret_cast<int32_t *>(len) + nb;
            e = hipMemcpy(l32, h->ch.len, nb * 4, hipMemcpyDeviceToHost);
            for (size_t c = 0; c < nb && e == hipSuccess; ++c) len[c] = l32[c];
        }
        return e == hipSuccess ? ZO_OK : ZO_EHIP;
    }
    for (int64_t c = 0; c < h->nchunks; ++c) {
        if (start) start[c] = h->hstart[c];
        if (len) len[c] = h->hlen[c];
        if (word) word[c] = h->hword[c];
    }
    return ZO_OK;
}

int zo_inexact_chunks(zo_adam *h, int64_t *count)
{
    if (!h || !count) return ZO_EINVAL;
    const int64_t nch = h->c1 - h->c0;
    *count = 0;
    if (nch <= 0) return ZO_OK;
    std::vector<uint8_t> f((size_t)nch);
    hipError_t e = hipMemcpyAsync(f.data(), h->dflags, (size_t)nch, hipMemcpyDeviceToHost,
                                  h->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(h->stream);
    if (e != hipSuccess) return h->hip_fail(e);
    int64_t c = 0;
    for (uint8_t v : f) c += v ? 1 : 0;
    *count = c;
    return ZO_OK;
}

const char *zo_strerror(int status)
{
    switch (status) {
    case ZO_OK: return "ok";
    case ZO_EINVAL: return "invalid argument";
    case ZO_EALIGN: return "misaligned pointer or segment offset";
    case ZO_ESTATE: return "call out of order for the current step";
    case ZO_EHIP: return "HIP runtime error";
    case ZO_ENOMEM: return "out of memory";
    case ZO_ESCRATCH:
        return "configuration exceeds the static scratch of zo_adam_init_static";
    default: return "unknown status";
    }
}

const char *zo_last_hip_error(const zo_adam *h) { return h ? h->hip_err : ""; }

int zo_diag_divsqrt(const float *a, const float *b, float *q, float *r, int64_t n,
                    hipStream_t stream)
{
    if (n < 0 || (n > 0 && (!a || !b || !q || !r))) return ZO_EINVAL;
    hipError_t e = zo::launch_divsqrt(a, b, q, r, n, stream);
    return e == hipSuccess ? ZO_OK : ZO_EHIP;
}

int zo_diag_copy(const float *src, float *dst, int64_t n, int nontemporal, hipStream_t stream)
{
    if (n < 0 || n % 4 || (n > 0 && (!src || !dst))) return ZO_EINVAL;
    if (!aligned(src, 16) || !aligned(dst, 16)) return ZO_EALIGN;
    hipError_t e = zo::launch_copy(src, dst, n, nontemporal != 0, stream);
    return e == hipSuccess ? ZO_OK : ZO_EHIP;
}

int zo_diag_server_pattern(zo_adam *h, const uint64_t *packed)
{
    if (!h) return ZO_EINVAL;
    const int64_t nch = h->c1 - h->c0;
    if (nch > 0 && !packed) return ZO_EINVAL;
    if (!aligned(packed, 8)) return ZO_EALIGN;
    // the server's one-chunk-per-workgroup shapes, aligned chunks only
    if (h->chunk <= 1024 || !h->al) return ZO_EINVAL;
    hipError_t e = zo::launch_srv_pattern(h->chunk, packed, h->world, h->w1 - h->w0, h->ch, h->c0,
                                          nch, h->w0, h->e0, h->st.srv_err, h->stream);
    return e == hipSuccess ? ZO_OK : h->hip_fail(e);
}

int zo_diag_stream(const float *const *src, int32_t nsrc, float *const *dst, int32_t ndst,
                   int64_t n, hipStream_t stream)
{
    if (nsrc < 1 || nsrc > 6 || ndst < 1 || ndst > 5 || !src || !dst) return ZO_EINVAL;
    if (n < 0 || n % 4) return ZO_EINVAL;
    zo::StreamPtrs p{};
    for (int32_t r = 0; r < nsrc; ++r) {
        if (n > 0 && !src[r]) return ZO_EINVAL;
        if (!aligned(src[r], 16)) return ZO_EALIGN;
        p.src[r] = src[r];
    }
    for (int32_t w = 0; w < ndst; ++w) {
        if (n > 0 && !dst[w]) return ZO_EINVAL;
        if (!aligned(dst[w], 16)) return ZO_EALIGN;
        for (int32_t k = 0; k < w; ++k)
            if (n > 0 && dst[k] == dst[w]) return ZO_EINVAL;  // one writer per array
        p.dst[w] = dst[w];
    }
    hipError_t e = zo::launch_stream(nsrc, ndst, p, n, stream);
    return e == hipSuccess ? ZO_OK : ZO_EHIP;
}

}  // extern "C"
