// C-ABI host side of the MTI k-means hot path: argument checks, scratch
// ownership, launch configuration, the run loop and error reporting.  The
// declarations and their contracts are in include/kmeans_mti.h.
#include <math.h>
#include <stdio.h>
#include <string.h>

#include <climits>
#include <mutex>
#include <new>

#include "kmeans_mti.h"
#include "km_internal.h"

namespace {

thread_local char g_last_hip[256] = "";

int hip_fail(hipError_t e, const char* what) {
    snprintf(g_last_hip, sizeof g_last_hip, "%s: %s (%d)", what, hipGetErrorString(e), (int)e);
    return e == hipErrorOutOfMemory ? KM_ERR_OOM : KM_ERR_HIP;
}

#define KM_HIP(call)                                  \
    do {                                              \
        hipError_t e_ = (call);                       \
        if (e_ != hipSuccess) return hip_fail(e_, #call); \
    } while (0)

int ceil_log2_u64(uint64_t v) {
    int c = 0;
    while (c < 64 && (1ull << c) < v) ++c;
    return c;
}

// Checks that [p, p + bytes) lies inside one device allocation of the
// current device, so that a host pointer or a short buffer is refused here
// instead of faulting in a kernel.
int check_device_range(const void* p, size_t bytes, int device, const char* what) {
    hipPointerAttribute_t attr;
    hipError_t e = hipPointerGetAttributes(&attr, p);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        snprintf(g_last_hip, sizeof g_last_hip, "%s is not a HIP device pointer", what);
        return KM_ERR_INVALID_ARG;
    }
    if (attr.type != hipMemoryTypeDevice && attr.type != hipMemoryTypeManaged) {
        snprintf(g_last_hip, sizeof g_last_hip, "%s is not device memory", what);
        return KM_ERR_INVALID_ARG;
    }
    if (attr.device != device) {
        snprintf(g_last_hip, sizeof g_last_hip, "%s is on device %d, current device is %d", what,
                 attr.device, device);
        return KM_ERR_INVALID_ARG;
    }
    hipDeviceptr_t base = nullptr;
    size_t size = 0;
    e = hipMemGetAddressRange(&base, &size, (hipDeviceptr_t)p);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return KM_OK;   // range unknown (e.g. managed memory): trust the caller
    }
    const uintptr_t lo = (uintptr_t)base, hi = lo + size, q = (uintptr_t)p;
    if (q < lo || q + bytes > hi) {
        snprintf(g_last_hip, sizeof g_last_hip, "%s: buffer too small (%zu bytes needed)", what,
                 bytes);
        return KM_ERR_INVALID_ARG;
    }
    return KM_OK;
}

// Device buffers of released contexts, kept per device and size for the
// next context that needs the same size: repeated runs of a problem then
// make no hipMalloc / hipFree calls (hipFree also waits for the device).
// A context returns its buffers only after its stream has drained, so a
// buffer handed out again has no work pending.  At most kCacheMax bytes are
// kept; kmeans_mti_release_cache frees them.
struct CachedBuf {
    int dev;
    size_t bytes;
    void* p;
};
constexpr size_t kCacheMax = (size_t)8 << 30;
constexpr int kCacheSlots = 256;
std::mutex g_cache_mu;
CachedBuf g_cache[kCacheSlots];
int g_cache_n = 0;
size_t g_cache_bytes = 0;

void* cache_take(int dev, size_t bytes) {
    std::lock_guard<std::mutex> lock(g_cache_mu);
    for (int i = g_cache_n - 1; i >= 0; --i)
        if (g_cache[i].dev == dev && g_cache[i].bytes == bytes) {
            void* p = g_cache[i].p;
            g_cache[i] = g_cache[--g_cache_n];
            g_cache_bytes -= bytes;
            return p;
        }
    return nullptr;
}

// Keeps p for reuse, or frees it when the cache is full.
void cache_give(int dev, size_t bytes, void* p) {
    {
        std::lock_guard<std::mutex> lock(g_cache_mu);
        if (g_cache_n < kCacheSlots && g_cache_bytes + bytes <= kCacheMax) {
            g_cache[g_cache_n++] = CachedBuf{dev, bytes, p};
            g_cache_bytes += bytes;
            return;
        }
    }
    (void)hipFree(p);
}

// Pinned host blocks (256 bytes, coherent: kernels may store to them while
// the host polls) for a run's progress word and read-backs, reused across
// runs (hipHostMalloc and hipHostFree cost tens of microseconds each).
std::mutex g_pin_mu;
int32_t* g_pin_free[64];
int g_pin_n = 0;

int32_t* pinned_take() {
    {
        std::lock_guard<std::mutex> lock(g_pin_mu);
        if (g_pin_n > 0) return g_pin_free[--g_pin_n];
    }
    void* p = nullptr;
    if (hipHostMalloc(&p, 256, hipHostMallocCoherent) != hipSuccess) return nullptr;
    return static_cast<int32_t*>(p);
}

void pinned_give(int32_t* p) {
    if (!p) return;
    {
        std::lock_guard<std::mutex> lock(g_pin_mu);
        if (g_pin_n < 64) {
            g_pin_free[g_pin_n++] = p;
            return;
        }
    }
    (void)hipHostFree(p);
}

// Launch configuration of a kernel: its dynamic-LDS limit raised to lds
// bytes and the resident blocks per CU for (block, lds), both remembered per
// device (hipFuncSetAttribute costs tens of microseconds a call).
struct KernelCfg {
    int dev;
    const void* sym;
    int block, lds, per_cu;
};
constexpr int kCfgSlots = 256;
std::mutex g_cfg_mu;
KernelCfg g_cfg[kCfgSlots];
int g_cfg_n = 0;

int kernel_config(int dev, const void* sym, int block, int lds, int* per_cu) {
    {
        std::lock_guard<std::mutex> lock(g_cfg_mu);
        for (int i = 0; i < g_cfg_n; ++i)
            if (g_cfg[i].dev == dev && g_cfg[i].sym == sym && g_cfg[i].block == block && g_cfg[i].lds == lds) {
                *per_cu = g_cfg[i].per_cu;
                return KM_OK;
            }
    }
    KM_HIP(hipFuncSetAttribute(sym, hipFuncAttributeMaxDynamicSharedMemorySize, lds));
    int pc = 0;
    KM_HIP(hipOccupancyMaxActiveBlocksPerMultiprocessor(&pc, sym, block, lds));
    std::lock_guard<std::mutex> lock(g_cfg_mu);
    if (g_cfg_n < kCfgSlots) g_cfg[g_cfg_n++] = KernelCfg{dev, sym, block, lds, pc};
    *per_cu = pc;
    return KM_OK;
}

}  // namespace

struct km_ctx {
    int64_t n = 0;
    int32_t d = 0, k = 0;
    uint32_t flags = 0;
    hipStream_t stream = nullptr;
    int device = 0;
    int tp = 0, lds = 0;
    int variant = 0;   // assignment-kernel specialisation
    bool large = false;   // global-memory path (centroids / sums too large for LDS)
    bool small = false;   // streaming step (d = 16, k <= 16)
    bool inc = false;     // ... with incremental steps after the first
    bool incmm = false;   // incremental matrix-core step (d = 16 or 32, k <= 128)
    int gim = 0, lds_im = 0;   // its grid and LDS
    int gi = 0, lds_inc = 0;   // grid and LDS of the incremental kernel
    int gf = 0, lds_first = 0;  // grid and LDS of the matrix-core first step (0: k_small runs it)
    bool fuse_scan = false;     // that first step also finds the largest |x| (no set-up scan of X)
    int64_t enq = 0;      // steps enqueued so far
    km::Fused fz{};
    km::Large lg{};
    int gb = 0;           // blocks of the large path's bound pass
    km::Dev dv{};
    static constexpr int kMaxBufs = 32;
    void* bufs[kMaxBufs] = {};
    size_t buf_bytes[kMaxBufs] = {};
    int nbufs = 0;
    bool broken = false;
    bool stepped = false;
    bool pending = false;   // streaming path: the end of the last incremental step has not run

    // KM_FLAG_TIMING: events around the four launches of each iteration,
    // harvested into per-kernel totals when the pool fills or on request.
    static constexpr int kEvIters = 256;
    bool timing = false;
    hipEvent_t ev[kEvIters][5] = {};
    int ev_used = 0;
    double t_ms[4] = {0, 0, 0, 0};
    int64_t t_iters = 0;

    // Small buffers (the per-step sums, counters, tables and state) are
    // carved from shared chunks, so that the few pages every block touches at
    // the start of a step stay few: fewer address-translation misses when all
    // blocks start at once.
    static constexpr size_t kSmallBuf = 256 << 10, kChunk = 2 << 20, kAlign = 256;
    unsigned char* chunk = nullptr;
    size_t chunk_used = 0;

    template <class T>
    int alloc(T** p, size_t count) {
        const size_t bytes = count * sizeof(T) > 0 ? count * sizeof(T) : 16;
        if (bytes <= kSmallBuf) {
            const size_t at = (chunk_used + kAlign - 1) / kAlign * kAlign;
            if (!chunk || at + bytes > kChunk) {
                void* q = nullptr;
                if (int rc = raw_alloc(&q, kChunk)) return rc;
                chunk = static_cast<unsigned char*>(q);
                chunk_used = 0;
                return alloc(p, count);
            }
            chunk_used = at + bytes;
            *p = reinterpret_cast<T*>(chunk + at);
            return KM_OK;
        }
        void* q = nullptr;
        if (int rc = raw_alloc(&q, bytes)) return rc;
        *p = static_cast<T*>(q);
        return KM_OK;
    }
    int raw_alloc(void** q, size_t bytes) {
        if (nbufs >= kMaxBufs) {
            snprintf(g_last_hip, sizeof g_last_hip, "internal: more than %d device buffers", kMaxBufs);
            return KM_ERR_STATE;
        }
        *q = cache_take(device, bytes);
        if (!*q) {
            hipError_t e = hipMalloc(q, bytes);
            if (e != hipSuccess) return hip_fail(e, "hipMalloc");
        }
        buf_bytes[nbufs] = bytes;
        bufs[nbufs++] = *q;
        return KM_OK;
    }
    ~km_ctx() {
        // Buffers go back to the cache only once no work on them is pending.
        if (hipStreamSynchronize(stream) == hipSuccess && !broken) {
            for (int i = 0; i < nbufs; ++i) cache_give(device, buf_bytes[i], bufs[i]);
        } else {
            (void)hipGetLastError();
            (void)hipDeviceSynchronize();
            for (int i = 0; i < nbufs; ++i) (void)hipFree(bufs[i]);
        }
        for (auto& row : ev)
            for (auto& e : row)
                if (e) (void)hipEventDestroy(e);
    }
};

namespace {

int fail_ctx(km_ctx* c, int rc) {
    if (c) c->broken = true;
    return rc;
}

// Accumulate the elapsed times of the recorded iterations and free the pool.
int harvest_timing(km_ctx* c) {
    if (!c->timing || c->ev_used == 0) return KM_OK;
    hipError_t e = hipEventSynchronize(c->ev[c->ev_used - 1][4]);
    if (e != hipSuccess) return fail_ctx(c, hip_fail(e, "hipEventSynchronize"));
    for (int i = 0; i < c->ev_used; ++i)
        for (int s = 0; s < 4; ++s) {
            float ms = 0.f;
            e = hipEventElapsedTime(&ms, c->ev[i][s], c->ev[i][s + 1]);
            if (e != hipSuccess) return fail_ctx(c, hip_fail(e, "hipEventElapsedTime"));
            c->t_ms[s] += ms;
        }
    c->t_iters += c->ev_used;
    c->ev_used = 0;
    return KM_OK;
}

int enqueue_iteration(km_ctx* c) {
    hipError_t e;
    hipEvent_t* ev = nullptr;
    if (c->timing) {
        if (c->ev_used == km_ctx::kEvIters) {
            int rc = harvest_timing(c);
            if (rc != KM_OK) return rc;
        }
        ev = c->ev[c->ev_used++];
    }
    auto mark = [&](int i) -> hipError_t { return ev ? hipEventRecord(ev[i], c->stream) : hipSuccess; };
    if ((e = mark(0)) != hipSuccess) return fail_ctx(c, hip_fail(e, "hipEventRecord"));
    if (c->small) {
        // Streaming step t then its end in one block; or an incremental step
        // that first ends step t - 1 itself when that has not run yet (one
        // launch per step while incremental steps follow each other).
        const int t = (int)c->enq;
        km::Dev dv = c->dv;
        dv.C64 = c->fz.c64 + (size_t)km::slot2(t) * c->k * c->d;   // C^t
        const bool inc = c->inc && t > 0;
        e = inc                 ? km::launch_inc(dv, c->fz, c->gi, c->lds_inc, t, c->pending ? 1 : 0,
                                                 t <= km::kIncDenseSteps, c->stream)
            : t == 0 && c->gf ? km::launch_first(dv, c->fz, c->gf, c->lds_first, t, c->stream)
                              : km::launch_small(dv, c->fz, c->lds, t, c->stream);
        if (e != hipSuccess) return fail_ctx(c, hip_fail(e, "streaming step kernel"));
        if (t == 0 && c->gf && c->fuse_scan && (e = km::launch_first_fix(dv, c->fz, c->gf, c->stream)) != hipSuccess)
            return fail_ctx(c, hip_fail(e, "first step correction kernel"));
        if ((e = mark(1)) != hipSuccess || (e = mark(2)) != hipSuccess)
            return fail_ctx(c, hip_fail(e, "hipEventRecord"));
        if (!inc && (e = km::launch_small_finish(dv, c->fz, t, 0, c->stream)) != hipSuccess)
            return fail_ctx(c, hip_fail(e, "streaming step finish kernel"));
        c->pending = inc;
        ++c->enq;
        if ((e = mark(3)) != hipSuccess || (e = mark(4)) != hipSuccess)
            return fail_ctx(c, hip_fail(e, "hipEventRecord"));
        c->stepped = true;
        return KM_OK;
    }
    e = c->incmm   ? km::launch_inc_mm(c->dv, c->gim, c->lds_im, c->enq == 0 ? 1 : 0, c->stream)
        : c->large ? km::launch_large_assign(c->dv, c->lg, c->gb, c->stream)
                   : km::launch_assign(c->dv, c->variant, c->tp, c->lds, c->stream);
    if (e != hipSuccess) return fail_ctx(c, hip_fail(e, "assign kernel"));
    if ((e = mark(1)) != hipSuccess) return fail_ctx(c, hip_fail(e, "hipEventRecord"));
    e = c->large ? km::launch_large_reduce(c->dv, c->lg, c->stream) : km::launch_reduce(c->dv, c->stream);
    if (e != hipSuccess) return fail_ctx(c, hip_fail(e, "reduce kernel"));
    if ((e = mark(2)) != hipSuccess) return fail_ctx(c, hip_fail(e, "hipEventRecord"));
    if ((e = km::launch_update(c->dv, c->stream)) != hipSuccess)
        return fail_ctx(c, hip_fail(e, "update kernel"));
    if ((e = mark(3)) != hipSuccess) return fail_ctx(c, hip_fail(e, "hipEventRecord"));
    e = c->large ? km::launch_large_table(c->dv, c->lg, 0, c->stream)
                 : km::launch_centroid_table(c->dv, 0, c->stream);
    if (e != hipSuccess) return fail_ctx(c, hip_fail(e, "centroid table kernel"));
    if ((e = mark(4)) != hipSuccess) return fail_ctx(c, hip_fail(e, "hipEventRecord"));
    ++c->enq;
    c->stepped = true;
    return KM_OK;
}

// Streaming path: enqueue the end of the last step if it has not run (its
// results are about to be read).
int flush_pending(km_ctx* c) {
    if (!c->pending) return KM_OK;
    const int t = (int)c->enq - 1;
    km::Dev dv = c->dv;
    dv.C64 = c->fz.c64 + (size_t)km::slot2(t) * c->k * c->d;
    hipError_t e = km::launch_small_finish(dv, c->fz, t, 1, c->stream);
    if (e != hipSuccess) return fail_ctx(c, hip_fail(e, "streaming step finish kernel"));
    c->pending = false;
    return KM_OK;
}

int read_state(km_ctx* c, km::IterState* out) {
    int rc = flush_pending(c);
    if (rc != KM_OK) return rc;
    hipError_t e = hipStreamSynchronize(c->stream);
    if (e != hipSuccess) return fail_ctx(c, hip_fail(e, "hipStreamSynchronize"));
    e = hipMemcpy(out, c->dv.st, sizeof(km::IterState), hipMemcpyDeviceToHost);
    if (e != hipSuccess) return fail_ctx(c, hip_fail(e, "hipMemcpy state"));
    return KM_OK;
}

// Set-up of a context.  max_iters / tol_n: the stop rule written into the
// loop state; sync: wait for the set-up work before returning.
int init_impl(km_ctx* c, const float* X, int64_t n, int32_t d, int32_t k, const float* C0, int32_t max_iters,
              double tol_n, bool sync, int32_t* host_word) {
    KM_HIP(hipGetDevice(&c->device));
    km::ZeroRanges zr{};   // buffers cleared by the set-up launch
    int rc0;
    if ((rc0 = check_device_range(X, (size_t)n * (size_t)d * sizeof(float), c->device, "X")) != KM_OK)
        return rc0;
    if ((rc0 = check_device_range(C0, (size_t)k * (size_t)d * sizeof(float), c->device, "C0")) != KM_OK)
        return rc0;

    // Spherical k-means: the context works on its own copy of X projected to
    // the unit sphere (X itself is only read here).
    if (c->flags & KM_FLAG_SPHERICAL) {
        float* Xn = nullptr;
        int rcn;
        if ((rcn = c->alloc(&Xn, (size_t)n * (size_t)d))) return rcn;
        KM_HIP(km::launch_normalize_rows(X, n, d, Xn, c->stream));
        X = Xn;
    }

    int cus = 0, max_lds = 0;
    KM_HIP(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, c->device));
    KM_HIP(hipDeviceGetAttribute(&max_lds, hipDeviceAttributeMaxSharedMemoryPerBlock, c->device));

    km::Dev& v = c->dv;
    v.X = X;
    v.n = n;
    v.d = d;
    v.k = k;
    v.L = km::row_len(d, k);
    v.flags = c->flags;
    v.gamma = (float)((d + 4) * 0x1p-23);
    int rc2;

    // LDS path: the largest tile of 256/128/64 points whose LDS image
    // (centroids, fixed-point sums, X tile) fits; else the global-memory path.
    c->tp = 0;
    const bool aligned = reinterpret_cast<uintptr_t>(X) % 16 == 0;
    const bool elkan = (c->flags & KM_FLAG_ELKAN) != 0;
    if (elkan && (c->flags & KM_FLAG_LARGE_PATH)) return KM_ERR_INVALID_ARG;
    if (!elkan && !(c->flags & (KM_FLAG_LARGE_PATH | KM_FLAG_GENERIC)) && km::small_applies(n, d, k, aligned)) {
        c->small = true;
        c->tp = km::kSmallTile;
        c->lds = km::small_lds_bytes(k);
        if (c->lds > max_lds || km::small_finish_lds_bytes(k) > max_lds) return KM_ERR_UNSUPPORTED;
        const void* sym = km::small_kernel_symbol(k);
        int per_cu = 0, rcc;
        if ((rcc = kernel_config(c->device, sym, c->tp, c->lds, &per_cu)) != KM_OK) return rcc;
        if (per_cu < 1) return KM_ERR_UNSUPPORTED;
        const int64_t ntiles = (n + c->tp - 1) / c->tp;
        int64_t G = (int64_t)per_cu * cus;
        if (G > ntiles) G = ntiles;
        v.G = (int32_t)G;
        c->inc = !(c->flags & (KM_FLAG_FULL_SUMS | KM_FLAG_STATS));
        if (!(c->flags & KM_FLAG_STATS)) {
            // The first step on the matrix cores (no inertia to sum): resident
            // blocks, at most one 64-point tile per wave.
            c->lds_first = km::first_lds_bytes(k);
            int per_cu_f = 0;
            if (c->lds_first > max_lds) return KM_ERR_UNSUPPORTED;
            if ((rcc = kernel_config(c->device, km::first_kernel_symbol(k), c->tp, c->lds_first, &per_cu_f)) != KM_OK)
                return rcc;
            if (per_cu_f < 1) return KM_ERR_UNSUPPORTED;
            const int64_t want = ((n + 63) / 64 + 3) / 4;
            int64_t gf = (int64_t)per_cu_f * cus;
            if (gf > want) gf = want > 0 ? want : 1;
            c->gf = (int)gf;
        }
        if (c->inc) {
            c->lds_inc = km::inc_lds_bytes(k);
            if (c->lds_inc > max_lds) return KM_ERR_UNSUPPORTED;
            int per_cu_i = 0, per_cu_d = 0;
            if ((rcc = kernel_config(c->device, km::inc_kernel_symbol(k, false), km::kIncThreads, c->lds_inc,
                                     &per_cu_i)) != KM_OK ||
                (rcc = kernel_config(c->device, km::inc_kernel_symbol(k, true), km::kIncThreads, c->lds_inc,
                                     &per_cu_d)) != KM_OK)
                return rcc;
            if (per_cu_d < per_cu_i) per_cu_i = per_cu_d;   // one grid for both forms
            if (per_cu_i < 1) return KM_ERR_UNSUPPORTED;
            // Resident blocks (the same count on every CU), at least one wave
            // tile per wave; small inputs still spread over up to one block
            // per CU (one tile per block), which shortens each block's chain
            // of dependent tiles.
            const int64_t nwt = (n + km::kIncWaveTile - 1) / km::kIncWaveTile;
            int64_t gi = (int64_t)per_cu_i * cus;
            const int64_t spread = nwt < cus ? nwt : cus;
            const int64_t want = nwt / km::kIncWaves > spread ? nwt / km::kIncWaves : spread;
            if (gi > want) gi = want > 0 ? want : 1;
            c->gi = (int)gi;
        }
    } else if (!elkan && !(c->flags & (KM_FLAG_LARGE_PATH | KM_FLAG_GENERIC | KM_FLAG_VECTOR_ONLY | KM_FLAG_STATS |
                                         KM_FLAG_FULL_SUMS | KM_FLAG_NO_PRUNE)) &&
               km::inc_mm_applies(n, d, k, aligned) && km::inc_mm_lds(d, km::inc_mm_kb(k)).bytes <= max_lds) {
        // Incremental matrix-core step: only the Clause-1 survivors' rows are read.
        c->incmm = true;
        c->lds_im = km::inc_mm_lds(d, km::inc_mm_kb(k)).bytes;
        const void* sym = km::inc_mm_symbol(d, k);
        int per_cu = 0, rcc;
        if ((rcc = kernel_config(c->device, sym, km::kIMWaves * 64, c->lds_im, &per_cu)) != KM_OK) return rcc;
        if (per_cu < 1) return KM_ERR_UNSUPPORTED;
        // Resident blocks, at most one wave tile per wave.
        const int64_t nwt = (n + km::kIMTile - 1) / km::kIMTile;
        int64_t G = (int64_t)per_cu * cus;
        const int64_t want = (nwt + km::kIMWaves - 1) / km::kIMWaves;
        if (G > want) G = want > 0 ? want : 1;
        c->gim = (int)G;
        v.G = (int32_t)G;
    } else if (!(c->flags & KM_FLAG_LARGE_PATH)) {
        c->variant = km::assign_variant(d, k, aligned, (c->flags & KM_FLAG_VECTOR_ONLY) != 0, elkan);
        const bool h_lds = km::assign_h_lds(c->variant % 16, k);
        const bool wide = km::assign_wide(c->variant);   // blocks of 512 threads only
        for (int tp = wide ? 512 : 256; c->tp == 0 && tp >= (wide ? 512 : 64); tp /= 2) {
            int bytes = km::assign_lds(d, k, tp, h_lds, wide).bytes;
            if (bytes <= max_lds) {
                c->tp = tp;
                c->lds = bytes;
            }
        }
    }
    if (c->small || c->incmm) {
        // configured above
    } else if (c->tp > 0) {
        const void* sym = km::assign_kernel_symbol(c->variant);
        int per_cu = 0, rcc;
        if ((rcc = kernel_config(c->device, sym, c->tp, c->lds, &per_cu)) != KM_OK) return rcc;
        if (per_cu < 1) return KM_ERR_UNSUPPORTED;
        const int64_t ntiles = (n + c->tp - 1) / c->tp;
        int64_t G = (int64_t)per_cu * cus;
        if (G > ntiles) G = ntiles;
        v.G = (int32_t)G;
    } else if (elkan) {
        snprintf(g_last_hip, sizeof g_last_hip, "Elkan's lower bounds need the centroids and sums in LDS");
        return KM_ERR_UNSUPPORTED;
    } else {
        c->large = true;
        km::Large& L = c->lg;
        const int mlds = km::large_mfma_lds();
        if (d > km::kLgMaxD || mlds > max_lds || 4 * k > max_lds || km::large_table_lds(d) > max_lds) {
            snprintf(g_last_hip, sizeof g_last_hip,
                     "k = %d, d = %d: no kernel path (d <= %d and k <= %d needed)", k, d, km::kLgMaxD,
                     max_lds / 4);
            return KM_ERR_UNSUPPORTED;
        }
        const void* sym = km::large_mfma_symbol();
        KM_HIP(km::large_set_attributes(k, d));
        int per_cu = 0;
        KM_HIP(hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, sym, 256, mlds));
        if (per_cu < 1) return KM_ERR_UNSUPPORTED;
        L.Gm = per_cu * cus;
        L.Gr = 4 * cus;
        L.nch = km::split_chunks(d);
        L.nct = (k + km::kLgN - 1) / km::kLgN;
        L.mvcap = (int32_t)(n / 16 > 1024 ? n / 16 : (n < 1024 ? n : 1024));
        int64_t gs = (n + 4095) / 4096;
        if (gs > 2048) gs = 2048;
        L.Gs = (int32_t)gs;
        L.span = (n + gs - 1) / gs;
        L.NCmax = (int32_t)(n / km::kLgChunkRows + k + 1);
        const int64_t gb = (n + km::kLgBoundSpan - 1) / km::kLgBoundSpan;   // one block per span of points
        if (gb > INT_MAX) return KM_ERR_INVALID_ARG;
        c->gb = (int)gb;
        v.G = 1;
        if ((rc2 = c->alloc(&L.surv, (size_t)n)) || (rc2 = c->alloc(&L.nsurv, 4)) ||
            (rc2 = c->alloc(&L.cnt, (size_t)L.Gs * k)) || (rc2 = c->alloc(&L.off, (size_t)L.Gs * k)) ||
            (rc2 = c->alloc(&L.base, (size_t)k + 1)) || (rc2 = c->alloc(&L.cbase, (size_t)k + 1)) ||
            (rc2 = c->alloc(&L.perm, (size_t)n)) || (rc2 = c->alloc(&L.cpart, (size_t)L.NCmax * d)) ||
            (rc2 = c->alloc(&L.ciq, (size_t)L.NCmax)) ||
            (rc2 = c->alloc(&L.xs, (size_t)n * L.nch * 16)) || (rc2 = c->alloc(&L.x2, (size_t)n)) ||
            (rc2 = c->alloc(&L.sx2, (size_t)n)) || (rc2 = c->alloc(&L.fq, (size_t)n)) ||
            (rc2 = c->alloc(&L.nfull, 4)) || (rc2 = c->alloc(&L.nmv, 4)) || (rc2 = c->alloc(&L.nmq, 4)) ||
            (rc2 = c->alloc(&L.mq, (size_t)n)) || (rc2 = c->alloc(&L.fpart, (size_t)km::kFullCap * km::kFullSplit)) ||
            (rc2 = c->alloc(&L.fcnt, (size_t)km::kFullCap)) ||
            (rc2 = c->alloc(&L.mv, (size_t)L.mvcap)) || (rc2 = c->alloc(&v.sums, (size_t)k * d + k)) ||
            (rc2 = c->alloc(&L.cs, (size_t)L.nct * km::kLgN * L.nch * 16)) ||
            (rc2 = c->alloc(&L.cn2p, (size_t)L.nct * km::kLgN)) || (rc2 = c->alloc(&L.smin, (size_t)km::kLgTableSplit * k)) ||
            (rc2 = c->alloc(&L.cand, (size_t)n * L.nct * 8)))
            return rc2;
        zr.add(L.nsurv, 4 * sizeof(uint32_t));
        zr.add(L.nfull, 4 * sizeof(uint32_t));
        zr.add(L.nmv, 4 * sizeof(uint32_t));
        zr.add(L.nmq, 4 * sizeof(uint32_t));
        zr.add(L.fcnt, sizeof(uint32_t) * (size_t)km::kFullCap);
        zr.add(v.sums, sizeof(uint64_t) * ((size_t)k * d + k));
    }

    int rc;
    if (!c->small && !c->incmm && ((rc = c->alloc(&v.a, (size_t)n)) || (rc = c->alloc(&v.u, (size_t)n))))
        return rc;
    if (c->incmm) {   // point states padded to whole wave tiles, running sums, cumulative drifts
        const size_t nw = (size_t)((n + km::kIMTile - 1) / km::kIMTile) * km::kIMTile;
        if ((rc = c->alloc(&v.w, nw)) || (rc = c->alloc(&v.sums, (size_t)k * d + k)) ||
            (rc = c->alloc(&v.dhi, (size_t)k)) || (rc = c->alloc(&v.dlo, (size_t)k)) ||
            (rc = c->alloc(&v.dupf, (size_t)k)) || (rc = c->alloc(&v.ddnf, (size_t)k)) ||
            (rc = c->alloc(&v.hm, (size_t)4 * k)))
            return rc;
        const size_t n4 = (size_t)n & ~(size_t)3;   // states are written by the first step; padding cleared
        zr.add(v.w + n4, sizeof(uint32_t) * (nw - n4));
        zr.add(v.sums, sizeof(uint64_t) * ((size_t)k * d + k));
        zr.add(v.dhi, sizeof(double) * (size_t)k);
        zr.add(v.dlo, sizeof(double) * (size_t)k);
        zr.add(v.dupf, sizeof(float) * (size_t)k);
        zr.add(v.ddnf, sizeof(float) * (size_t)k);
    }
    if (elkan) {   // O(nk) lower bounds (zero: valid before any distance is known)
        if ((uint64_t)n > (uint64_t)INT64_MAX / 4 / (uint64_t)k) return KM_ERR_INVALID_ARG;
        if ((rc = c->alloc(&v.lb, (size_t)n * (size_t)k)) || (rc = c->alloc(&v.dhi, (size_t)k)) ||
            (rc = c->alloc(&v.dlo, (size_t)k)) || (rc = c->alloc(&v.dupf, (size_t)k)))
            return rc;
        zr.add(v.dupf, sizeof(float) * (size_t)k);
        zr.add(v.lb, sizeof(float) * (size_t)n * (size_t)k);
        zr.add(v.dhi, sizeof(double) * (size_t)k);
        zr.add(v.dlo, sizeof(double) * (size_t)k);
    }
    // The streaming path keeps C^t in two slots (t % 2); slot 0 holds C0.
    if ((rc = c->alloc(&v.C64, (size_t)k * d * (c->small ? 2 : 1))) || (rc = c->alloc(&v.C32, (size_t)k * d)) ||
        (rc = c->alloc(&v.ec, (size_t)k)) || (rc = c->alloc(&v.h, (size_t)k * k)) ||
        (rc = c->alloc(&v.s, (size_t)k)) || (rc = c->alloc(&v.f, (size_t)k)) ||
        (rc = c->alloc(&v.cn2, (size_t)k)) ||
        (rc = c->alloc(&v.part, (size_t)v.G * v.L)) || (rc = c->alloc(&v.total, (size_t)v.L)) ||
        (rc = c->alloc(&v.st, 1)) || (rc = c->alloc(&v.rec, (size_t)km::kHistCap)))
        return rc;
    if (c->small) {
        // Point states padded to whole incremental tiles (the padding stays zero).
        const size_t nw = (size_t)((n + km::kIncTile - 1) / km::kIncTile) * km::kIncTile;
        c->fz.c64 = v.C64;
        const size_t nrows = (size_t)3 * km::kSmallRows * v.L;
        if ((rc = c->alloc(&c->fz.rows, nrows)) || (rc = c->alloc(&c->fz.stat, 3 * km::kNumStat)) ||
            (rc = c->alloc(&c->fz.sum, (size_t)2 * (k * d + k))) || (rc = c->alloc(&c->fz.w, nw)) ||
            (rc = c->alloc(&c->fz.dhi, (size_t)2 * k)) || (rc = c->alloc(&c->fz.dlo, (size_t)2 * k)) ||
            (rc = c->alloc(&c->fz.dup, (size_t)k)) || (rc = c->alloc(&c->fz.ddn, (size_t)k)))
            return rc;
        zr.add(c->fz.rows, sizeof(uint64_t) * nrows);
        zr.add(c->fz.stat, sizeof(uint64_t) * 3 * km::kNumStat);
        zr.add(c->fz.sum, sizeof(uint64_t) * 2 * (size_t)(k * d + k));
        // The first step writes every point's state; only the padding (read,
        // never used) is cleared.
        const size_t n4 = (size_t)n & ~(size_t)3;
        zr.add(c->fz.w + n4, sizeof(uint32_t) * (nw - n4));
        zr.add(c->fz.dhi, sizeof(double) * 2 * (size_t)k);
        zr.add(c->fz.dlo, sizeof(double) * 2 * (size_t)k);
        zr.add(c->fz.dup, sizeof(float) * (size_t)k);
        zr.add(c->fz.ddn, sizeof(float) * (size_t)k);
    }
    uint32_t* scratch = nullptr;
    if ((rc = c->alloc(&scratch, 8))) return rc;
    zr.add(scratch, 8 * sizeof(uint32_t));
    zr.add(v.total, sizeof(uint64_t) * (size_t)v.L);
    zr.add(v.rec, sizeof(km::IterRec) * km::kHistCap);
    zr.st = v.st;
    zr.max_iters = max_iters;
    zr.tol_n = tol_n;
    zr.host = host_word;
    KM_HIP(km::launch_init_buffers(zr, cus, c->stream));

    // Largest magnitude of X (and non-finite detection), of C0 and of a fixed
    // sample of X -> fixed-point scales; with spherical k-means also the unit
    // centroids and whether C0 has a zero row.  The matrix-core first step of
    // the stream path reads every row anyway: there it finds the largest |x|
    // itself and X is not scanned here (not with KM_FLAG_VALIDATE, whose check
    // needs it before any step, nor with spherical k-means; nor below
    // kFuseScanMin values, where the scan costs less than the correction
    // kernel's launch).
    c->fuse_scan = c->gf && n * d >= km::kFuseScanMin && !(c->flags & (KM_FLAG_VALIDATE | KM_FLAG_SPHERICAL));
    if (c->small) c->fz.amax = c->fuse_scan ? scratch : nullptr;
    KM_HIP(km::launch_absmax(X, c->fuse_scan ? 0 : n * d, C0, (int64_t)k * d, X, n, d, cus, scratch, c->stream));
    if (c->flags & KM_FLAG_SPHERICAL)
        KM_HIP(km::launch_set_centroids_unit(C0, v.C64, v.C32, v.ec, k, d, reinterpret_cast<int32_t*>(scratch + 4),
                                             c->stream));
    // Fixed-point scales: computed on the device from the largest |x| (the
    // host does not wait for them).  Only the checks that decide the call's
    // status read the set-up back: non-finite input (KM_FLAG_VALIDATE) and a
    // zero C0 row (spherical k-means).
    KM_HIP(km::launch_set_scales(v.st, scratch, n, d, (c->flags & KM_FLAG_SPHERICAL) ? 1 : 0, c->stream));
    if (c->flags & (KM_FLAG_VALIDATE | KM_FLAG_SPHERICAL)) {
        uint32_t host[5];
        int32_t* pin = pinned_take();
        if (!pin) return KM_ERR_OOM;
        hipError_t ec5 = hipMemcpyAsync(pin, scratch, sizeof host, hipMemcpyDeviceToHost, c->stream);
        if (ec5 == hipSuccess) ec5 = hipStreamSynchronize(c->stream);
        if (ec5 == hipSuccess) memcpy(host, pin, sizeof host);
        pinned_give(pin);
        if (ec5 != hipSuccess) return hip_fail(ec5, "set-up read-back");
        if ((c->flags & KM_FLAG_VALIDATE) && (host[1] || host[3])) return KM_ERR_NONFINITE;
        if (host[4]) {
            snprintf(g_last_hip, sizeof g_last_hip, "spherical k-means: C0 has a zero row");
            return KM_ERR_INVALID_ARG;
        }
    }

    if (c->flags & KM_FLAG_TIMING) {
        c->timing = true;
        for (auto& row : c->ev)
            for (auto& e : row) KM_HIP(hipEventCreate(&e));
    }

    if (!(c->flags & KM_FLAG_SPHERICAL))
        KM_HIP(km::launch_set_centroids(C0, v.C64, v.C32, v.ec, (int64_t)k * d, k, c->stream));
    if (c->large) {
        KM_HIP(km::launch_large_table(v, c->lg, 1, c->stream));
        KM_HIP(km::launch_large_split_x(v, c->lg, cus, c->stream));
    } else {
        KM_HIP(km::launch_centroid_table(v, 1, c->stream));
    }
    if (sync) KM_HIP(hipStreamSynchronize(c->stream));
    return KM_OK;
}

int check_shape(const float* X, int64_t n, int32_t d, int32_t k, const float* C0) {
    if (!X || !C0 || n < 1 || d < 1 || k < 1 || k > n) return KM_ERR_INVALID_ARG;
    if (n > INT64_MAX / 4 / d) return KM_ERR_INVALID_ARG;                     // n*d*4 overflow
    if ((int64_t)k * d + k + km::kNumStat > INT_MAX / 8) return KM_ERR_INVALID_ARG;
    return KM_OK;
}

// Workspace of kmeans_pp_seed: 256-byte aligned segments.
struct PPLayout {
    size_t d2, a, bs, mb, dcc, cnt, u, idx, total;
};

PPLayout pp_layout(int64_t n, int32_t k) {
    auto up = [](size_t v) { return (v + 255) & ~(size_t)255; };
    const size_t G = (size_t)((n + km::kPPChunk - 1) / km::kPPChunk);
    PPLayout L{};
    size_t o = 0;
    L.d2 = o;  o += up((size_t)n * 8);
    L.a = o;   o += up((size_t)n * 4);
    L.bs = o;  o += up(G * 8);
    L.mb = o;  o += up((size_t)k * 8);
    L.dcc = o; o += up((size_t)k * 8);
    L.cnt = o; o += up((size_t)k * 16);
    L.u = o;   o += up((size_t)k * 8);
    L.idx = o; o += up((size_t)k * 8);
    L.total = o;
    return L;
}

// Static workspace of kmeans_pp_seed_noalloc: one array per device, allocated
// with the code object when the library loads on that device and held until
// the process ends.  Host code never passes the array's name to a kernel or
// a copy (on the host it is a stand-in, not a device address): the device
// address is looked up once per device with hipGetSymbolAddress and kept.
__device__ __align__(256) unsigned char pp_scratch[KMEANS_PP_STATIC_WORKSPACE_BYTES];

constexpr int kMaxDevices = 256;
void* g_pp_scratch_addr[kMaxDevices] = {};
std::mutex g_pp_scratch_mu;

int pp_static_workspace(void** out) {
    int dev = 0;
    KM_HIP(hipGetDevice(&dev));
    if (dev < 0 || dev >= kMaxDevices) return KM_ERR_UNSUPPORTED;
    std::lock_guard<std::mutex> lock(g_pp_scratch_mu);
    if (!g_pp_scratch_addr[dev]) {
        void* p = nullptr;
        KM_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(pp_scratch)));
        if (!p || (reinterpret_cast<uintptr_t>(p) & 255)) {
            snprintf(g_last_hip, sizeof g_last_hip, "static workspace: unexpected device address");
            return KM_ERR_HIP;
        }
        g_pp_scratch_addr[dev] = p;
    }
    *out = g_pp_scratch_addr[dev];
    return KM_OK;
}

}  // namespace

extern "C" {

// A new context; max_iters / tol_n: its stop rule; sync: wait for the set-up;
// host_word (nullable, device address of pinned host memory): the progress
// word the ends of steps write.
static int create_ctx(km_ctx** out, const float* X, int64_t n, int32_t d, int32_t k, const float* C0,
                      void* hip_stream, uint32_t flags, int32_t max_iters, double tol_n, bool sync,
                      int32_t* host_word = nullptr) {
    if (!out) return KM_ERR_INVALID_ARG;
    *out = nullptr;
    int rc = check_shape(X, n, d, k, C0);
    if (rc != KM_OK) return rc;
    if (flags & ~(uint32_t)(KM_FLAG_NO_PRUNE | KM_FLAG_STATS | KM_FLAG_VALIDATE | KM_FLAG_TIMING |
                            KM_FLAG_VECTOR_ONLY | KM_FLAG_LARGE_PATH | KM_FLAG_GENERIC |
                            KM_FLAG_FULL_SUMS | KM_FLAG_SPHERICAL | KM_FLAG_ELKAN))
        return KM_ERR_INVALID_ARG;
    km_ctx* c = new (std::nothrow) km_ctx;
    if (!c) return KM_ERR_OOM;
    c->n = n;
    c->d = d;
    c->k = k;
    c->flags = flags;
    c->stream = static_cast<hipStream_t>(hip_stream);
    rc = init_impl(c, X, n, d, k, C0, max_iters, tol_n, sync, host_word);
    if (rc != KM_OK) {
        delete c;
        return rc;
    }
    *out = c;
    return KM_OK;
}

int kmeans_mti_init(km_ctx** out, const float* X, int64_t n, int32_t d, int32_t k, const float* C0,
                    void* hip_stream, uint32_t flags) {
    return create_ctx(out, X, n, d, k, C0, hip_stream, flags, INT_MAX, -1.0, true);
}

int kmeans_mti_iterate(km_ctx* ctx, int64_t* changed_out) {
    if (!ctx) return KM_ERR_INVALID_ARG;
    if (ctx->broken) return KM_ERR_STATE;
    int rc = enqueue_iteration(ctx);
    if (rc != KM_OK) return rc;
    if (changed_out) {
        km::IterState st;
        if ((rc = read_state(ctx, &st)) != KM_OK) return rc;
        *changed_out = st.changed_last;
    }
    return KM_OK;
}

// kmeans_mti_get once the output ranges are checked.
static int get_outputs(km_ctx* ctx, int32_t* assign_out, float* C_out) {
    int rc;
    if ((rc = flush_pending(ctx)) != KM_OK) return rc;
    hipError_t e;
    if (assign_out && ctx->small &&
        (e = km::launch_small_unpack(ctx->fz, ctx->n, assign_out, ctx->stream)) != hipSuccess)
        return fail_ctx(ctx, hip_fail(e, "assignment unpack kernel"));
    if (assign_out && ctx->incmm && (e = km::launch_inc_mm_unpack(ctx->dv, assign_out, ctx->stream)) != hipSuccess)
        return fail_ctx(ctx, hip_fail(e, "assignment unpack kernel"));
    if (assign_out && !ctx->small && !ctx->incmm &&
        (e = hipMemcpyAsync(assign_out, ctx->dv.a, (size_t)ctx->n * sizeof(int32_t),
                            hipMemcpyDeviceToDevice, ctx->stream)) != hipSuccess)
        return fail_ctx(ctx, hip_fail(e, "hipMemcpyAsync assign"));
    if (C_out &&
        (e = hipMemcpyAsync(C_out, ctx->dv.C32, (size_t)ctx->k * ctx->d * sizeof(float),
                            hipMemcpyDeviceToDevice, ctx->stream)) != hipSuccess)
        return fail_ctx(ctx, hip_fail(e, "hipMemcpyAsync centroids"));
    return KM_OK;
}

int kmeans_mti_get(km_ctx* ctx, int32_t* assign_out, float* C_out) {
    if (!ctx) return KM_ERR_INVALID_ARG;
    if (ctx->broken) return KM_ERR_STATE;
    if (assign_out && !ctx->stepped) return KM_ERR_STATE;
    int rc;
    if (assign_out &&
        (rc = check_device_range(assign_out, (size_t)ctx->n * 4, ctx->device, "assign_out")) != KM_OK)
        return rc;
    if (C_out && (rc = check_device_range(C_out, (size_t)ctx->k * ctx->d * 4, ctx->device, "C_out")) !=
                     KM_OK)
        return rc;
    return get_outputs(ctx, assign_out, C_out);
}

int kmeans_mti_get_centroids64(km_ctx* ctx, double* C_out) {
    if (!ctx || !C_out) return KM_ERR_INVALID_ARG;
    if (ctx->broken) return KM_ERR_STATE;
    km::IterState st;
    int rc = read_state(ctx, &st);   // ends the last step, synchronizes
    if (rc != KM_OK) return rc;
    const double* src = ctx->small ? ctx->fz.c64 + (size_t)km::slot2(st.t) * ctx->k * ctx->d : ctx->dv.C64;
    hipError_t e = hipMemcpy(C_out, src, (size_t)ctx->k * ctx->d * sizeof(double), hipMemcpyDeviceToHost);
    if (e != hipSuccess) return fail_ctx(ctx, hip_fail(e, "hipMemcpy centroids"));
    return KM_OK;
}

static void fill_stats(const km_ctx* c, const km::IterState& st, km_stats* s) {
    s->iterations = st.t;
    s->converged = st.converged;
    s->changed_last = st.changed_last;
    s->dist_computed = st.tot_computed;
    s->dist_lloyd = c->n * (int64_t)c->k * st.t;
    s->clause1_skips = st.tot_clause1;
    s->rechecks = st.tot_rechecks;
    s->inertia_last = (c->flags & KM_FLAG_STATS) && st.t > 0 ? st.inertia_last : NAN;
    s->device_ms = 0.0;
}

int kmeans_mti_get_stats(km_ctx* ctx, km_stats* stats) {
    if (!ctx || !stats) return KM_ERR_INVALID_ARG;
    if (ctx->broken) return KM_ERR_STATE;
    km::IterState st;
    int rc = read_state(ctx, &st);
    if (rc != KM_OK) return rc;
    fill_stats(ctx, st, stats);
    return KM_OK;
}

int kmeans_mti_get_history(km_ctx* ctx, int64_t* changed, int64_t* computed, int64_t* clause1,
                           int64_t* rechecks, double* inertia, int32_t cap) {
    if (!ctx || cap < 0) return KM_ERR_INVALID_ARG;
    if (ctx->broken) return KM_ERR_STATE;
    km::IterState st;
    int rc = read_state(ctx, &st);
    if (rc != KM_OK) return rc;
    int m = st.t < cap ? st.t : cap;
    if (m > km::kHistCap) m = km::kHistCap;
    if (m == 0) return 0;
    km::IterRec* rec = new (std::nothrow) km::IterRec[km::kHistCap];
    if (!rec) return KM_ERR_OOM;
    hipError_t e = hipMemcpy(rec, ctx->dv.rec, sizeof(km::IterRec) * km::kHistCap, hipMemcpyDeviceToHost);
    if (e != hipSuccess) {
        delete[] rec;
        return fail_ctx(ctx, hip_fail(e, "hipMemcpy history"));
    }
    for (int i = 0; i < m; ++i) {
        const km::IterRec& r = rec[(st.t - m + i) % km::kHistCap];
        if (changed) changed[i] = r.changed;
        if (computed) computed[i] = r.computed;
        if (clause1) clause1[i] = r.clause1;
        if (rechecks) rechecks[i] = r.rechecks;
        if (inertia) inertia[i] = (ctx->flags & KM_FLAG_STATS) ? r.inertia : NAN;
    }
    delete[] rec;
    return m;
}

int kmeans_mti_get_timing(km_ctx* ctx, double* ms, int64_t* iters) {
    if (!ctx || !ms) return KM_ERR_INVALID_ARG;
    if (ctx->broken) return KM_ERR_STATE;
    if (!ctx->timing) return KM_ERR_STATE;
    int rc = harvest_timing(ctx);
    if (rc != KM_OK) return rc;
    for (int s = 0; s < 4; ++s) ms[s] = ctx->t_ms[s];
    if (iters) *iters = ctx->t_iters;
    return KM_OK;
}

int kmeans_mti_run(const float* X, int64_t n, int32_t d, int32_t k, const float* C0, int32_t max_iters,
                   double tol, int32_t* assign_out, float* C_out, void* hip_stream, uint32_t flags,
                   km_stats* stats) {
    if (max_iters < 1 || !(tol >= 0.0) || !assign_out || !C_out) return KM_ERR_INVALID_ARG;
    int rc = check_shape(X, n, d, k, C0);
    if (rc != KM_OK) return rc;
    int dev = 0;
    hipError_t e0 = hipGetDevice(&dev);
    if (e0 != hipSuccess) return hip_fail(e0, "hipGetDevice");
    if ((rc = check_device_range(assign_out, (size_t)n * 4, dev, "assign_out")) != KM_OK) return rc;
    if ((rc = check_device_range(C_out, (size_t)k * d * 4, dev, "C_out")) != KM_OK) return rc;
    // The progress word: pinned host memory that the end of every step sets
    // (steps ended, negated at the stop), polled below.
    int32_t* pinned = pinned_take();
    if (!pinned) return KM_ERR_OOM;
    volatile int32_t* word = pinned;
    word[0] = 0;
    int32_t* word_dev = nullptr;
    hipError_t eh = hipHostGetDevicePointer(reinterpret_cast<void**>(&word_dev), pinned, 0);
    if (eh != hipSuccess) {
        pinned_give(pinned);
        return hip_fail(eh, "hipHostGetDevicePointer");
    }
    km_ctx* c = nullptr;
    if ((rc = create_ctx(&c, X, n, d, k, C0, hip_stream, flags, max_iters, tol * (double)n, false, word_dev)) !=
        KM_OK) {
        pinned_give(pinned);
        return rc;
    }

    hipEvent_t ev0 = nullptr, ev1 = nullptr;
    float ms = 0.f;
    auto cleanup = [&]() {
        if (ev0) (void)hipEventDestroy(ev0);
        if (ev1) (void)hipEventDestroy(ev1);
        kmeans_mti_destroy(c);   // waits for the stream: no kernel writes the word afterwards
        pinned_give(pinned);
    };
#define RUN_HIP(call)                                   \
    do {                                                \
        hipError_t e_ = (call);                         \
        if (e_ != hipSuccess) {                         \
            int r_ = hip_fail(e_, #call);               \
            cleanup();                                  \
            return r_;                                  \
        }                                               \
    } while (0)

    RUN_HIP(hipEventCreate(&ev0));
    RUN_HIP(hipEventCreate(&ev1));

    // Keep kAhead steps enqueued past the last one whose end the device has
    // reported (on the streaming path a step's end runs at the start of the
    // next launch); the device stop flag makes launches past the stop return
    // at once, so at most kAhead - 1 are enqueued past convergence.  While
    // waiting, the stream is queried now and then, so that an error ends the
    // wait; an idle stream whose steps reported nothing new is an error too.
    constexpr int kAhead = 2;   // measured best: fewer launches past the stop outweigh the bubbles
    RUN_HIP(hipEventRecord(ev0, c->stream));
    int enq = 0;
    while (enq < max_iters) {
        const int32_t v = word[0];
        if (v < 0) break;
        if (enq < v + kAhead) {
            if ((rc = enqueue_iteration(c)) != KM_OK) {
                cleanup();
                return rc;
            }
            ++enq;
            continue;
        }
        bool stalled = false;
        for (int spin = 1; word[0] == v; ++spin) {
            if ((spin & 1023) == 0) {
                const hipError_t q = hipStreamQuery(c->stream);
                if (q == hipSuccess) {
                    stalled = word[0] == v;
                    break;
                }
                if (q != hipErrorNotReady) RUN_HIP(q);
            }
        }
        if (stalled) {
            snprintf(g_last_hip, sizeof g_last_hip, "run loop: the steps ended without reporting progress");
            cleanup();
            return KM_ERR_STATE;
        }
    }
    RUN_HIP(hipEventRecord(ev1, c->stream));
    if ((rc = get_outputs(c, assign_out, C_out)) != KM_OK) {   // ranges checked on entry
        cleanup();
        return rc;
    }
    // The loop state after the last step, read back with the outputs' stream
    // work (one wait for both).
    km::IterState st;
    static_assert(sizeof(km::IterState) <= 256 - 64, "loop state fits the pinned block");
    km::IterState* pst = reinterpret_cast<km::IterState*>(reinterpret_cast<char*>(pinned) + 64);
    RUN_HIP(hipMemcpyAsync(pst, c->dv.st, sizeof(km::IterState), hipMemcpyDeviceToHost, c->stream));
    RUN_HIP(hipStreamSynchronize(c->stream));
    memcpy(&st, pst, sizeof st);
    RUN_HIP(hipEventElapsedTime(&ms, ev0, ev1));
    if (stats) {
        fill_stats(c, st, stats);
        stats->device_ms = ms;
    }
    cleanup();
    return KM_OK;
#undef RUN_HIP
}

size_t kmeans_pp_workspace_bytes(int64_t n, int32_t d, int32_t k) {
    if (n < 1 || d < 1 || k < 1 || k > n || n > INT64_MAX / 16 / d) return 0;
    return pp_layout(n, k).total;
}

// kmeans_pp_seed on a given workspace; own_ws: the workspace is the
// library's static array (its range is known, not looked up).
static int pp_seed_impl(const float* X, int64_t n, int32_t d, int32_t k, const double* u, float* C_out,
                        int64_t* idx_out, double* d2_out, void* workspace, size_t workspace_bytes, uint32_t flags,
                        void* hip_stream, km_pp_stats* stats, bool own_ws) {
    if (!X || !u || !C_out || !workspace || n < 1 || d < 1 || k < 1 || k > n || n > INT64_MAX / 16 / d)
        return KM_ERR_INVALID_ARG;
    if (flags & ~(uint32_t)(KM_PP_NO_PRUNE | KM_PP_TIMING)) return KM_ERR_INVALID_ARG;
    if ((n + km::kPPChunk - 1) / km::kPPChunk > INT_MAX) return KM_ERR_INVALID_ARG;
    for (int32_t t = 0; t < k; ++t)
        if (!(u[t] >= 0.0 && u[t] < 1.0)) {
            snprintf(g_last_hip, sizeof g_last_hip, "u[%d] is not in [0, 1)", (int)t);
            return KM_ERR_INVALID_ARG;
        }
    const PPLayout L = pp_layout(n, k);
    if (workspace_bytes < L.total || ((uintptr_t)workspace & 255)) {
        snprintf(g_last_hip, sizeof g_last_hip, "workspace: %zu bytes, 256-byte aligned, needed", L.total);
        return KM_ERR_INVALID_ARG;
    }
    int dev = 0, rc;
    KM_HIP(hipGetDevice(&dev));
    if ((rc = check_device_range(X, (size_t)n * d * 4, dev, "X")) != KM_OK) return rc;
    if ((rc = check_device_range(C_out, (size_t)k * d * 4, dev, "C_out")) != KM_OK) return rc;
    if (!own_ws && (rc = check_device_range(workspace, L.total, dev, "workspace")) != KM_OK) return rc;
    if (idx_out && (rc = check_device_range(idx_out, (size_t)k * 8, dev, "idx_out")) != KM_OK) return rc;
    if (d2_out && (rc = check_device_range(d2_out, (size_t)n * 8, dev, "d2_out")) != KM_OK) return rc;
    hipStream_t st = static_cast<hipStream_t>(hip_stream);
    char* ws = static_cast<char*>(workspace);

    km::PPArgs P{};
    P.X = X;
    P.n = n;
    P.d = d;
    P.k = k;
    P.C = C_out;
    P.idx = reinterpret_cast<int64_t*>(ws + L.idx);
    P.u = reinterpret_cast<const double*>(ws + L.u);
    P.D2 = reinterpret_cast<double*>(ws + L.d2);
    P.A = reinterpret_cast<int32_t*>(ws + L.a);
    P.bs = reinterpret_cast<uint64_t*>(ws + L.bs);
    P.Mb = reinterpret_cast<uint64_t*>(ws + L.mb);
    P.dcc = reinterpret_cast<double*>(ws + L.dcc);
    P.cnt = stats ? reinterpret_cast<uint64_t*>(ws + L.cnt) : nullptr;
    P.G = (int32_t)((n + km::kPPChunk - 1) / km::kPPChunk);
    P.L = ceil_log2_u64((uint64_t)n);
    P.prune = (flags & KM_PP_NO_PRUNE) ? 0 : 1;
    const bool vec4 = d % 4 == 0 && ((uintptr_t)X & 15) == 0 && ((uintptr_t)C_out & 15) == 0;
    const int vw = vec4 ? (d % 32 == 0 && d >= 64 ? 2 : 1) : 0;

    int64_t i0 = (int64_t)(u[0] * (double)n);   // first seed: uniform
    if (i0 > n - 1) i0 = n - 1;
    KM_HIP(hipMemcpyAsync(ws + L.u, u, (size_t)k * 8, hipMemcpyHostToDevice, st));
    if (!stats) {
        KM_HIP(km::launch_pp_seed(P, i0, vw, nullptr, nullptr, st));
        if (idx_out) KM_HIP(hipMemcpyAsync(idx_out, P.idx, (size_t)k * 8, hipMemcpyDeviceToDevice, st));
        if (d2_out) KM_HIP(hipMemcpyAsync(d2_out, P.D2, (size_t)n * 8, hipMemcpyDeviceToDevice, st));
        return KM_OK;
    }
    // With stats: counters (and with KM_PP_TIMING events around every
    // launch), then one synchronisation.  Host memory released on every path.
    const int nev = (flags & KM_PP_TIMING) ? km::pp_launches(k, d, P.prune != 0) + 1 : 0;
    hipEvent_t* ev = nev ? new (std::nothrow) hipEvent_t[nev]() : nullptr;
    int8_t* kind = nev ? new (std::nothrow) int8_t[nev]() : nullptr;
    uint64_t* h = new (std::nothrow) uint64_t[2 * (size_t)k];
    auto release = [&]() {
        for (int j = 0; ev && j < nev; ++j)
            if (ev[j]) (void)hipEventDestroy(ev[j]);
        delete[] ev;
        delete[] kind;
        delete[] h;
    };
    if (!h || (nev && (!ev || !kind))) {
        release();
        return KM_ERR_OOM;
    }
    hipError_t e = hipSuccess;
    for (int j = 0; j < nev && e == hipSuccess; ++j) e = hipEventCreate(&ev[j]);
    if (e == hipSuccess) e = km::launch_pp_seed(P, i0, vw, ev, kind, st);
    if (e == hipSuccess && idx_out) e = hipMemcpyAsync(idx_out, P.idx, (size_t)k * 8, hipMemcpyDeviceToDevice, st);
    if (e == hipSuccess && d2_out) e = hipMemcpyAsync(d2_out, P.D2, (size_t)n * 8, hipMemcpyDeviceToDevice, st);
    if (e == hipSuccess) e = hipMemcpyAsync(h, P.cnt, (size_t)k * 16, hipMemcpyDeviceToHost, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    km_pp_stats out{};
    out.passes = k;
    for (int32_t t = 0; t < k && e == hipSuccess; ++t) {
        out.computed += (int64_t)h[2 * t];
        if (t > 0) out.improved += (int64_t)h[2 * t + 1];
    }
    for (int j = 0; j + 1 < nev && e == hipSuccess; ++j) {
        float ms = 0.f;
        e = hipEventElapsedTime(&ms, ev[j], ev[j + 1]);
        if (kind[j] != 2) out.pass_ms += ms;
        if (kind[j] == 1) out.later_pass_ms += ms;
        if (kind[j] == 2) out.draw_ms += ms;
    }
    release();
    if (e != hipSuccess) return hip_fail(e, "kmeans_pp_seed");
    *stats = out;
    return KM_OK;
}

int kmeans_pp_seed(const float* X, int64_t n, int32_t d, int32_t k, const double* u, float* C_out,
                   int64_t* idx_out, double* d2_out, void* workspace, size_t workspace_bytes, uint32_t flags,
                   void* hip_stream, km_pp_stats* stats) {
    return pp_seed_impl(X, n, d, k, u, C_out, idx_out, d2_out, workspace, workspace_bytes, flags, hip_stream,
                        stats, false);
}

int kmeans_pp_seed_noalloc(const float* X, int64_t n, int32_t d, int32_t k, const double* u, float* C_out,
                           int64_t* idx_out, double* d2_out, uint32_t flags, void* hip_stream) {
    if (!X || !u || !C_out || n < 1 || d < 1 || k < 1 || k > n) return KM_ERR_INVALID_ARG;
    if (flags & ~(uint32_t)KM_PP_NO_PRUNE) {   // KM_PP_TIMING would create events
        snprintf(g_last_hip, sizeof g_last_hip, "kmeans_pp_seed_noalloc: only KM_PP_NO_PRUNE is accepted");
        return KM_ERR_INVALID_ARG;
    }
    const size_t need = kmeans_pp_workspace_bytes(n, d, k);
    if (need == 0) return KM_ERR_INVALID_ARG;
    if (need > KMEANS_PP_STATIC_WORKSPACE_BYTES) {
        snprintf(g_last_hip, sizeof g_last_hip,
                 "kmeans_pp_seed_noalloc: n = %lld, k = %d need %zu workspace bytes, more than the %zu of the "
                 "static workspace", (long long)n, (int)k, need, (size_t)KMEANS_PP_STATIC_WORKSPACE_BYTES);
        return KM_ERR_INVALID_ARG;
    }
    void* ws = nullptr;
    const int rc = pp_static_workspace(&ws);
    if (rc != KM_OK) return rc;
    return pp_seed_impl(X, n, d, k, u, C_out, idx_out, d2_out, ws, KMEANS_PP_STATIC_WORKSPACE_BYTES, flags,
                        hip_stream, nullptr, true);
}

int kmeans_pp_run_best(const float* X, int64_t n, int32_t d, int32_t k, const double* U, int32_t r,
                       int32_t max_iters, double tol, int32_t* assign_out, float* C_out, void* hip_stream,
                       uint32_t flags, int32_t* best_out, double* inertia_out, km_stats* stats) {
    if (!U || r < 1 || max_iters < 1 || !(tol >= 0.0) || !assign_out || !C_out) return KM_ERR_INVALID_ARG;
    int rc = check_shape(X, n, d, k, X);
    if (rc != KM_OK) return rc;
    if ((int64_t)r > INT64_MAX / k) return KM_ERR_INVALID_ARG;
    for (int64_t j = 0; j < (int64_t)r * k; ++j)
        if (!(U[j] >= 0.0 && U[j] < 1.0)) {
            snprintf(g_last_hip, sizeof g_last_hip, "U[%lld] is not in [0, 1)", (long long)j);
            return KM_ERR_INVALID_ARG;
        }
    const size_t wsb = kmeans_pp_workspace_bytes(n, d, k);
    if (wsb == 0) return KM_ERR_INVALID_ARG;
    int dev = 0;
    KM_HIP(hipGetDevice(&dev));
    if ((rc = check_device_range(assign_out, (size_t)n * 4, dev, "assign_out")) != KM_OK) return rc;
    if ((rc = check_device_range(C_out, (size_t)k * d * 4, dev, "C_out")) != KM_OK) return rc;
    hipStream_t st = static_cast<hipStream_t>(hip_stream);
    // One allocation: seeding workspace | seeds | spare assignment | spare centroids.
    auto up = [](size_t v) { return (v + 255) & ~(size_t)255; };
    const size_t o_seed = up(wsb), o_a = o_seed + up((size_t)k * d * 4), o_c = o_a + up((size_t)n * 4);
    const size_t total = o_c + up((size_t)k * d * 4);
    char* buf = nullptr;
    KM_HIP(hipMalloc(reinterpret_cast<void**>(&buf), total));
    float* seeds = reinterpret_cast<float*>(buf + o_seed);
    int32_t* spare_a = reinterpret_cast<int32_t*>(buf + o_a);
    float* spare_c = reinterpret_cast<float*>(buf + o_c);
    const uint32_t ppf = (flags & KM_FLAG_NO_PRUNE) ? KM_PP_NO_PRUNE : 0u;
    int32_t best = -1;
    km_stats best_st{};
    for (int32_t q = 0; q < r && rc == KM_OK; ++q) {
        rc = kmeans_pp_seed(X, n, d, k, U + (int64_t)q * k, seeds, nullptr, nullptr, buf, wsb, ppf, hip_stream,
                            nullptr);
        if (rc != KM_OK) break;
        // The first run writes the outputs directly; later runs write the
        // spare buffers, copied over the outputs when they are better.
        int32_t* a_dst = q == 0 ? assign_out : spare_a;
        float* c_dst = q == 0 ? C_out : spare_c;
        km_stats s{};
        rc = kmeans_mti_run(X, n, d, k, seeds, max_iters, tol, a_dst, c_dst, hip_stream, flags | KM_FLAG_STATS, &s);
        if (rc != KM_OK) break;
        if (inertia_out) inertia_out[q] = s.inertia_last;
        if (best < 0 || s.inertia_last < best_st.inertia_last) {
            best = q;
            best_st = s;
            if (q > 0) {
                hipError_t e = hipMemcpyAsync(assign_out, spare_a, (size_t)n * 4, hipMemcpyDeviceToDevice, st);
                if (e == hipSuccess)
                    e = hipMemcpyAsync(C_out, spare_c, (size_t)k * d * 4, hipMemcpyDeviceToDevice, st);
                if (e == hipSuccess) e = hipStreamSynchronize(st);
                if (e != hipSuccess) rc = hip_fail(e, "kmeans_pp_run_best copy");
            }
        }
    }
    (void)hipStreamSynchronize(st);
    hipError_t ef = hipFree(buf);
    if (rc != KM_OK) return rc;
    if (ef != hipSuccess) return hip_fail(ef, "hipFree");
    if (best_out) *best_out = best;
    if (stats) *stats = best_st;
    return KM_OK;
}

const char* kmeans_mti_path(const km_ctx* ctx) {
    if (!ctx) return "";
    if (ctx->small) return ctx->inc ? "stream-d16" : "stream-d16-full";
    if (ctx->large) return "global-mfma";
    if (ctx->incmm) return "lds-inc";
    if (ctx->variant % 16 == 8) return "lds-elkan";
    return ctx->variant % 16 ? "lds-mfma" : "lds-vector";
}

void kmeans_mti_destroy(km_ctx* ctx) { delete ctx; }

void kmeans_mti_release_cache(void) {
    CachedBuf held[kCacheSlots];
    int m = 0;
    {
        std::lock_guard<std::mutex> lock(g_cache_mu);
        for (int i = 0; i < g_cache_n; ++i) held[m++] = g_cache[i];
        g_cache_n = 0;
        g_cache_bytes = 0;
    }
    for (int i = 0; i < m; ++i) (void)hipFree(held[i].p);
}

const char* kmeans_mti_strerror(int status) {
    switch (status) {
        case KM_OK: return "ok";
        case KM_ERR_INVALID_ARG: return "invalid argument";
        case KM_ERR_OOM: return "out of memory";
        case KM_ERR_HIP: return "HIP runtime error";
        case KM_ERR_UNSUPPORTED: return "unsupported shape";
        case KM_ERR_STATE: return "context unusable";
        case KM_ERR_NONFINITE: return "non-finite input";
        default: return "unknown status";
    }
}

const char* kmeans_mti_last_hip_error(void) { return g_last_hip; }

}  // extern "C"
