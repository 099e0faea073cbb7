// Streaming MTI iteration for small k (k <= 16) and d = 16: two launches per
// merged ||Lloyd's step (paper section III-B).
//
// k_small streams X once in 256-point tiles (persistent blocks, one tile
// prefetched into registers), and per tile
//   1. updates every point's bound with the drift of its cluster and applies
//      Clause 1 (section III-C, Table I);
//   2. adds every point to the fixed-point sums of its PREVIOUS cluster
//      (no dependence on the distance work, so it overlaps the stream);
//   3. compacts the Clause-1 survivors into a queue; a tile with many
//      survivors gives each one lane that scans the centroids in index order,
//      skipping a centroid for the whole wave when Clause 2 (u <= h(a, c),
//      Elkan's lemma) holds for every lane; a tile with few gives each
//      survivor a group of G >= k lanes, lane j evaluating centroid j unless
//      Clause 2 skips it, and the group takes the minimum with the oracle's
//      tie rule and the second-best value with DPP row reductions; near ties
//      are decided in float64;
//   4. moves a point whose assignment changed from its old cluster's sums to
//      the new one (exact integer subtraction and addition, one coordinate
//      per lane of the group).
// The block's sums are integers, so their order does not matter; each block
// adds its row into one of kSmallRows accumulation rows with device atomics.
// k_small_finish (one block) then adds those rows, forms the new centroids
// (member means; an empty cluster keeps its centroid), the drift f(c), the
// stop test and the centroid table h, s(c) for the next step (sections III-C
// and IV-A), and clears the rows.  No block waits for another and no fence
// is needed inside a kernel: the launch boundary orders the two.
#include <float.h>
#include <limits.h>
#include <math.h>

#include "kmeans_mti.h"
#include "km_device.h"
#include "km_internal.h"

namespace km {

extern __shared__ __align__(16) unsigned char km_smem[];

namespace {

constexpr int kTp = kSmallTile;    // points per tile = threads per block
constexpr int kCopies = kSmallCopies;
constexpr int kFinishThreads = 256;   // threads of the finishing block
constexpr int kLaneScanMin = 32;      // more survivors per tile: one lane per survivor

template <int D>
__device__ inline float sqd_row(const float (&x)[D], const float* c) {
    float acc = 0.f;
#pragma unroll
    for (int m = 0; m < D; m += 4) {
        const f32x4 cv = *reinterpret_cast<const f32x4*>(c + m);
        const float t0 = x[m] - cv.x, t1 = x[m + 1] - cv.y, t2 = x[m + 2] - cv.z, t3 = x[m + 3] - cv.w;
        acc = fmaf(t0, t0, acc);
        acc = fmaf(t1, t1, acc);
        acc = fmaf(t2, t2, acc);
        acc = fmaf(t3, t3, acc);
    }
    return acc;
}

// Float64 decision of a near tie against the master centroids, with the
// oracle's rule: the incumbent keeps exact ties, then the lowest index wins.
// Returns the winner; Db and ub become its squared distance and distance
// bound.
__device__ inline int recheck64(const float* x, const double* C64, int d, int k, int inc, float& Db,
                                 float& ub) {
    int bb = -1;
    double Dbb = INFINITY;
    auto dist = [&](int j) {
        double acc = 0.0;
        for (int m = 0; m < d; ++m) {
            const double t = (double)x[m] - C64[(int64_t)j * d + m];
            acc = fma(t, t, acc);
        }
        return acc;
    };
    if (inc >= 0) {
        Dbb = dist(inc);
        bb = inc;
    }
    for (int j = 0; j < k; ++j) {
        if (j == inc) continue;
        const double Dj = dist(j);
        if (Dj < Dbb) {
            Dbb = Dj;
            bb = j;
        }
    }
    Db = (float)Dbb;
    ub = f32_up(sqrt(Dbb) * (1.0 + 0x1p-40));
    return bb;
}

}  // namespace

// All-reduce minimum within aligned groups of G lanes (G = 4, 8 or 16) on DPP
// row operations.
template <int G>
__device__ inline uint32_t group_min_u32(uint32_t v) {
    v = min(v, (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0xB1, 0xF, 0xF, false));   // xor 1
    v = min(v, (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0x4E, 0xF, 0xF, false));   // xor 2
    if constexpr (G >= 8)
        v = min(v, (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0x141, 0xF, 0xF, false));   // half mirror
    if constexpr (G >= 16)
        v = min(v, (uint32_t)__builtin_amdgcn_update_dpp((int)v, (int)v, 0x140, 0xF, 0xF, false));   // mirror
    return v;
}

// ---------------------------------------------------------------------------
// Survivor processing shared by the streaming and the incremental kernel.

struct SurvCtx {
    const float* Cs;       // LDS centroid rows (stride D + 4)
    const float* ecs;      // LDS rounding errors of the float32 centroids
    const float* hs;       // LDS half-distance table
    uint64_t* acc;         // LDS sums, kCopies copies of stride csu
    uint32_t* cnt;         // LDS counts, kCopies copies of stride kp
    int csu, kp;
    const double* C64;     // float64 master centroids (near-tie decisions)
    int32_t* a;            // point assignments
    float* u;              // point bounds
    int k;
    bool prune, first, want_inertia;
    float gamma, ecmax;
    double qscale, iscale;
};

// One survivor: its LDS row, incumbent (-1 in the first step), drift-updated
// bound, global index and tile row.
struct Surv {
    const float* xrow;
    int inc;
    float u;
    int64_t p;
    int r;
};

// Moves point row x from cluster inc to b in the LDS sums (coordinates
// m0, m0 + step, ...; counts when count is set).
template <int D>
__device__ inline void move_sums(const SurvCtx& S, int cp, const float* x, int inc, int b, int m0, int step,
                                 bool count) {
    uint64_t* to = S.acc + cp * S.csu + b * D;
    uint64_t* from = S.acc + cp * S.csu + inc * D;
    for (int m = m0; m < D; m += step) {
        const uint64_t v = fixed_bits((double)x[m], S.qscale);
        atomicAdd(reinterpret_cast<unsigned long long*>(to + m), (unsigned long long)v);
        atomicAdd(reinterpret_cast<unsigned long long*>(from + m), (unsigned long long)(0 - v));
    }
    if (count) {
        atomicAdd(&S.cnt[cp * S.kp + b], 1u);
        atomicAdd(&S.cnt[cp * S.kp + inc], 0xFFFFFFFFu);
    }
}

// Survivors 0 .. nq-1 (nq <= kTp) of a block.  Many: one lane each, scanning
// the centroids in index order and skipping one for the whole wave when
// Clause 2 holds for every lane.  Few: G lanes each, lane j for centroid j.
// Writes the bound, the assignment if it changed, sa[r] = b in the first
// step, and moves the sums of a changed point (not in the first step).
template <int D, int G, class Entry>
__device__ inline void process_survivors(const SurvCtx& S, int nq, Entry entry, int* sa, uint64_t& changed,
                                         uint64_t& comp, uint64_t& rechecks, uint64_t& iq) {
    constexpr int CR = D + 4;
    constexpr int PER = kTp / G;
    const int tid = threadIdx.x, lane = tid & 63;
    const int k = S.k;
    if (nq > kLaneScanMin) {
        if (tid >= nq) return;
        const Surv v = entry(tid);
        const int inc = v.inc;
        float x[D];
#pragma unroll
        for (int m = 0; m < D; m += 4) {
            const f32x4 q = *reinterpret_cast<const f32x4*>(v.xrow + m);
            x[m] = q.x;
            x[m + 1] = q.y;
            x[m + 2] = q.z;
            x[m + 3] = q.w;
        }
        // Best so far under the oracle's order: smaller distance, then the
        // incumbent, then the lower index (key 0 = incumbent).
        int b = -1;
        uint32_t kb = 0xFFFFFFFFu;
        float Db = INFINITY, D2 = INFINITY;
        uint64_t nc = 0;
        for (int jj = 0; jj < k; ++jj) {
            // Clause 2: c_jj cannot be strictly closer than the incumbent.
            const bool need = !(S.prune && inc >= 0 && jj != inc && v.u <= S.hs[max(inc, 0) * k + jj]);
            if (!__any(need)) continue;   // the whole wave skips c_jj
            const float Dj = sqd_row<D>(x, S.Cs + jj * CR);
            if (need) {
                nc += 1;
                const uint32_t key = jj == inc ? 0u : (uint32_t)jj + 1u;
                if (Dj < Db || (Dj == Db && key < kb)) {
                    D2 = Db;
                    Db = Dj;
                    b = jj;
                    kb = key;
                } else {
                    D2 = fminf(D2, Dj);
                }
            }
        }
        if (b < 0) b = 0;   // only for non-finite rows (no comparison succeeded)
        float ub = upper_bound(Db, S.ecs[b], S.gamma);
        if (D2 != INFINITY) {
            const float band = 2.f * S.gamma * (Db + D2) + 4.f * (sqrtf(Db) + sqrtf(D2)) * S.ecmax +
                               8.f * S.ecmax * S.ecmax;
            if (D2 - Db <= band) {   // near tie: float64 decision, the oracle's tie rule
                b = recheck64(v.xrow, S.C64, D, k, inc, Db, ub);
                rechecks += 1;
            }
        }
        S.u[v.p] = ub;
        comp += nc;
        if (S.want_inertia) iq += fixed_bits((double)Db, S.iscale) - kMagicBits;
        if (b != inc) {
            S.a[v.p] = b;
            changed += 1;
        }
        if (S.first) sa[v.r] = b;
        else if (b != inc) move_sums<D>(S, tid & (kCopies - 1), x, inc, b, 0, 1, true);
        return;
    }
    const int g = tid / G, j = tid % G;
    const uint64_t gmask = ((1ull << G) - 1ull) << (lane - j);
    for (int p0 = 0; p0 < nq; p0 += PER) {
        const int slot = p0 + g;
        const bool act = slot < nq;
        const Surv v = entry(act ? slot : p0);
        const int inc = v.inc;
        // Clause 2: c_j cannot be strictly closer than the incumbent.
        const bool want = act && j < k && !(S.prune && inc >= 0 && j != inc && v.u <= S.hs[max(inc, 0) * k + j]);
        float Dj = INFINITY;
        if (want) {
            float x[D];
#pragma unroll
            for (int m = 0; m < D; m += 4) {
                const f32x4 q = *reinterpret_cast<const f32x4*>(v.xrow + m);
                x[m] = q.x;
                x[m + 1] = q.y;
                x[m + 2] = q.z;
                x[m + 3] = q.w;
            }
            Dj = sqd_row<D>(x, S.Cs + j * CR);
        }
        // D >= 0, so float order is the order of the bit patterns.
        const uint32_t dbits = __float_as_uint(Dj);
        const uint32_t m1 = group_min_u32<G>(dbits);
        // Among the minimal lanes the incumbent wins, then the lowest index.
        const uint32_t key = dbits == m1 && want ? (j == inc ? 0u : (uint32_t)j + 1u) : 0xFFFFFFFFu;
        const uint32_t kmin = group_min_u32<G>(key);
        int b = kmin == 0u ? inc : (int)kmin - 1;
        const uint32_t m2 = group_min_u32<G>(want && j != b ? dbits : 0x7F800000u);
        float Db = __uint_as_float(m1);
        const float D2 = __uint_as_float(m2);
        const uint64_t wm = __ballot(want);
        if (b < 0) b = 0;   // only for non-finite rows (no comparison succeeded)
        float ub = upper_bound(Db, S.ecs[b], S.gamma);
        bool re = false;
        if (D2 != INFINITY) {
            const float band = 2.f * S.gamma * (Db + D2) + 4.f * (sqrtf(Db) + sqrtf(D2)) * S.ecmax +
                               8.f * S.ecmax * S.ecmax;
            re = act && D2 - Db <= band;
        }
        if (re) b = recheck64(v.xrow, S.C64, D, k, inc, Db, ub);   // every lane of the group alike
        if (act && j == 0) {
            S.u[v.p] = ub;
            if (b != inc) {
                S.a[v.p] = b;
                changed += 1;
            }
            if (S.first) sa[v.r] = b;
            comp += (uint64_t)__popcll(wm & gmask);
            if (re) rechecks += 1;
            if (S.want_inertia) iq += fixed_bits((double)Db, S.iscale) - kMagicBits;
        }
        if (act && !S.first && b != inc) move_sums<D>(S, g & (kCopies - 1), v.xrow, inc, b, j, G, j == 0);
    }
}

// ---------------------------------------------------------------------------
// The streaming kernel.  Block = kTp threads; wave w of a tile owns points
// 64w .. 64w+63.  X is prefetched per wave as D/4 coalesced 16-byte loads per
// lane: load i of lane l holds the 4-float chunk q = (64i + l) % (D/4) of the
// wave's row rho = (64i + l) / (D/4).  G: lanes per survivor (k <= G).

template <int D, int G>
__global__ __launch_bounds__(kTp) __attribute__((amdgpu_waves_per_eu(4))) void k_small(Dev P, Fused F) {
    static_assert(D == 16, "streaming kernel is specialised for d = 16");
    static_assert(G == 4 || G == 8 || G == 16, "survivor groups are DPP rows or parts of one");
    constexpr int QD = D / 4;      // 16-byte chunks per row
    constexpr int CH = QD;         // chunks per lane per tile (64 rows * QD / 64 lanes)
    constexpr int XS = D + 4;      // padded LDS row stride of the tile (floats)
    constexpr int CR = D + 4;      // padded LDS centroid row stride (floats)

    IterState* st = P.st;
    if (st->done) {
        if (blockIdx.x == 0 && threadIdx.x == 0) st->active = 0;
        return;
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) st->active = 1;

    const int k = P.k;
    const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
    const bool first = st->t == 0;
    const bool prune = !(P.flags & KM_FLAG_NO_PRUNE);
    const bool want_inertia = (P.flags & KM_FLAG_STATS) != 0;
    const float ecmax = st->ec_max;
    const float gamma = P.gamma;

    const SmallLds lay = small_lds(k);
    float* Cs = reinterpret_cast<float*>(km_smem + lay.off_c);
    float* fs = reinterpret_cast<float*>(km_smem + lay.off_f);
    float* ss = reinterpret_cast<float*>(km_smem + lay.off_s);
    float* ecs = reinterpret_cast<float*>(km_smem + lay.off_ec);
    float* hs = reinterpret_cast<float*>(km_smem + lay.off_h);
    uint64_t* acc = reinterpret_cast<uint64_t*>(km_smem + lay.off_acc);
    uint32_t* cnt = reinterpret_cast<uint32_t*>(km_smem + lay.off_cnt);
    float* Xs = reinterpret_cast<float*>(km_smem + lay.off_x);
    int* sq = reinterpret_cast<int*>(km_smem + lay.off_sq);
    int* sa = reinterpret_cast<int*>(km_smem + lay.off_sa);
    float* su = reinterpret_cast<float*>(km_smem + lay.off_su);
    int* qlen = reinterpret_cast<int*>(km_smem + lay.off_misc);
    uint64_t* bst = reinterpret_cast<uint64_t*>(km_smem + lay.off_misc + 16);
    const int csu = lay.csu, kp = lay.kp;

    for (int i = tid; i < k * D; i += kTp) Cs[(i / D) * CR + i % D] = P.C32[i];
    for (int i = tid; i < k; i += kTp) {
        fs[i] = P.f[i];
        ss[i] = P.s[i];
        ecs[i] = P.ec[i];
    }
    for (int i = tid; i < k * k; i += kTp) hs[i] = P.h[i];
    for (int i = tid; i < kCopies * csu; i += kTp) acc[i] = 0;
    for (int i = tid; i < kCopies * kp; i += kTp) cnt[i] = 0;
    if (tid < kNumStat) bst[tid] = 0;
    if (tid < 2) qlen[tid] = 0;

    uint64_t my_changed = 0, my_comp = 0, my_c1 = 0, my_rc = 0, my_iq = 0;
    const int64_t n = P.n;
    const int64_t ntiles = (n + kTp - 1) / kTp;
    const int64_t nchunks = n * QD;

    f32x4 xbuf[CH];
    int abuf = 0;
    float ubuf = 0.f;
    auto prefetch = [&](int64_t tl) {
        const f32x4* s4 = reinterpret_cast<const f32x4*>(P.X);
        const int64_t c0 = (tl * kTp + 64 * w) * QD + lane;
#pragma unroll
        for (int i = 0; i < CH; ++i) xbuf[i] = __builtin_nontemporal_load(s4 + min(c0 + 64 * i, nchunks - 1));
        const int64_t q = min(tl * kTp + tid, n - 1);
        abuf = P.a[q];   // unset before the first step: read but not used then
        ubuf = P.u[q];
    };
    if ((int64_t)blockIdx.x < ntiles) prefetch(blockIdx.x);
    int it = 0;

    for (int64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x, ++it) {
        const int64_t base = tile * kTp;
        const int rows = (int)min((int64_t)kTp, n - base);
        __syncthreads();   // the previous tile's queue and rows are consumed
        if (tid == 0) qlen[(it + 1) & 1] = 0;
        int* qn = qlen + (it & 1);

        // 1. Bound update and Clause 1 for this lane's point.
        const bool valid = tid < rows;
        const int64_t p = base + tid;
        int a_old = -1;
        float u_cur = INFINITY;
        bool surv = false;
        if (valid) {
            if (first) {
                surv = true;
            } else {
                a_old = abuf;
                u_cur = (ubuf + fs[a_old]) * kUp;
                surv = !prune || u_cur > ss[a_old];
            }
        }

        // 2. Stage the rows (for the survivor groups and the sums), start the
        //    next tile's loads, and add every row to the sums of its previous
        //    cluster.  Each wave reads back only rows it staged itself.
#pragma unroll
        for (int i = 0; i < CH; ++i) {
            const int c = 64 * i + lane;
            const int rho = c / QD, q = c - rho * QD;
            *reinterpret_cast<f32x4*>(Xs + (64 * w + rho) * XS + 4 * q) = xbuf[i];
        }
        if (tile + gridDim.x < ntiles) prefetch(tile + gridDim.x);
        if (!first) {
#pragma unroll
            for (int i = 0; i < CH; ++i) {
                const int c = 64 * i + lane;
                const int rho = c / QD, q = c - rho * QD;
                const int ar = __shfl(a_old, rho);
                if (64 * w + rho < rows) {
                    const f32x4 xv = *reinterpret_cast<const f32x4*>(Xs + (64 * w + rho) * XS + 4 * q);
                    const int cp = rho & (kCopies - 1);
                    uint64_t* dst = acc + cp * csu + ar * D + 4 * q;
                    atomicAdd(reinterpret_cast<unsigned long long*>(dst + 0),
                              (unsigned long long)fixed_bits((double)xv.x, P.qscale));
                    atomicAdd(reinterpret_cast<unsigned long long*>(dst + 1),
                              (unsigned long long)fixed_bits((double)xv.y, P.qscale));
                    atomicAdd(reinterpret_cast<unsigned long long*>(dst + 2),
                              (unsigned long long)fixed_bits((double)xv.z, P.qscale));
                    atomicAdd(reinterpret_cast<unsigned long long*>(dst + 3),
                              (unsigned long long)fixed_bits((double)xv.w, P.qscale));
                    if (q == 0) atomicAdd(&cnt[cp * kp + ar], 1u);
                }
            }
        }

        // Clause-1 points are done: only the bound moves.
        if (valid && !surv) {
            P.u[p] = u_cur;
            my_c1 += 1;
        }
        if (surv) su[tid] = u_cur;
        {   // survivor queue: one LDS atomic per wave, ranks from the ballot
            const uint64_t bm = __ballot(surv);
            int wbase = 0;
            if (lane == 0 && bm) wbase = atomicAdd(qn, __popcll(bm));
            wbase = __shfl(wbase, 0);
            if (surv) sq[wbase + __popcll(bm & ((1ull << lane) - 1ull))] = tid | ((a_old + 1) << 16);
        }
        __syncthreads();

        if (want_inertia && valid && !surv) {   // inertia of an unmoved point
            float x[D];
#pragma unroll
            for (int m = 0; m < D; m += 4) {
                const f32x4 v = *reinterpret_cast<const f32x4*>(Xs + tid * XS + m);
                x[m] = v.x;
                x[m + 1] = v.y;
                x[m + 2] = v.z;
                x[m + 3] = v.w;
            }
            my_iq += fixed_bits((double)sqd_row<D>(x, Cs + a_old * CR), P.iscale) - kMagicBits;
        }

        // 3. Survivors; 4. moves of the changed points' sums.
        const int nq = *qn;
        {
            const SurvCtx S{Cs, ecs, hs, acc, cnt, csu, kp, P.C64, P.a, P.u, k, prune, first, want_inertia,
                            gamma, ecmax, P.qscale, P.iscale};
            process_survivors<D, G>(S, nq, [&](int i) {
                const int e = sq[i];
                const int r = e & 0xffff;
                return Surv{Xs + r * XS, (e >> 16) - 1, su[r], base + r, r};
            }, sa, my_changed, my_comp, my_rc, my_iq);
        }
        if (first) {   // first step: sums of the new assignment, from the staged rows
            __syncthreads();
#pragma unroll
            for (int i = 0; i < CH; ++i) {
                const int c = 64 * i + lane;
                const int rho = c / QD, q = c - rho * QD;
                const int r = 64 * w + rho;
                if (r < rows) {
                    const int ar = sa[r];
                    const f32x4 v = *reinterpret_cast<const f32x4*>(Xs + r * XS + 4 * q);
                    const int cp = rho & (kCopies - 1);
                    uint64_t* dst = acc + cp * csu + ar * D + 4 * q;
                    atomicAdd(reinterpret_cast<unsigned long long*>(dst + 0),
                              (unsigned long long)fixed_bits((double)v.x, P.qscale));
                    atomicAdd(reinterpret_cast<unsigned long long*>(dst + 1),
                              (unsigned long long)fixed_bits((double)v.y, P.qscale));
                    atomicAdd(reinterpret_cast<unsigned long long*>(dst + 2),
                              (unsigned long long)fixed_bits((double)v.z, P.qscale));
                    atomicAdd(reinterpret_cast<unsigned long long*>(dst + 3),
                              (unsigned long long)fixed_bits((double)v.w, P.qscale));
                    if (q == 0) atomicAdd(&cnt[cp * kp + ar], 1u);
                }
            }
        }
    }
    __syncthreads();

    // Block counters, then the block's row (copies of the sums added) into
    // accumulation row blockIdx % kSmallRows.
    my_changed = wave_sum_u64(my_changed);
    my_comp = wave_sum_u64(my_comp);
    my_c1 = wave_sum_u64(my_c1);
    my_rc = wave_sum_u64(my_rc);
    my_iq = wave_sum_u64(my_iq);
    if (lane == 0) {
        atomicAdd(reinterpret_cast<unsigned long long*>(&bst[kStChanged]), my_changed);
        atomicAdd(reinterpret_cast<unsigned long long*>(&bst[kStComputed]), my_comp);
        atomicAdd(reinterpret_cast<unsigned long long*>(&bst[kStClause1]), my_c1);
        atomicAdd(reinterpret_cast<unsigned long long*>(&bst[kStRecheck]), my_rc);
        atomicAdd(reinterpret_cast<unsigned long long*>(&bst[kStInertia]), my_iq);
    }
    __syncthreads();
    unsigned long long* row =
        reinterpret_cast<unsigned long long*>(F.rows + (int64_t)(blockIdx.x % kSmallRows) * P.L);
    for (int i = tid; i < k * D; i += kTp) {
        uint64_t v = 0;
#pragma unroll
        for (int c = 0; c < kCopies; ++c) v += acc[c * csu + i];
        atomicAdd(row + i, (unsigned long long)v);
    }
    for (int i = tid; i < k; i += kTp) {
        uint32_t v = 0;
#pragma unroll
        for (int c = 0; c < kCopies; ++c) v += cnt[c * kp + i];
        atomicAdd(row + k * D + i, (unsigned long long)v);
    }
    if (tid < kNumStat) atomicAdd(row + k * D + k + tid, (unsigned long long)bst[tid]);
}

// ---------------------------------------------------------------------------
// The incremental kernel (the paper's skipping of the data of points that
// Clause 1 keeps, section III-C; ||Lloyd's per-thread sums, section V).
// Steps after the first only.  Block b owns a contiguous range of tiles of
// kIncTile points (PT per thread).  Phase 1 streams their assignments and
// bounds: a Clause-1 point moves only its bound and its X row is never read;
// a survivor is appended to the block's list in global memory.  Phase 2
// takes the list kTp survivors at a time: their rows and state are gathered
// into LDS and they are scanned as in the streaming kernel.  The block's row
// then holds the moves of the points that changed, which the finishing block
// adds to the exact sums of the previous step.

template <int D, int G>
__global__ __launch_bounds__(kTp) __attribute__((amdgpu_waves_per_eu(4))) void k_inc(Dev P, Fused F) {
    static_assert(D == 16, "incremental kernel is specialised for d = 16");
    constexpr int QD = D / 4;               // 16-byte chunks per row
    constexpr int XS = D + 4;               // padded LDS row stride of the gathered rows
    constexpr int CR = D + 4;               // padded LDS centroid row stride
    constexpr int PT = kIncTile / kTp;      // points per thread per tile

    IterState* st = P.st;
    if (st->done || st->t == 0) {   // the first step always runs the streaming kernel
        if (blockIdx.x == 0 && threadIdx.x == 0) st->active = 0;
        return;
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) st->active = 1;

    const int k = P.k;
    const int tid = threadIdx.x, lane = tid & 63;
    const bool prune = !(P.flags & KM_FLAG_NO_PRUNE);
    const float ecmax = st->ec_max;

    const SmallLds lay = inc_lds(k);
    float* Cs = reinterpret_cast<float*>(km_smem + lay.off_c);
    float* fs = reinterpret_cast<float*>(km_smem + lay.off_f);
    float* ss = reinterpret_cast<float*>(km_smem + lay.off_s);
    float* ecs = reinterpret_cast<float*>(km_smem + lay.off_ec);
    float* hs = reinterpret_cast<float*>(km_smem + lay.off_h);
    uint64_t* acc = reinterpret_cast<uint64_t*>(km_smem + lay.off_acc);
    uint32_t* cnt = reinterpret_cast<uint32_t*>(km_smem + lay.off_cnt);
    float* Xs = reinterpret_cast<float*>(km_smem + lay.off_x);
    int* cq = reinterpret_cast<int*>(km_smem + lay.off_sq);
    int* ca = reinterpret_cast<int*>(km_smem + lay.off_sa);
    float* cu = reinterpret_cast<float*>(km_smem + lay.off_su);
    int* lenp = reinterpret_cast<int*>(km_smem + lay.off_misc);
    uint64_t* bst = reinterpret_cast<uint64_t*>(km_smem + lay.off_misc + 16);
    const int csu = lay.csu, kp = lay.kp;

    for (int i = tid; i < k * D; i += kTp) Cs[(i / D) * CR + i % D] = P.C32[i];
    for (int i = tid; i < k; i += kTp) {
        fs[i] = P.f[i];
        ss[i] = P.s[i];
        ecs[i] = P.ec[i];
    }
    for (int i = tid; i < k * k; i += kTp) hs[i] = P.h[i];
    for (int i = tid; i < kCopies * csu; i += kTp) acc[i] = 0;
    for (int i = tid; i < kCopies * kp; i += kTp) cnt[i] = 0;
    if (tid < kNumStat) bst[tid] = 0;
    if (tid == 0) *lenp = 0;
    __syncthreads();

    uint64_t my_changed = 0, my_comp = 0, my_c1 = 0, my_rc = 0, my_iq = 0;
    const int64_t n = P.n;
    const int64_t ntiles = (n + kIncTile - 1) / kIncTile;
    const int64_t tpb = F.span / kIncTile;
    const int64_t t_begin = (int64_t)blockIdx.x * tpb;
    const int64_t t_end = min(ntiles, t_begin + tpb);
    const int64_t lbase = (int64_t)blockIdx.x * F.span;   // this block's list

    // Phase 1: stream the assignments and bounds, two tiles in flight.
    int abA[PT], abB[PT];
    float ubA[PT], ubB[PT];
    auto prefetch = [&](int (&ab)[PT], float (&ub)[PT], int64_t tl) {
        if (tl >= t_end) return;
#pragma unroll
        for (int i = 0; i < PT; ++i) {
            const int64_t q = min(tl * kIncTile + tid + kTp * i, n - 1);
            ab[i] = P.a[q];
            ub[i] = P.u[q];
        }
    };
    prefetch(abA, ubA, t_begin);
    prefetch(abB, ubB, t_begin + 1);
    auto tile_body = [&](int (&ab)[PT], float (&ub)[PT], int64_t tile) {
        const int64_t base = tile * kIncTile;
        const int rows = (int)min((int64_t)kIncTile, n - base);
        int a_old[PT];
        float u_cur[PT];
        bool surv[PT];
#pragma unroll
        for (int i = 0; i < PT; ++i) {
            const bool valid = tid + kTp * i < rows;
            a_old[i] = valid ? ab[i] : 0;
            u_cur[i] = (ub[i] + fs[a_old[i]]) * kUp;
            surv[i] = valid && (!prune || u_cur[i] > ss[a_old[i]]);
            if (valid && !surv[i]) {   // Clause 1: only the bound moves
                P.u[base + tid + kTp * i] = u_cur[i];
                my_c1 += 1;
            }
        }
        prefetch(ab, ub, tile + 2);
#pragma unroll
        for (int i = 0; i < PT; ++i) {   // append to the list: one LDS atomic per wave and i
            const uint64_t bm = __ballot(surv[i]);
            int wbase = 0;
            if (lane == 0 && bm) wbase = atomicAdd(lenp, __popcll(bm));
            wbase = __shfl(wbase, 0);
            if (surv[i]) {
                const int64_t e = lbase + wbase + __popcll(bm & ((1ull << lane) - 1ull));
                F.lq[e] = (int)(base + tid + kTp * i);
                F.la[e] = a_old[i];
                F.lu[e] = u_cur[i];
            }
        }
    };
    for (int64_t tile = t_begin; tile < t_end; tile += 2) {
        tile_body(abA, ubA, tile);
        if (tile + 1 < t_end) tile_body(abB, ubB, tile + 1);
    }
    __syncthreads();   // the list (global, this block's own writes) and its length are complete

    // Phase 2: the survivors, kTp at a time.
    const SurvCtx S{Cs, ecs, hs, acc, cnt, csu, kp, P.C64, P.a, P.u, k, prune, false, false,
                    P.gamma, ecmax, P.qscale, P.iscale};
    const f32x4* X4 = reinterpret_cast<const f32x4*>(P.X);
    const int len = *lenp;
    for (int c0 = 0; c0 < len; c0 += kTp) {
        const int nc = min(kTp, len - c0);
        // Gather: the chunk's state, then its rows (QD 16-byte loads per thread).
        int qi = 0;
        if (tid < nc) {
            qi = F.lq[lbase + c0 + tid];
            cq[tid] = qi;
            ca[tid] = F.la[lbase + c0 + tid];
            cu[tid] = F.lu[lbase + c0 + tid];
        }
        __syncthreads();
        f32x4 gbuf[QD];
#pragma unroll
        for (int i = 0; i < QD; ++i) {
            const int idx = tid + kTp * i;
            const int sl = idx < nc * QD ? idx / QD : 0;
            gbuf[i] = __builtin_nontemporal_load(X4 + (int64_t)cq[sl] * QD + idx % QD);
        }
#pragma unroll
        for (int i = 0; i < QD; ++i) {
            const int idx = tid + kTp * i;
            if (idx < nc * QD) *reinterpret_cast<f32x4*>(Xs + (idx / QD) * XS + 4 * (idx % QD)) = gbuf[i];
        }
        __syncthreads();
        process_survivors<D, G>(S, nc, [&](int i) {
            return Surv{Xs + i * XS, ca[i], cu[i], (int64_t)cq[i], 0};
        }, nullptr, my_changed, my_comp, my_rc, my_iq);
        __syncthreads();   // rows and chunk state consumed
        (void)qi;
    }

    // Block counters, then the block's moves into accumulation row
    // blockIdx % kSmallRows.
    my_changed = wave_sum_u64(my_changed);
    my_comp = wave_sum_u64(my_comp);
    my_c1 = wave_sum_u64(my_c1);
    my_rc = wave_sum_u64(my_rc);
    if (lane == 0) {
        atomicAdd(reinterpret_cast<unsigned long long*>(&bst[kStChanged]), my_changed);
        atomicAdd(reinterpret_cast<unsigned long long*>(&bst[kStComputed]), my_comp);
        atomicAdd(reinterpret_cast<unsigned long long*>(&bst[kStClause1]), my_c1);
        atomicAdd(reinterpret_cast<unsigned long long*>(&bst[kStRecheck]), my_rc);
    }
    __syncthreads();
    unsigned long long* row =
        reinterpret_cast<unsigned long long*>(F.rows + (int64_t)(blockIdx.x % kSmallRows) * P.L);
    for (int i = tid; i < k * D; i += kTp) {
        uint64_t v = 0;
#pragma unroll
        for (int c = 0; c < kCopies; ++c) v += acc[c * csu + i];
        if (v) atomicAdd(row + i, (unsigned long long)v);
    }
    for (int i = tid; i < k; i += kTp) {
        uint32_t v = 0;
#pragma unroll
        for (int c = 0; c < kCopies; ++c) v += cnt[c * kp + i];
        if (v) atomicAdd(row + k * D + i, (unsigned long long)(int64_t)(int32_t)v);
    }
    if (tid < kNumStat && bst[tid]) atomicAdd(row + k * D + k + tid, (unsigned long long)bst[tid]);
    (void)my_iq;
}

// ---------------------------------------------------------------------------
// End of a step (one block): totals of the accumulation rows (which it
// clears), new centroids, drift, stop test, centroid table for the next step.

__global__ __launch_bounds__(kFinishThreads) void k_small_finish(Dev P, Fused F, int delta) {
    constexpr int nt = kFinishThreads;
    IterState* st = P.st;
    const int tid = threadIdx.x;
    const int k = P.k, d = P.d, L = P.L;
    uint64_t* tot = reinterpret_cast<uint64_t*>(km_smem);
    double* cn = reinterpret_cast<double*>(tot + L);
    double* dr = cn + k * d;
    double* de = dr + k * d;
    float* hl = reinterpret_cast<float*>(de + k * d);
    float* ecn = hl + k * k;
    // One round of loads: the old centroids and every accumulation row.
    double cold[kSmallMaxK * 16 / 256 + 1];
#pragma unroll
    for (int q = 0; q * nt < kSmallMaxK * 16; ++q) {
        const int e = tid + q * nt;
        cold[q] = e < k * d ? P.C64[e] : 0.0;
    }
    // (Issued before the state flag is known: the loads are in bounds either way.)
    const bool active = st->active != 0;
    for (int col = tid; col < L; col += nt) {
        uint64_t t[kSmallRows];
#pragma unroll
        for (int r = 0; r < kSmallRows; ++r) t[r] = F.rows[(int64_t)r * L + col];
        uint64_t v = 0;
#pragma unroll
        for (int r = 0; r < kSmallRows; ++r) v += t[r];
        if (col < k * d + k) {   // sums and counts: after the moves, or the full sums
            if (delta) v += F.sum[col];
            if (active) F.sum[col] = v;
        }
        tot[col] = v;
        if (active) {
#pragma unroll
            for (int r = 0; r < kSmallRows; ++r) F.rows[(int64_t)r * L + col] = 0;
        }
    }
    if (!active) return;
    __syncthreads();
    // New centroids: member means of the exact sums; empty clusters keep theirs.
#pragma unroll
    for (int q = 0; q * nt < kSmallMaxK * 16; ++q) {
        const int e = tid + q * nt;
        if (e >= k * d) break;
        const int jc = e / d;
        const uint64_t count = tot[k * d + jc];
        double cnew = cold[q];
        if (count > 0) {
            const int64_t qs = (int64_t)(tot[e] - count * kMagicBits);
            cnew = ((double)qs * P.qinv) / (double)count;
        }
        const double df = cnew - cold[q];
        const float c32 = (float)cnew;
        const double rr = (double)c32 - cnew;
        dr[e] = df * df;
        de[e] = rr * rr;
        cn[e] = cnew;
        P.C64[e] = cnew;
        P.C32[e] = c32;
    }
    __syncthreads();
    for (int jc = tid; jc < k; jc += nt) {
        double a = 0.0, b = 0.0, c2 = 0.0;
        for (int m = 0; m < d; ++m) {
            a += dr[jc * d + m];
            b += de[jc * d + m];
            const double cv = (double)(float)cn[jc * d + m];
            c2 = fma(cv, cv, c2);
        }
        P.f[jc] = f32_up(sqrt(a) * (1.0 + 0x1p-40));
        const float e = f32_up(sqrt(b) * (1.0 + 0x1p-40));
        P.ec[jc] = e;
        ecn[jc] = e;
        P.cn2[jc] = (float)c2;
    }
    // Half centroid distances of the new centroids, rounded down.
    for (int pr = tid; pr < k * k; pr += nt) {
        const int i = pr / k, jc = pr - i * k;
        float hv = 0.f;
        if (i != jc) {
            double acc = 0.0;
            for (int m = 0; m < d; ++m) {
                const double t = cn[i * d + m] - cn[jc * d + m];
                acc = fma(t, t, acc);
            }
            hv = f32_down(0.5 * sqrt(acc) * (1.0 - 0x1p-40));
        }
        hl[pr] = hv;
        P.h[pr] = hv;
    }
    __syncthreads();
    for (int i = tid; i < k; i += nt) {
        float mn = INFINITY;
        for (int jc = 0; jc < k; ++jc)
            if (jc != i) mn = fminf(mn, hl[i * k + jc]);
        P.s[i] = mn;
    }
    if (tid == 0) {
        float em = 0.f;
        for (int jc = 0; jc < k; ++jc) em = fmaxf(em, ecn[jc]);
        st->ec_max = em;
        const uint64_t* sc = tot + k * d + k;
        const int64_t changed = (int64_t)sc[kStChanged];
        const int64_t computed = (int64_t)sc[kStComputed];
        const int64_t c1 = (int64_t)sc[kStClause1];
        const int64_t rc = (int64_t)sc[kStRecheck];
        const int64_t iq = (int64_t)sc[kStInertia];
        const double inertia = (P.flags & KM_FLAG_STATS) ? (double)iq * P.iinv : NAN;
        const int t = st->t;
        IterRec& r = P.rec[t % kHistCap];
        r.changed = changed;
        r.computed = computed;
        r.clause1 = c1;
        r.rechecks = rc;
        r.inertia = inertia;
        st->changed_last = changed;
        st->tot_computed += computed;
        st->tot_clause1 += c1;
        st->tot_rechecks += rc;
        st->inertia_last = inertia;
        st->t = t + 1;
        const bool tol_hit = (double)changed < st->tol_n;
        if (tol_hit || t + 1 >= st->max_iters) {
            st->done = 1;
            st->converged = tol_hit ? 1 : 0;
        }
    }
}

// ---------------------------------------------------------------------------
// Host-side launchers and configuration.

bool small_applies(int64_t n, int d, int k, bool aligned) {
    return aligned && d == 16 && k <= kSmallMaxK && n <= INT_MAX;   // int32 point indices in the ring
}

int small_group(int k) { return k <= 4 ? 4 : (k <= 8 ? 8 : 16); }

const void* small_kernel_symbol(int k) {
    switch (small_group(k)) {
        case 4: return reinterpret_cast<const void*>(&k_small<16, 4>);
        case 8: return reinterpret_cast<const void*>(&k_small<16, 8>);
        default: return reinterpret_cast<const void*>(&k_small<16, 16>);
    }
}

const void* inc_kernel_symbol(int k) {
    switch (small_group(k)) {
        case 4: return reinterpret_cast<const void*>(&k_inc<16, 4>);
        case 8: return reinterpret_cast<const void*>(&k_inc<16, 8>);
        default: return reinterpret_cast<const void*>(&k_inc<16, 16>);
    }
}

int small_lds_bytes(int k) { return small_lds(k).bytes; }

int inc_lds_bytes(int k) { return inc_lds(k).bytes; }

int small_finish_lds_bytes(int k) { return finish_lds(16, k); }

hipError_t launch_small(const Dev& dv, const Fused& F, int lds_bytes, hipStream_t s) {
    switch (small_group(dv.k)) {
        case 4: hipLaunchKernelGGL((k_small<16, 4>), dim3(dv.G), dim3(kTp), lds_bytes, s, dv, F); break;
        case 8: hipLaunchKernelGGL((k_small<16, 8>), dim3(dv.G), dim3(kTp), lds_bytes, s, dv, F); break;
        default: hipLaunchKernelGGL((k_small<16, 16>), dim3(dv.G), dim3(kTp), lds_bytes, s, dv, F); break;
    }
    return hipGetLastError();
}

hipError_t launch_inc(const Dev& dv, const Fused& F, int grid, int lds_bytes, hipStream_t s) {
    switch (small_group(dv.k)) {
        case 4: hipLaunchKernelGGL((k_inc<16, 4>), dim3(grid), dim3(kTp), lds_bytes, s, dv, F); break;
        case 8: hipLaunchKernelGGL((k_inc<16, 8>), dim3(grid), dim3(kTp), lds_bytes, s, dv, F); break;
        default: hipLaunchKernelGGL((k_inc<16, 16>), dim3(grid), dim3(kTp), lds_bytes, s, dv, F); break;
    }
    return hipGetLastError();
}

hipError_t launch_small_finish(const Dev& dv, const Fused& F, int delta, hipStream_t s) {
    hipLaunchKernelGGL(k_small_finish, dim3(1), dim3(kFinishThreads), finish_lds(dv.d, dv.k), s, dv, F, delta);
    return hipGetLastError();
}

}  // namespace km
