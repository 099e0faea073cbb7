// Streaming MTI iteration for small k (k <= 16) and d = 16 (paper section
// III-B's merged ||Lloyd's step).
//
// Point state.  Every point keeps one 32-bit word: its cluster in the low 4
// bits and, in the rest, a float32 value v such that v plus the cumulative
// drift D_a = sum over updates of f(c_a) (Table I) is an upper bound on the
// point's distance to its centroid.  This is the bound of section III-C,
// u^t = u^{t0} + f^{t0+1} + ... + f^t, kept as v = u^{t0} - D_a^{t0} so that a
// point whose bound is not tightened is never rewritten; the reader adds
// D_a^t.  v is rounded up and D is held rounded up (when read) and down (when
// subtracted), so the bound stays valid for the float64 master centroids.
//
// k_small streams every row of X (persistent blocks, 256-point tiles, two
// tiles in flight per block).  Per tile it
//   1. applies Clause 1 to each point's drift-updated bound: u <= s(c_a) with
//      s(c) half the distance to the nearest other centroid (Elkan's lemma),
//      tested as v <= s(c_a) - D_a with the right side computed per cluster;
//   2. adds every row, from registers, to the fixed-point sums of its
//      PREVIOUS cluster (all points contribute, the sums are Lloyd's);
//   3. queues the Clause-1 survivors, rows included, in LDS.
// Whenever 256 survivors are queued, each lane scans one of them: the
// distance to its incumbent (the tightening of the bound), then the other
// centroids in index order, skipping c_j when the tightened bound is at most
// half the distance from the incumbent to c_j (Clause 3), with the oracle's
// tie rule and a float64 decision of near ties.  A point whose
// cluster changed moves its row from the old cluster's sums to the new one's
// (exact integer subtraction and addition).  In the first step there is no
// bound: every point is scanned and adds itself to its new cluster.
//
// k_inc (steps after the first, the paper's skipping of the data of points
// Clause 1 keeps, section III-C) reads only the point states, one 16-byte
// load of four states per thread; the survivors are queued by index and
// their rows gathered from X when a batch is scanned.  Its sums hold only the
// moves, which the end of the step adds to the exact sums of the previous
// step.
//
// The block's sums are integers, so their order does not matter; each block
// adds its row into one of kSmallRows accumulation rows of the step's slot
// with device atomics, and its counters into the step's counter slot.  The
// end of step t (eos_load + eos_finish) then adds those rows, forms the new
// centroids (member means; an empty cluster keeps its centroid), the drift,
// the cumulative drift and the centroid table h, s(c) for the next step
// (sections III-C and IV-A), and step_books the history and the stop test.
// It runs inside the next k_inc (every block, block 0 storing) when
// incremental steps follow each other, else as the one-block k_small_finish.
#include <float.h>
#include <limits.h>
#include <math.h>

#include "kmeans_mti.h"
#include "km_device.h"
#include "km_internal.h"

namespace km {

extern __shared__ __align__(16) unsigned char km_smem[];

namespace {

constexpr int kTp = kSmallTile;       // threads per block
constexpr int kCopies = kSmallCopies;
constexpr int kD = 16;                // dimension of this path
constexpr int kQD = kD / 4;           // 16-byte chunks per row
constexpr int kCR = kSmallRowStride;  // padded LDS row stride (floats)
// Error factor of a float32 squared distance in the expanded form, relative
// to (|x| + |c|)^2.
constexpr float kExpGamma = (float)(kD + 8) * 0x1p-24f;

// Point state word: v rounded up to a multiple of 16 units in the last place
// (for v >= 0 the bit pattern grows, for v < 0 the magnitude shrinks), with
// the cluster in the cleared bits.
__device__ __forceinline__ uint32_t pack_state(float v, int a) {
    uint32_t b = __float_as_uint(v);
    if (!(b >> 31)) b += 15u;
    return (b & ~15u) | (uint32_t)a;
}
__device__ __forceinline__ int state_cluster(uint32_t w) { return (int)(w & 15u); }
__device__ __forceinline__ float state_value(uint32_t w) { return __uint_as_float(w & ~15u); }

// State of a point now assigned to b with distance bound ub: v = ub - D_b,
// with D_b rounded down and the subtraction rounded up.
__device__ __forceinline__ uint32_t settle_state(float ub, float ddn_b, int b) {
    const float r = ub - ddn_b;
    return pack_state(r + fabsf(r) * 0x1p-22f, b);
}

// Upper bound on sqrt(v): the hardware square root (within a few units in
// the last place) scaled up by 2^-20.
__device__ __forceinline__ float sqrt_up(float v) { return __builtin_amdgcn_sqrtf(v) * (1.0f + 0x1p-20f); }

// Upper bound on the exact distance to the float64 centroid from a float32
// squared distance D (relative error <= gamma) and the centroid's float32
// rounding error ec.
__device__ __forceinline__ float bound_of(float D, float ec, float gamma) {
    return (sqrt_up(D) * (1.0f + gamma) + ec) * kUp;
}


// Squared float32 distance, coordinates in order (the same rounding as the
// other kernels of the library).
__device__ __forceinline__ float sqd_row(const float (&x)[kD], const float* c) {
    float acc = 0.f;
#pragma unroll
    for (int m = 0; m < kD; m += 4) {
        const f32x4 cv = *reinterpret_cast<const f32x4*>(c + m);
        const float t0 = x[m] - cv.x, t1 = x[m + 1] - cv.y, t2 = x[m + 2] - cv.z, t3 = x[m + 3] - cv.w;
        acc = fmaf(t0, t0, acc);
        acc = fmaf(t1, t1, acc);
        acc = fmaf(t2, t2, acc);
        acc = fmaf(t3, t3, acc);
    }
    return acc;
}

// Continues the squared-distance sum over one 4-coordinate chunk.
__device__ __forceinline__ float sqd_chunk(const f32x4 x, const float* c, float acc) {
    const f32x4 cv = *reinterpret_cast<const f32x4*>(c);
    const float t0 = x.x - cv.x, t1 = x.y - cv.y, t2 = x.z - cv.z, t3 = x.w - cv.w;
    acc = fmaf(t0, t0, acc);
    acc = fmaf(t1, t1, acc);
    acc = fmaf(t2, t2, acc);
    return fmaf(t3, t3, acc);
}

// Float64 decision of a near tie against the master centroids, with the
// oracle's rule: the incumbent keeps exact ties, then the lowest index wins.
// Returns the winner; Db and ub become its squared distance and distance
// bound.
__device__ __forceinline__ int recheck64(const float (&x)[kD], const double* C64, int k, int inc, float& Db,
                                 float& ub) {
    auto dist = [&](int j) __attribute__((always_inline)) {
        double acc = 0.0;
#pragma unroll
        for (int m = 0; m < kD; ++m) {
            const double t = (double)x[m] - C64[j * kD + m];
            acc = fma(t, t, acc);
        }
        return acc;
    };
    int bb = -1;
    double Dbb = INFINITY;
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
    return bb < 0 ? 0 : bb;
}

// Exact fixed-point image of a row added to (or, neg, subtracted from) one
// LDS sum row.
__device__ __forceinline__ void add_row(uint64_t* dst, const float (&x)[kD], double qscale, bool neg) {
#pragma unroll
    for (int m = 0; m < kD; ++m) {
        const uint64_t v = fixed_bits((double)x[m], qscale);
        if (neg)
            lds_sub64(dst + m, v);
        else
            atomicAdd(reinterpret_cast<unsigned long long*>(dst + m), (unsigned long long)v);
    }
}

// Per-block tables and sums in LDS, shared by both kernels.
struct Tables {
    float* C;      // k rows of kCR floats: float32 centroids
    float* h;      // k rows of kSmallMaxK: half centroid distances, rounded down
    float* thr;    // k: Clause-1 threshold on a state value (below)
    float* ec;     // k: float32 rounding error of each centroid, rounded up
    float* ddn;    // k: cumulative drift, rounded down
    float* cn;     // k: squared norms of the float32 centroids (float32 of the float64 sum)
    uint64_t* acc; // copies (stride csu) of the k rows (stride kSmallAccRow) of 16 fixed-point sums
    uint32_t* cnt; // copies of the k counts (stride kp)
    int* qc;       // three queue counters
    uint64_t* bst; // kNumStat block counters
    int csu, kp, copies;
};

// Place of h(r, j) in the LDS table: rows of kSmallMaxK, the four 16-byte
// chunks of row r permuted by (r / 4) mod 4 so that rows read at the same
// chunk by different lanes fall on different banks; entries past k hold +inf.
__device__ __forceinline__ int hpos(int r, int j) {
    return r * kSmallMaxK + 4 * ((j >> 2) ^ ((r >> 2) & 3)) + (j & 3);
}

// Table pointers into LDS, and the block's sums and counters cleared.
__device__ __forceinline__ Tables table_ptrs(const Dev& P, const SmallLds& lay) {
    Tables T;
    T.C = reinterpret_cast<float*>(km_smem + lay.off_c);
    T.h = reinterpret_cast<float*>(km_smem + lay.off_h);
    T.thr = reinterpret_cast<float*>(km_smem + lay.off_s);
    T.ec = reinterpret_cast<float*>(km_smem + lay.off_ec);
    T.ddn = reinterpret_cast<float*>(km_smem + lay.off_dd);
    T.cn = reinterpret_cast<float*>(km_smem + lay.off_cn);
    T.acc = reinterpret_cast<uint64_t*>(km_smem + lay.off_acc);
    T.cnt = reinterpret_cast<uint32_t*>(km_smem + lay.off_cnt);
    T.qc = reinterpret_cast<int*>(km_smem + lay.off_misc);
    T.bst = reinterpret_cast<uint64_t*>(km_smem + lay.off_misc + 16);
    T.csu = lay.csu;
    T.copies = lay.copies;
    T.kp = lay.kp;
    const int tid = threadIdx.x;
    const int nt = (int)blockDim.x;
    for (int i = tid; i < T.copies * T.csu; i += nt) T.acc[i] = 0;
    for (int i = tid; i < T.copies * T.kp; i += nt) T.cnt[i] = 0;
    if (tid < kNumStat) T.bst[tid] = 0;
    if (tid < 3) T.qc[tid] = 0;
    return T;
}

// The tables of step t from memory into T (the end of step t - 1 has run).
__device__ __forceinline__ void fill_tables(const Dev& P, const Fused& F, const Tables& T, int t) {
    const int k = P.k, tid = threadIdx.x;
    const double* dhi = F.dhi + (int64_t)slot2(t) * k;
    const int nt = (int)blockDim.x;
    for (int i = tid; i < k * kD; i += nt) T.C[(i / kD) * kCR + i % kD] = P.C32[i];
    for (int i = tid; i < k * kSmallMaxK; i += nt) {
        const int r = i / kSmallMaxK, j = i % kSmallMaxK;
        T.h[hpos(r, j)] = j < k ? P.h[r * k + j] : INFINITY;
    }
    for (int i = tid; i < k; i += nt) {
        T.thr[i] = clause1_thr(P.s[i], dhi[i]);
        T.ec[i] = P.ec[i];
        T.ddn[i] = F.ddn[i];
        T.cn[i] = P.cn2[i];
    }
}

// The tables of step t from memory (the end of step t - 1 has run).
__device__ __forceinline__ Tables load_tables(const Dev& P, const Fused& F, const SmallLds& lay, int t) {
    Tables T = table_ptrs(P, lay);
    fill_tables(P, F, T, t);
    return T;
}

// Block 0 of a step kernel clears the slots that step t + 1 accumulates into
// (last read by the end of step t - 2, which has run).
__device__ __forceinline__ void clear_next_slots(const Dev& P, const Fused& F, int t) {
    if (blockIdx.x != 0) return;
    uint64_t* r = F.rows + (int64_t)slot3(t + 1) * kSmallRows * P.L;
    for (int i = threadIdx.x; i < kSmallRows * P.L; i += (int)blockDim.x) r[i] = 0;
    if (threadIdx.x < kNumStat) F.stat[slot3(t + 1) * kNumStat + threadIdx.x] = 0;
}

// Per-lane step counters (32 bits: a lane counts far fewer than 2^32
// events; fewer live registers keep the incremental kernel free of spills).
struct Counters {
    uint32_t changed = 0, comp = 0, c1 = 0, rc = 0;
    uint64_t iq = 0;
};

struct StepFlags {
    bool first, prune, want_inertia;
    float gamma, ecmax;
    float cnmax;   // largest centroid norm, rounded up (bound of the expanded form)
};

// Largest norm of the step's float32 centroids, rounded up (from the squared
// norms in LDS).
__device__ __forceinline__ float centroid_norm_max(const Tables& T, int k) {
    float m2 = 0.f;
    for (int j = 0; j < k; ++j) m2 = fmaxf(m2, T.cn[j]);
    return sqrtf(m2) * kUp * kUp;
}

// The nearest of the candidate centroids (bits of cmask) on their
// direct-form distances, in ascending index: the incumbent wins an exact tie,
// then the lower index; a near tie is decided again in float64 against the
// master centroids.  Db and ub become the winner's squared distance and
// distance bound.
__device__ __forceinline__ int decide_direct(const Tables& T, const StepFlags& fl, const double* C64,
                                             const float (&x)[kD], int k, int inc, uint32_t cmask, float& Db,
                                             float& ub, Counters& cn) {
    float d2 = INFINITY;
    int rk1 = INT_MAX;
    int b = 0;
    Db = INFINITY;
    while (cmask) {
        const int j = __builtin_ctz(cmask);
        cmask &= cmask - 1;
        const float dj = sqd_row(x, T.C + j * kCR);
        const int rk = j == inc ? -1 : j;
        if (dj < Db || (dj == Db && rk < rk1)) {
            d2 = Db;
            Db = dj;
            rk1 = rk;
            b = j;
        } else if (dj < d2) {
            d2 = dj;
        }
    }
    ub = bound_of(Db, T.ec[b], fl.gamma);
    if (d2 != INFINITY) {
        const float band = 2.f * fl.gamma * (Db + d2) + 4.f * (sqrt_up(Db) + sqrt_up(d2)) * fl.ecmax +
                           8.f * fl.ecmax * fl.ecmax;
        if (d2 - Db <= band) {   // near tie: float64 decision, the oracle's tie rule
            b = recheck64(x, C64, k, inc, Db, ub);
            cn.rc += 1;
        }
    }
    return b;
}

// One survivor, row x in registers: its assignment, the new state word and,
// after the first step, the move of a changed point's row between the sums
// (cp selects the copy of the LDS sums).  In the first step the new cluster
// is stored to *first_b instead.  KC >= k: distance slots.
//
// The k squared distances are first formed in the expanded form
// |x|^2 + |c|^2 - 2 x.c (one fused multiply-add per coordinate and centroid,
// half the work of the direct form).  Its float32 error is at most
// E = (d + 8) 2^-24 (|x| + |c|)^2 + 4 (|x| + |c|) ec + 2 ec^2, with ec the
// centroids' float32 rounding errors, so every centroid whose expanded value
// exceeds the smallest by more than 2E is strictly farther than the nearest
// and only the others are candidates:
//   - a single candidate is the nearest centroid; its bound is the square
//     root of its expanded value plus E (with inertia, its direct-form
//     distance is formed for the sum);
//   - several candidates are decided on their direct-form distances with the
//     oracle's tie rule, and a near tie again in float64 against the master
//     centroids.
// The decision is therefore the same as a scan of all direct-form distances.
// The count of distances is that of the MTI scan: in later steps the
// incumbent (the tightening of the bound) and every c_j that Clause 3 does
// not skip (the tightened bound at most half the distance from the incumbent
// to c_j); in the first step, which has no bound, all k.
// The MTI scan's count of distances for a point with incumbent inc: the
// incumbent's (which tightens its bound u), then one per other centroid that
// Clause 3 does not skip (u > half the distance from the incumbent to it).
// vi: the incumbent's expanded-form value, E its error bound; b, ub: the
// decision and its bound (u when b is the incumbent).  With h(inc, inc) = 0
// and +inf past k, the count is the number of row entries below u (the
// incumbent's own included when u > 0), at least one.
template <int KC>
__device__ __forceinline__ uint32_t mti_count(const float* h, float vi, int inc, int b, float ub, float E) {
    const float u = b == inc ? ub : sqrt_up(fmaxf(vi + E, 0.f)) * kUp;   // the incumbent's tightened bound
    uint32_t nc = 0;
#pragma unroll
    for (int j = 0; j < KC; j += 4) {
        const f32x4 hv = *reinterpret_cast<const f32x4*>(h + hpos(inc, j));
        nc += (u > hv.x ? 1u : 0u) + (u > hv.y ? 1u : 0u) + (u > hv.z ? 1u : 0u) + (u > hv.w ? 1u : 0u);
    }
    return nc > 1u ? nc : 1u;
}

template <int KC, bool INC_ONLY = false>
__device__ __forceinline__ void settle_survivor(const Dev& P, const Fused& F, const Tables& T, const StepFlags& fl,
                                       const double* C64, const float (&x)[kD], int64_t p, int inc, int cp,
                                       Counters& cn, int* first_b) {
    const int k = P.k;
    float x2 = 0.f;
#pragma unroll
    for (int m = 0; m < kD; ++m) x2 = fmaf(x[m], x[m], x2);
    float V[KC];
    float vmin = INFINITY;
#pragma unroll
    for (int j = 0; j < KC; ++j) {
        if (j < k) {   // uniform
            const float* c = T.C + j * kCR;
            float dt = 0.f;
#pragma unroll
            for (int m = 0; m < kD; m += 4) {
                const f32x4 cv = *reinterpret_cast<const f32x4*>(c + m);
                dt = fmaf(x[m], cv.x, dt);
                dt = fmaf(x[m + 1], cv.y, dt);
                dt = fmaf(x[m + 2], cv.z, dt);
                dt = fmaf(x[m + 3], cv.w, dt);
            }
            V[j] = fmaf(-2.f, dt, x2 + T.cn[j]);
        } else {
            V[j] = INFINITY;
        }
        vmin = fminf(vmin, V[j]);
    }
    const float R = sqrtf(x2) * (1.0f + 0x1p-20f) + fl.cnmax;
    const float E = (kExpGamma * R * R + 4.f * R * fl.ecmax + 2.f * fl.ecmax * fl.ecmax) * kUp;
    const float lim = vmin + 2.f * E;
    uint32_t cmask = 0;
#pragma unroll
    for (int j = 0; j < KC; ++j) cmask |= (V[j] <= lim ? 1u : 0u) << j;
    cmask &= (1u << k) - 1u;   // (an infinite minimum would admit the slots past k)
    int b;
    float Db, ub;
    if (__popc(cmask) == 1 && !fl.want_inertia) {
        b = __builtin_ctz(cmask);
        Db = vmin;
        ub = sqrt_up(fmaxf(vmin + E, 0.f)) * kUp;
    } else {
        b = decide_direct(T, fl, C64, x, k, inc, cmask, Db, ub, cn);
    }
    if ((INC_ONLY || inc >= 0) && fl.prune) {
        float vi = INFINITY;
#pragma unroll
        for (int j = 0; j < KC; ++j) vi = j == inc ? V[j] : vi;
        cn.comp += mti_count<KC>(T.h, vi, inc, b, ub, E);
    } else {
        cn.comp += (uint32_t)k;
    }
    if (fl.want_inertia) cn.iq += fixed_bits((double)Db, P.iscale) - kMagicBits;
    F.w[p] = settle_state(ub, T.ddn[b], b);
    if (b != inc) cn.changed += 1;
    if (fl.first) {
        *first_b = b;   // the caller adds the row to the sums of b
    } else if (b != inc) {
        add_row(T.acc + cp * T.csu + b * kSmallAccRow, x, P.qscale, false);
        add_row(T.acc + cp * T.csu + inc * kSmallAccRow, x, P.qscale, true);
        atomicAdd(&T.cnt[cp * T.kp + b], 1u);
        atomicAdd(&T.cnt[cp * T.kp + inc], 0xFFFFFFFFu);
    }
}

// A wave's moved rows out of their old clusters' sums and into the new ones',
// four lanes per row (chunk lane % 4 of the row) and sixteen rows per pass,
// so that the LDS atomics run with most lanes active (the dense incremental
// step, where a tile's 64 points move a few rows each).  Entry e of the list
// is the row's index among `rows` (stride kCR floats) | new cluster << 6 |
// old cluster << 10; nmov (at most 64) is uniform.
__device__ __forceinline__ void move_rows(const Tables& T, const float* rows, const int* list, int nmov, int lane,
                                          double qscale) {
    const int c = lane & 3;
    const int cp = (lane >> 2) & (kCopies - 1);
    for (int base = 0; base < nmov; base += 16) {
        const int e = base + (lane >> 2);
        if (e < nmov) {
            const int ent = list[e];
            const f32x4 xv = *reinterpret_cast<const f32x4*>(rows + (ent & 63) * kCR + 4 * c);
            uint64_t* dn = T.acc + cp * T.csu + ((ent >> 6) & 15) * kSmallAccRow + 4 * c;
            uint64_t* dp = T.acc + cp * T.csu + ((ent >> 10) & 15) * kSmallAccRow + 4 * c;
            const float xs[4] = {xv.x, xv.y, xv.z, xv.w};
#pragma unroll
            for (int m = 0; m < 4; ++m) {
                const uint64_t v = fixed_bits((double)xs[m], qscale);
                atomicAdd(reinterpret_cast<unsigned long long*>(dn + m), (unsigned long long)v);
                lds_sub64(dp + m, v);
            }
        }
    }
}

// Block counters into the block's counter slot, then the block's sums (copies
// added) into accumulation row blockIdx % kSmallRows.  skip_zero: only nonzero
// words are added.
__device__ __forceinline__ void flush_block(const Dev& P, const Fused& F, const Tables& T, Counters& cn,
                                   bool skip_zero, int t) {
    const int k = P.k, tid = threadIdx.x, lane = tid & 63;
    const uint64_t v0 = wave_sum_u64(cn.changed), v1 = wave_sum_u64(cn.comp), v2 = wave_sum_u64(cn.c1),
                   v3 = wave_sum_u64(cn.rc), v4 = wave_sum_u64(cn.iq);
    __syncthreads();   // every wave is done with the queue and the sums
    if (lane == 0) {
        unsigned long long* b = reinterpret_cast<unsigned long long*>(T.bst);
        atomicAdd(b + kStChanged, (unsigned long long)v0);
        atomicAdd(b + kStComputed, (unsigned long long)v1);
        atomicAdd(b + kStClause1, (unsigned long long)v2);
        atomicAdd(b + kStRecheck, (unsigned long long)v3);
        atomicAdd(b + kStInertia, (unsigned long long)v4);
    }
    __syncthreads();
    unsigned long long* row = reinterpret_cast<unsigned long long*>(
        F.rows + ((int64_t)slot3(t) * kSmallRows + blockIdx.x % kSmallRows) * P.L);
    const int nt = (int)blockDim.x;
    for (int i = tid; i < k * kD; i += nt) {
        uint64_t v = 0;
#pragma unroll
        for (int c = 0; c < T.copies; ++c) v += T.acc[c * T.csu + (i / kD) * kSmallAccRow + i % kD];
        if (v || !skip_zero) atomicAdd(row + i, (unsigned long long)v);
    }
    for (int i = tid; i < k; i += nt) {
        uint32_t v = 0;
#pragma unroll
        for (int c = 0; c < T.copies; ++c) v += T.cnt[c * T.kp + i];
        // A count change is a 32-bit two's-complement value (moves may be negative).
        if (v || !skip_zero) atomicAdd(row + k * kD + i, (unsigned long long)(int64_t)(int32_t)v);
    }
    // The block's counters into the step's totals (the next step's stop test
    // and bookkeeping read them).
    if (tid < kNumStat)
        atomicAdd(reinterpret_cast<unsigned long long*>(F.stat + slot3(t) * kNumStat + tid),
                  (unsigned long long)T.bst[tid]);
}

}  // namespace

// ---------------------------------------------------------------------------
// End of step t: exact sums, new centroids C^{t+1} (member means; an empty
// cluster keeps its centroid; spherical k-means projects them to the unit
// sphere), drift and cumulative drift, centroid table h and s for step t + 1
// (sections III-C and IV-A), as eos_load then eos_finish.  Run by one
// block of at least 256 threads: thread 16j + m
// owns coordinate m of centroid j (k <= 16, d = 16), so that the per-centroid
// terms are reductions over 16 lanes and one barrier separates the centroids
// from the table.  LDS scratch: finish_lds(16, k) bytes.  delta: the rows of
// step t hold the moves of an incremental step, added to the sums of step
// t - 1; else they hold the full sums.  writer: this block stores the
// results (sums of step t, C^{t+1}, D^{t+1}, the float32 tables).  T
// (nullable): the LDS tables of step t + 1 are filled too (Clause-1
// thresholds, float32 rows, h rows, ec, ddn) and c64n receives C^{t+1} in
// float64.  Returns the largest centroid rounding error ec.

__device__ __forceinline__ double sum16(double v) {
#pragma unroll
    for (int o = 8; o > 0; o >>= 1) v += __shfl_xor(v, o);
    return v;
}

// The loads of the end of step t (issued together; summed by eos_finish):
// the thread's old coordinate, its column of every accumulation row, the
// centroid's count column, the sums of step t - 1 (delta) and the
// cumulative drifts.
struct EosIn {
    double cold, dhi, dlo;
    uint64_t tv[kSmallRows], tc[kSmallRows], sv, sc;
};

__device__ __forceinline__ EosIn eos_load(const Dev& P, const Fused& F, int t, bool delta) {
    const int tid = threadIdx.x, j = tid >> 4, m = tid & 15;
    const int k = P.k, L = P.L, kd = k * kD;
    const bool live = j < k;
    const uint64_t* rows = F.rows + (int64_t)slot3(t) * kSmallRows * L;
    const uint64_t* sprev = F.sum + (int64_t)slot2(t - 1) * (kd + k);
    const int e = j * kD + m;
    const int ce = kd + j;
    EosIn in{};
    if (!live) return in;   // threads past the k centroids load nothing (whole waves skip)
    in.cold = F.c64[(int64_t)slot2(t) * kd + e];
#pragma unroll
    for (int r = 0; r < kSmallRows; ++r) {
        in.tv[r] = rows[(int64_t)r * L + e];
        in.tc[r] = rows[(int64_t)r * L + ce];
    }
    in.sv = delta ? sprev[e] : 0;   // the moves add to the sums of step t - 1
    in.sc = delta ? sprev[ce] : 0;
    in.dhi = F.dhi[(int64_t)slot2(t) * k + j];
    in.dlo = F.dlo[(int64_t)slot2(t) * k + j];
    return in;
}

__device__ float eos_finish(const Dev& P, const Fused& F, int t, const EosIn& in, bool writer, unsigned char* scratch,
                            const Tables* T, double* c64n) {
    const int tid = threadIdx.x, j = tid >> 4, m = tid & 15;
    const int k = P.k, kd = k * kD;
    const bool live = j < k;
    double* cn = reinterpret_cast<double*>(scratch);    // k x 16 new centroids
    float* ecn = reinterpret_cast<float*>(cn + kd);     // k rounding errors
    uint64_t* snow = F.sum + (int64_t)slot2(t) * (kd + k);
    double* cnew_p = F.c64 + (int64_t)slot2(t + 1) * kd;
    // Threads past the k centroids (whole 16-lane groups, so the group
    // reductions stay within live lanes; whole waves for the larger blocks)
    // skip the arithmetic and only meet the barrier.
    double hi = 0.0;
    if (live) {
        const int e = j * kD + m, ce = kd + j;
        const double cold = in.cold;
        uint64_t v = in.sv, cnt = in.sc;
#pragma unroll
        for (int r = 0; r < kSmallRows; ++r) {
            v += in.tv[r];
            cnt += in.tc[r];
        }
        if (writer) {
            snow[e] = v;
            if (m == 0) snow[ce] = cnt;
        }
        // Member mean of the exact sums; an empty cluster keeps its centroid.
        double cnew = cold;
        if (cnt > 0) cnew = ((double)(int64_t)(v - cnt * kMagicBits) * P.qinv) / (double)cnt;
        if (P.flags & KM_FLAG_SPHERICAL) {   // spherical k-means: the mean projected to the unit sphere
            const double ss = sum16(cnew * cnew);
            if (cnt > 0) cnew = ss > 0.0 ? cnew / sqrt(ss) : cold;   // a zero mean keeps the centroid
        }
        const float c32 = (float)cnew;
        const double df = cnew - cold, rr = (double)c32 - cnew;
        const double a = sum16(df * df), b = sum16(rr * rr), c2 = sum16((double)c32 * (double)c32);
        // Drift f(c) and its cumulative sums, with margins far above the
        // float64 rounding of the drift and of the running sums.
        const double fd = sqrt(a);
        hi = (in.dhi + fd * (1.0 + 0x1p-40)) * (1.0 + 0x1p-50);
        const double lo = (in.dlo + fd * (1.0 - 0x1p-40)) * (1.0 - 0x1p-50);
        const float ec = f32_up(sqrt(b) * (1.0 + 0x1p-40));
        cn[e] = cnew;
        if (m == 0) ecn[j] = ec;
        if (writer) {
            cnew_p[e] = cnew;
            P.C32[e] = c32;
            if (m == 0) {
                P.f[j] = f32_up(fd * (1.0 + 0x1p-40));
                F.dhi[(int64_t)slot2(t + 1) * k + j] = hi;
                F.dlo[(int64_t)slot2(t + 1) * k + j] = lo;
                F.dup[j] = f32_up(hi);
                F.ddn[j] = f32_down(lo);
                P.ec[j] = ec;
                P.cn2[j] = (float)c2;
            }
        }
        if (T) {
            T->C[j * kCR + m] = c32;
            c64n[e] = cnew;
            if (m == 0) {
                T->ec[j] = ec;
                T->ddn[j] = f32_down(lo);
                T->cn[j] = (float)c2;
            }
        }
    }
    __syncthreads();
    if (live) {
        // Half distance from centroid j to centroid m, rounded down; s(j) is
        // the smallest over m != j.
        float hv = 0.f;
        if (m < k && m != j) {
            double acc = 0.0;
#pragma unroll
            for (int q = 0; q < kD; ++q) {
                const double tq = cn[j * kD + q] - cn[m * kD + q];
                acc = fma(tq, tq, acc);
            }
            hv = f32_down(0.5 * sqrt(acc) * (1.0 - 0x1p-40));
        }
        float sv = (m < k && m != j) ? hv : INFINITY;
#pragma unroll
        for (int o = 8; o > 0; o >>= 1) sv = fminf(sv, __shfl_xor(sv, o));
        if (m < k && writer) P.h[j * k + m] = hv;
        if (T) T->h[hpos(j, m)] = m < k ? hv : INFINITY;
        if (m == 0) {
            if (writer) P.s[j] = sv;
            if (T) T->thr[j] = clause1_thr(sv, hi);
        }
    }
    float em = 0.f;
    for (int jc = 0; jc < k; ++jc) em = fmaxf(em, ecn[jc]);
    return em;
}

// Bookkeeping of step t by one thread: the step's counters, the history
// record and totals, the iteration count and the stop test.
__device__ void step_books(const Dev& P, const Fused& F, int t, float ecmax) {
    const uint64_t* sc = F.stat + slot3(t) * kNumStat;
    IterState* st = P.st;
    st->ec_max = ecmax;
    const int64_t changed = (int64_t)sc[kStChanged];
    const int64_t computed = (int64_t)sc[kStComputed];
    const int64_t c1 = (int64_t)sc[kStClause1];
    const int64_t rc = (int64_t)sc[kStRecheck];
    const int64_t iq = (int64_t)sc[kStInertia];
    const double inertia = (P.flags & KM_FLAG_STATS) ? (double)iq * P.iinv : NAN;
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
    report_step(st, t, tol_hit || t + 1 >= st->max_iters);
}

// ---------------------------------------------------------------------------
// The streaming kernel.  Wave w of a tile owns points 64w .. 64w+63; lane j
// holds the state of point 64w + j.  X is read per wave as 4 coalesced
// 16-byte loads per lane: load i of lane l holds chunk q = l % 4 of the
// wave's row rho = 16i + l / 4.

template <int KC>
__global__ __launch_bounds__(kTp) __attribute__((amdgpu_waves_per_eu(3))) void k_small(Dev P_, Fused F, int t) {
    const Dev P = with_scales(P_);
    IterState* st = P.st;
    if (st->done) {
        if (blockIdx.x == 0 && threadIdx.x == 0) st->active = 0;
        return;
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) st->active = 1;

    const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
    StepFlags fl{t == 0, !(P.flags & KM_FLAG_NO_PRUNE), (P.flags & KM_FLAG_STATS) != 0, P.gamma,
                 st->ec_max, 0.f};
    const SmallLds lay = small_lds(P.k, true);
    const Tables T = load_tables(P, F, lay, t);
    clear_next_slots(P, F, t);
    float* qr = reinterpret_cast<float*>(km_smem + lay.off_qr);   // queued rows
    int* qp = reinterpret_cast<int*>(km_smem + lay.off_qp);       // queued point index
    int* qa = reinterpret_cast<int*>(km_smem + lay.off_qa);       // queued incumbent (-1: none)
    __syncthreads();
    fl.cnmax = centroid_norm_max(T, P.k);

    Counters cn;
    const int64_t n = P.n;
    const int64_t ntiles = (n + kTp - 1) / kTp;
    const int64_t nchunks = n * kQD;
    const f32x4* X4 = reinterpret_cast<const f32x4*>(P.X);
    const int rho0 = lane >> 2, q = lane & 3;

    f32x4 xA[kQD], xB[kQD];
    uint32_t wA = 0, wB = 0;
    auto prefetch = [&](f32x4 (&xb)[kQD], uint32_t& wb, int64_t tl) __attribute__((always_inline)) {
        if (tl >= ntiles) return;
        const int64_t c0 = (tl * kTp + 64 * w) * kQD + lane;
#pragma unroll
        for (int i = 0; i < kQD; ++i) xb[i] = __builtin_nontemporal_load(X4 + min(c0 + 64 * i, nchunks - 1));
        wb = F.w[tl * kTp + tid];   // the state array is padded past n
    };
    prefetch(xA, wA, blockIdx.x);
    prefetch(xB, wB, (int64_t)blockIdx.x + gridDim.x);

    // Scans the queued survivors [e0, e0 + cnt), one per lane.
    auto scan_batch = [&](int e0, int cnt) __attribute__((always_inline)) {
        if (tid < cnt) {
            const int e = e0 + tid;
            float x[kD];
#pragma unroll
            for (int c = 0; c < kQD; ++c) {
                const f32x4 v = *reinterpret_cast<const f32x4*>(qr + e * kCR + 4 * c);
                x[4 * c] = v.x;
                x[4 * c + 1] = v.y;
                x[4 * c + 2] = v.z;
                x[4 * c + 3] = v.w;
            }
            settle_survivor<KC>(P, F, T, fl, P.C64, x, qp[e], qa[e], tid & (kCopies - 1), cn, qa + e);
        }
    };

    // First step: the scanned entries [e0, e0 + cnt) (new cluster in qa) into
    // the sums, four lanes per row as in the streaming sums.
    auto first_sums = [&](int e0, int cnt) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < kQD; ++i) {
            const int slot = 64 * w + 16 * i + rho0;
            if (slot < cnt) {
                const int e = e0 + slot;
                const int b = qa[e];
                const f32x4 v = *reinterpret_cast<const f32x4*>(qr + e * kCR + 4 * q);
                const int cp = slot & (kCopies - 1);
                uint64_t* dst = T.acc + cp * T.csu + b * kSmallAccRow + 4 * q;
                atomicAdd(reinterpret_cast<unsigned long long*>(dst + 0),
                          (unsigned long long)fixed_bits((double)v.x, P.qscale));
                atomicAdd(reinterpret_cast<unsigned long long*>(dst + 1),
                          (unsigned long long)fixed_bits((double)v.y, P.qscale));
                atomicAdd(reinterpret_cast<unsigned long long*>(dst + 2),
                          (unsigned long long)fixed_bits((double)v.z, P.qscale));
                atomicAdd(reinterpret_cast<unsigned long long*>(dst + 3),
                          (unsigned long long)fixed_bits((double)v.w, P.qscale));
                if (q == 0) atomicAdd(&T.cnt[cp * T.kp + b], 1u);
            }
        }
    };

    int queued = 0;   // block-uniform
    int it = 0;
    auto tile_body = [&](f32x4 (&xb)[kQD], uint32_t& wb, int64_t tile) __attribute__((always_inline)) {
        const int64_t base = tile * kTp;
        const int rows = (int)min((int64_t)kTp, n - base);
        const bool valid = tid < rows;
        int* qcount = T.qc + it % 3;
        if (tid == 0) T.qc[(it + 1) % 3] = 0;   // last read two barriers ago

        // 1. Clause 1 on the drift-updated bound.
        const uint32_t ws = wb;
        int a_old = -1;
        bool surv = valid;
        if (valid && !fl.first) {
            a_old = state_cluster(ws);
            surv = !fl.prune || !(state_value(ws) <= T.thr[a_old]);
            if (!surv) cn.c1 += 1;
        }

        // 2. Every row into the sums of its previous cluster; with inertia,
        //    the distance of each Clause-1 row to its centroid, summed over
        //    the row's four chunks in coordinate order.
        if (!fl.first) {
#pragma unroll
            for (int i = 0; i < kQD; ++i) {
                const int rho = 16 * i + rho0;
                const int ar = __shfl(a_old, rho);
                if (64 * w + rho < rows) {
                    const int cp = rho & (kCopies - 1);
                    uint64_t* dst = T.acc + cp * T.csu + ar * kSmallAccRow + 4 * q;
                    atomicAdd(reinterpret_cast<unsigned long long*>(dst + 0),
                              (unsigned long long)fixed_bits((double)xb[i].x, P.qscale));
                    atomicAdd(reinterpret_cast<unsigned long long*>(dst + 1),
                              (unsigned long long)fixed_bits((double)xb[i].y, P.qscale));
                    atomicAdd(reinterpret_cast<unsigned long long*>(dst + 2),
                              (unsigned long long)fixed_bits((double)xb[i].z, P.qscale));
                    atomicAdd(reinterpret_cast<unsigned long long*>(dst + 3),
                              (unsigned long long)fixed_bits((double)xb[i].w, P.qscale));
                    if (q == 0) atomicAdd(&T.cnt[cp * T.kp + ar], 1u);
                }
            }
            if (fl.want_inertia) {
                const bool keep = valid && !surv;
#pragma unroll
                for (int i = 0; i < kQD; ++i) {
                    const int rho = 16 * i + rho0;
                    const int ar = max(__shfl(a_old, rho), 0);
                    const int kept = __shfl(keep ? 1 : 0, rho);   // all lanes take part
                    const float* cr = T.C + ar * kCR + 4 * q;
                    float r = 0.f;
#pragma unroll
                    for (int qq = 0; qq < kQD; ++qq) {
                        const float prev = __shfl(r, (lane + 63) & 63);   // the lane of chunk q - 1
                        const float v = sqd_chunk(xb[i], cr, q == 0 ? 0.f : prev);
                        if (q == qq) r = v;
                    }
                    if (q == kQD - 1 && kept)
                        cn.iq += fixed_bits((double)r, P.iscale) - kMagicBits;
                }
            }
        }

        // 3. Queue the survivors: index and incumbent by the owning lane,
        //    the row's chunks by the lanes that loaded them.
        const uint64_t bm = __ballot(surv);
        int wbase = 0;
        if (lane == 0 && bm) wbase = atomicAdd(qcount, __popcll(bm));
        wbase = __shfl(wbase, 0);
        const int pos = queued + wbase + lanes_below(bm);
        if (surv) {
            qp[pos] = (int)(base + tid);
            qa[pos] = a_old;
        }
#pragma unroll
        for (int i = 0; i < kQD; ++i) {
            const int rho = 16 * i + rho0;
            const int rpos = __shfl(pos, rho);
            if ((bm >> rho) & 1ull) *reinterpret_cast<f32x4*>(qr + rpos * kCR + 4 * q) = xb[i];
        }
        prefetch(xb, wb, tile + 2 * (int64_t)gridDim.x);
        __syncthreads();
        queued += *qcount;
        if (queued >= kTp) {   // a full batch: the newest kTp entries
            queued -= kTp;
            scan_batch(queued, kTp);
            __syncthreads();   // its rows are consumed before the next tile queues over them
            if (fl.first) {
                first_sums(queued, kTp);
                __syncthreads();
            }
        }
        ++it;
    };
    for (int64_t tile = blockIdx.x; tile < ntiles; tile += 2 * (int64_t)gridDim.x) {
        tile_body(xA, wA, tile);
        if (tile + gridDim.x < ntiles) tile_body(xB, wB, tile + gridDim.x);
    }
    if (queued > 0) {
        scan_batch(0, queued);
        if (fl.first) {
            __syncthreads();
            first_sums(0, queued);
        }
    }
    flush_block(P, F, T, cn, false, t);
}

// ---------------------------------------------------------------------------
// The first step without statistics (no bounds yet: every point is scanned
// over all k centroids and adds its row to its new cluster's sums).  A wave
// takes 64-point tiles, four groups of 16 points.  The dot products of a
// group are a dense 16 x 16 x 16 product on the matrix cores
// (v_mfma_f32_16x16x4f32, four steps of four coordinates): lane
// l = 16 qd + pl loads chunk qd (coordinates 4qd .. 4qd+3) of point pl of the
// group, a coalesced kilobyte per group, and supplies coordinate 4qd + s at
// step s as the B operand; the A operand is coordinate 4qd + s of centroid pl
// (zero rows past k).  The lane then holds the dot products of point pl with
// centroids 4qd .. 4qd+3 and the partial squared norm of its chunk; through
// a wave-private LDS tile (one 16-byte store per group, four 16-byte loads),
// lane l gathers the k dot products and four partial norms of point l of
// the tile, and decides it alone: the expanded-form values, their minimum,
// and the candidates within twice the error bound E of the minimum (as in
// settle_survivor).  A single candidate is the nearest centroid; a point of
// several candidates reads its row and is decided on the direct-form
// distances (float64 for a near tie).  The clusters go back through LDS to
// the lanes that hold the rows, which add their chunks to the sums of the
// points' clusters.  Two tiles of loads are in flight per wave.
template <int KC>
__global__ __launch_bounds__(kTp) __attribute__((amdgpu_waves_per_eu(4))) void k_first(Dev P_, Fused F, int t) {
    const Dev P = with_scales(P_);
    IterState* st = P.st;
    if (st->done) {
        if (blockIdx.x == 0 && threadIdx.x == 0) st->active = 0;
        return;
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) st->active = 1;

    const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
    const int pl = lane & 15, qd = lane >> 4;
    StepFlags fl{true, true, false, P.gamma, st->ec_max, 0.f};
    const SmallLds lay = small_lds(P.k, false, false);
    const Tables T = load_tables(P, F, lay, t);
    clear_next_slots(P, F, t);
    // Wave-private tile: 64 rows of kCR floats (16 dot products, 4 partial
    // norms), then 64 cluster words ordered [pl][group].
    float* dt = reinterpret_cast<float*>(km_smem + lay.off_qr) + w * (64 * kCR + 64);
    int* bt = reinterpret_cast<int*>(dt + 64 * kCR);
    __syncthreads();
    fl.cnmax = centroid_norm_max(T, P.k);
    const int k = P.k;

    float a[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) a[s] = pl < k ? T.C[pl * kCR + 4 * qd + s] : 0.f;

    Counters cn;
    const int64_t n = P.n;
    const int64_t ntiles = (n + 63) / 64;
    const int64_t nw = 4 * (int64_t)gridDim.x;
    const f32x4* X4 = reinterpret_cast<const f32x4*>(P.X);

    f32x4 xA[4], xB[4];   // [g]: chunk qd of point 16g + pl of the tile
    auto prefetch = [&](f32x4 (&xb)[4], int64_t tl) __attribute__((always_inline)) {
        if (tl >= ntiles) return;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const int64_t row = min(tl * 64 + 16 * g + pl, n - 1);
            xb[g] = __builtin_nontemporal_load(X4 + row * kQD + qd);
        }
    };
    auto wave_sync = []() __attribute__((always_inline)) {
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    };

    float xm = 0.f;   // largest |x| of the rows this lane reads (NaN ignored)
    auto tile_body = [&](f32x4 (&xb)[4], int64_t tl) __attribute__((always_inline)) {
        const int64_t base = tl * 64;
        // 1. Products and partial norms of the four groups into the tile.
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const f32x4 xv = xb[g];
            xm = fmaxf(xm, fmaxf(fmaxf(fabsf(xv.x), fabsf(xv.y)), fmaxf(fabsf(xv.z), fabsf(xv.w))));
            f32x4 dot = __builtin_amdgcn_mfma_f32_16x16x4f32(a[0], xv.x, f32x4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
            dot = __builtin_amdgcn_mfma_f32_16x16x4f32(a[1], xv.y, dot, 0, 0, 0);
            dot = __builtin_amdgcn_mfma_f32_16x16x4f32(a[2], xv.z, dot, 0, 0, 0);
            dot = __builtin_amdgcn_mfma_f32_16x16x4f32(a[3], xv.w, dot, 0, 0, 0);
            float* row = dt + (16 * g + pl) * kCR;
            *reinterpret_cast<f32x4*>(row + 4 * qd) = dot;
            row[16 + qd] = fmaf(xv.x, xv.x, fmaf(xv.y, xv.y, fmaf(xv.z, xv.z, xv.w * xv.w)));
        }
        wave_sync();
        // 2. Point `lane` of the tile, decided by its own lane.
        const float* row = dt + lane * kCR;
        const f32x4 pn = *reinterpret_cast<const f32x4*>(row + 16);
        const float x2 = ((pn.x + pn.y) + pn.z) + pn.w;
        float V[KC];
        float vmin = INFINITY;
#pragma unroll
        for (int j = 0; j < KC; j += 4) {
            const f32x4 dv = *reinterpret_cast<const f32x4*>(row + j);
            const f32x4 cv = *reinterpret_cast<const f32x4*>(T.cn + j);
            const float dd[4] = {dv.x, dv.y, dv.z, dv.w};
            const float cc[4] = {cv.x, cv.y, cv.z, cv.w};
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                if (j + r < KC) {
                    V[j + r] = j + r < k ? fmaf(-2.f, dd[r], x2 + cc[r]) : INFINITY;
                    vmin = fminf(vmin, V[j + r]);
                }
            }
        }
        const float R = sqrtf(x2) * (1.0f + 0x1p-20f) + fl.cnmax;
        const float E = (kExpGamma * R * R + 4.f * R * fl.ecmax + 2.f * fl.ecmax * fl.ecmax) * kUp;
        const float lim = vmin + 2.f * E;
        uint32_t cm = 0;
#pragma unroll
        for (int j = 0; j < KC; ++j) cm |= (V[j] <= lim ? 1u : 0u) << j;
        cm &= (1u << k) - 1u;   // (an infinite minimum would admit the slots past k)
        int b = cm ? __builtin_ctz(cm) : 0;
        float ub = sqrt_up(fmaxf(vmin + E, 0.f)) * kUp;
        const bool valid = base + lane < n;
        if (__popc(cm) != 1 && valid) {   // rare: several candidates (none: a row that is not finite)
            float x[kD];
#pragma unroll
            for (int m = 0; m < kQD; ++m) {
                const f32x4 v = X4[(base + lane) * kQD + m];
                x[4 * m] = v.x;
                x[4 * m + 1] = v.y;
                x[4 * m + 2] = v.z;
                x[4 * m + 3] = v.w;
            }
            float Db;
            b = decide_direct(T, fl, P.C64, x, k, -1, cm, Db, ub, cn);
        }
        if (valid) {
            F.w[base + lane] = settle_state(ub, T.ddn[b], b);
            atomicAdd(&T.cnt[(lane & (2 * kCopies - 1)) * T.kp + b], 1u);
            cn.changed += 1;
            cn.comp += (uint32_t)k;
        }
        bt[(lane & 15) * 4 + (lane >> 4)] = b;
        wave_sync();
        // 3. The rows into the sums of their clusters, by the lanes that hold them.
        const int4 bs = *reinterpret_cast<const int4*>(bt + pl * 4);
        const int bb[4] = {bs.x, bs.y, bs.z, bs.w};
        const int cp = pl & (2 * kCopies - 1);
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            if (base + 16 * g + pl < n) {
                const f32x4 xv = xb[g];
                unsigned long long* dst =
                    reinterpret_cast<unsigned long long*>(T.acc + cp * T.csu + bb[g] * kSmallAccRow + 4 * qd);
                atomicAdd(dst + 0, (unsigned long long)fixed_bits((double)xv.x, P.qscale));
                atomicAdd(dst + 1, (unsigned long long)fixed_bits((double)xv.y, P.qscale));
                atomicAdd(dst + 2, (unsigned long long)fixed_bits((double)xv.z, P.qscale));
                atomicAdd(dst + 3, (unsigned long long)fixed_bits((double)xv.w, P.qscale));
            }
        }
        wave_sync();   // the tile is read before the next one is written
    };

    const int64_t w0 = 4 * (int64_t)blockIdx.x + w;
    prefetch(xA, w0);
    prefetch(xB, w0 + nw);
    for (int64_t tl = w0; tl < ntiles; tl += 2 * nw) {
        tile_body(xA, tl);
        prefetch(xA, tl + 2 * nw);
        if (tl + nw < ntiles) {
            tile_body(xB, tl + nw);
            prefetch(xB, tl + 3 * nw);
        }
    }
    if (F.amax) {   // this step scans X for the set-up: its largest |x| (infinity as the largest float)
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) xm = fmaxf(xm, __shfl_xor(xm, off));
        if (lane == 0) atomicMax(F.amax + kAmaxX, __float_as_uint(fminf(xm, FLT_MAX)));
    }
    flush_block(P, F, T, cn, false, t);
}

// After a first step that scanned X itself: its sums were formed at the scale
// of the sample's bound.  If X exceeded that bound, every row's image at the
// final scale minus its image at that scale is added to the step's
// accumulation rows, which then hold the sums at the final scale (exact
// modulo 2^64, whatever the first images were); else nothing is done.
__global__ __launch_bounds__(256) void k_first_fix(Dev P_, Fused F) {
    const Dev P = with_scales(P_);
    const int ex = sum_exp(F.amax);
    if (ex == bound_exp((double)__uint_as_float(F.amax[kAmaxSample])) + 4) return;   // the bound held
    __shared__ unsigned long long acc[kSmallMaxK * kD];
    for (int i = threadIdx.x; i < kSmallMaxK * kD; i += blockDim.x) acc[i] = 0;
    __syncthreads();
    const double qt = ldexp(1.0, sum_shift(ex, P.n));
    const int64_t total = P.n * kD;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int b = state_cluster(F.w[i / kD]);
        const double x = (double)P.X[i];
        atomicAdd(&acc[b * kD + (int)(i % kD)], (unsigned long long)(fixed_bits(x, qt) - fixed_bits(x, P.qscale)));
    }
    __syncthreads();
    unsigned long long* row = reinterpret_cast<unsigned long long*>(
        F.rows + ((int64_t)slot3(0) * kSmallRows + blockIdx.x % kSmallRows) * P.L);
    for (int i = threadIdx.x; i < P.k * kD; i += blockDim.x)
        if (acc[i]) atomicAdd(row + i, acc[i]);
}

// ---------------------------------------------------------------------------
// The incremental kernel (steps after the first).  Block b owns an equal
// share of the tiles of kIncWaveTile points; its waves take them one at a time
// from an LDS counter until none is left (the GPU form of the paper's work
// stealing against pruning skew), 16 points per lane loaded together, in four
// sub-tiles of four per lane.  The
// waves of a block run independently (no block barrier before the end): each
// queues its Clause-1 survivors in its own LDS queue and, whenever 64 are
// queued, gathers their rows (16-byte loads, four lanes per row), stages them
// in its own LDS rows and scans them one per lane.  Only the sums in LDS are
// shared, through atomics.

template <int KC, bool DENSE>
__global__ __launch_bounds__(kIncThreads) __attribute__((amdgpu_waves_per_eu(4))) void k_inc(Dev P_, Fused F, int t,
                                                                                      int fused) {
    const Dev P = with_scales(P_);
    IterState* st = P.st;
    // The wave index is uniform across the wave: held in a scalar register, so
    // that the tile loop below branches on scalars instead of lane masks.
    const int tid = threadIdx.x, w = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
    // Every load that does not depend on the stop flag is issued before the
    // flag is tested: the end of step t - 1 (fused start), the changed count
    // of step t - 1 and the stop settings, and (below) the first states.
    EosIn ein;
    if (fused) ein = eos_load(P, F, t - 1, true);
    const uint64_t chg_prev = fused ? F.stat[slot3(t - 1) * kNumStat + kStChanged] : 0;
    const double tol_n = st->tol_n;
    const int max_iters = st->max_iters;
    const int64_t n = P.n;
    const int nwt = (int)((n + kIncWaveTile - 1) / kIncWaveTile);   // wave tiles
    // Block b owns wave tiles [b * nwt / G, (b + 1) * nwt / G); its waves take
    // them one at a time from an LDS counter (work stealing within the block).
    const int wt_lo = (int)((int64_t)blockIdx.x * nwt / gridDim.x);
    const int wt_hi = (int)((int64_t)(blockIdx.x + 1) * nwt / gridDim.x);
    const uint4* W4 = reinterpret_cast<const uint4*>(F.w);
    // The states of a wave tile: sub-tile c of lane l holds points
    // base + 256c + 4l .. +3.
    uint4 sn[4];
    // Addressed as a scalar tile base plus the lane's 32-bit offset (kept
    // opaque so that it is not folded into a 64-bit per-lane address, which
    // would hold two more registers through the loop).
    auto load_states = [&](int wt) __attribute__((always_inline)) {
        const char* tw = reinterpret_cast<const char*>(W4) + (int64_t)wt * (4 * kIncWaveTile);   // padded past n
        uint32_t off = 16u * (uint32_t)lane;
        asm volatile("" : "+v"(off));
#pragma unroll
        for (int c = 0; c < 4; ++c) sn[c] = *reinterpret_cast<const uint4*>(tw + off + 1024 * c);
    };
    int wt = wt_lo + w;   // each wave's first tile
    if (st->done) {   // an earlier end of step stopped the run
        if (blockIdx.x == 0 && tid == 0) st->active = 0;
        return;
    }

    // The layout for the largest k: every LDS offset is a constant of the
    // code (immediate offsets, no registers held for them).
    const SmallLds lay = small_lds(kSmallMaxK, false);
    // Fused start: every block forms the end of step t - 1 itself (the same
    // integer totals and float64 operations, so the same tables) in the LDS of
    // the gathered rows, and block 0 stores it (and the bookkeeping).  The
    // float64 centroids of near-tie decisions are then the LDS copy.
    double* c64n = reinterpret_cast<double*>(km_smem + lay.off_c64);
    // (T is set once: its pointers stay constants of the code.)
    const Tables T = table_ptrs(P, lay);
    float ecmax;
    if (fused) {
        unsigned char* scr = km_smem + lay.off_qr;
        ecmax = eos_finish(P, F, t - 1, ein, blockIdx.x == 0, scr, &T, c64n);
        if (blockIdx.x == 0 && tid == 0) step_books(P, F, t - 1, ecmax);
        if ((double)chg_prev < tol_n || t >= max_iters) {   // the run stops after step t - 1
            if (blockIdx.x == 0 && tid == 0) st->active = 0;
            return;
        }
    } else {
        fill_tables(P, F, T, t);
        ecmax = st->ec_max;
        for (int i = tid; i < P.k * kD; i += kIncThreads) c64n[i] = P.C64[i];
    }
    // Dense form (DENSE): all rows streamed in order instead of the
    // survivors' gathered, for a step where most points survive Clause 1.
    constexpr bool dense = DENSE;
    // The first states are requested once the tables are formed (the end of
    // step holds many registers; the loads arrive during the table staging).
    if (wt < wt_hi && !dense) load_states(wt);
    if (blockIdx.x == 0 && tid == 0) st->active = 1;
    clear_next_slots(P, F, t);
    StepFlags fl{false, !(P.flags & KM_FLAG_NO_PRUNE), false, P.gamma, ecmax, 0.f};
    // Near-tie decisions read the float64 centroids from LDS (one address
    // space: plain LDS loads, whose waits the compiler counts exactly).
    const double* C64 = c64n;
    // Further tiles: lane 0 takes one from the block's counter (in the queue
    // counters, which this kernel does not otherwise use).
    auto grab = [&]() __attribute__((always_inline)) {
        int t = 0;
        if (lane == 0) t = wt_lo + kIncWaves + atomicAdd(T.qc, 1);
        return __builtin_amdgcn_readfirstlane(t);
    };
    int* wq_p = reinterpret_cast<int*>(km_smem + lay.off_qp) + w * kIncWaveQ;   // this wave's queue
    int* wq_a = reinterpret_cast<int*>(km_smem + lay.off_qa) + w * kIncWaveQ;
    float* wg = reinterpret_cast<float*>(km_smem + lay.off_qr) + 64 * w * kCR;  // its staged rows
    __syncthreads();
    fl.cnmax = centroid_norm_max(T, P.k);

    Counters cn;
    const f32x4* X4 = reinterpret_cast<const f32x4*>(P.X);
    const int rho0 = lane >> 2, q = lane & 3;

    // Batches of up to 64 of this wave's survivors, software-pipelined: a
    // batch's rows are requested when it is taken from the queue (16-byte
    // loads, load i of lane l = chunk l % 4 of batch entry 16i + l / 4) and
    // staged and scanned, one survivor per lane, at the next batch point or
    // at the end, so that the loads overlap the next tile's Clause-1 work.
    f32x4 r[kQD];
    // The batch in flight: its size, and each lane's entry (point, cluster)
    // parked in the spare words of the lane's staged row.
    int bcnt = 0;
    auto take_batch = [&](int e0, int cnt) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < kQD; ++i) {
            const int slot = 16 * i + rho0;
            const int64_t rp = slot < cnt ? (int64_t)wq_p[e0 + slot] : 0;
            r[i] = __builtin_nontemporal_load(X4 + rp * kQD + q);
        }
        int* park = reinterpret_cast<int*>(wg + lane * kCR + kD);
        park[0] = lane < cnt ? wq_p[e0 + lane] : 0;
        park[1] = lane < cnt ? wq_a[e0 + lane] : 0;
        bcnt = cnt;
    };
    auto scan_batch = [&]() __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < kQD; ++i) *reinterpret_cast<f32x4*>(wg + (16 * i + rho0) * kCR + 4 * q) = r[i];
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        if (lane < bcnt) {
            float x[kD];
#pragma unroll
            for (int c = 0; c < kQD; ++c) {
                const f32x4 v = *reinterpret_cast<const f32x4*>(wg + lane * kCR + 4 * c);
                x[4 * c] = v.x;
                x[4 * c + 1] = v.y;
                x[4 * c + 2] = v.z;
                x[4 * c + 3] = v.w;
            }
            const int* park = reinterpret_cast<const int*>(wg + lane * kCR + kD);
            settle_survivor<KC, true>(P, F, T, fl, C64, x, park[0], park[1], lane & (kCopies - 1), cn, nullptr);
        }
        bcnt = 0;
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();   // staged rows consumed before the next batch is staged
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    };

    if constexpr (dense) {
        // Dense form of an incremental step (all rows streamed): wave w of
        // the block takes 64-point tiles with a stride of all the grid's
        // waves, two tiles in flight.  The products are those of the first
        // step's tiles (16x16x4 matrix-core dot products through a
        // wave-private LDS tile, one point per lane, certified expanded-form
        // candidates), with each point's state: a point Clause 1 keeps is
        // counted and left alone (its state is not rewritten); a survivor with
        // a single candidate takes it (its state rewritten and, when its
        // cluster changed, its row moved between the sums by the lanes that
        // hold its chunks); a survivor with several candidates (or a row that
        // is not finite) is listed and settled as in the gathered form.
        const int pl = lane & 15, qd = lane >> 4, k = P.k;
        // (the tables' fields as plain locals: kept in registers)
        const float* __restrict__ t_thr = T.thr;
        const float* __restrict__ t_cn = T.cn;
        const float* __restrict__ t_h = T.h;
        const float* __restrict__ t_ddn = T.ddn;
        uint32_t* __restrict__ t_cnt = T.cnt;
        const int t_kp = T.kp;
        float* dt = wg;            // the wave's tile: its staged rows
        int* bt = wq_p;            // its moved-row list: the first 64 queue entries
        int* rl = wq_p + 64;       // its list: the rest of the queue
        int* ra = wq_a + 64;
        constexpr int rcap = kIncWaveQ - 64;
        float a[4];
#pragma unroll
        for (int s = 0; s < 4; ++s) a[s] = pl < k ? T.C[pl * kCR + 4 * qd + s] : 0.f;
        const int64_t ntiles = (n + 63) / 64;
        const int64_t nw = (int64_t)kIncWaves * gridDim.x;

        f32x4 xA[4], xB[4];   // [g]: chunk qd of point 16g + pl of the tile
        uint32_t sA = 0, sB = 0;   // the state of point `lane` of the tile
        int nl = 0;   // listed survivors (wave-uniform)
        // (A tile past the end loads the last tile again, unused: the registers
        // are then written on every path, so none is held across a drain.)
        auto prefetch = [&](f32x4 (&xb)[4], uint32_t& sb, int64_t tl) __attribute__((always_inline)) {
            const int64_t tc = min(tl, ntiles - 1);
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int64_t row = min(tc * 64 + 16 * g + pl, n - 1);
                xb[g] = __builtin_nontemporal_load(X4 + row * kQD + qd);
            }
            sb = F.w[tc * 64 + lane];   // the state array is padded past n
        };
        auto wave_sync = []() __attribute__((always_inline)) {
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        };
        auto tile_body = [&](const f32x4 (&xb)[4], uint32_t ws, int64_t tl) __attribute__((always_inline)) {
            const int64_t base = tl * 64;
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const f32x4 xv = xb[g];
                f32x4 dot = __builtin_amdgcn_mfma_f32_16x16x4f32(a[0], xv.x, f32x4{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
                dot = __builtin_amdgcn_mfma_f32_16x16x4f32(a[1], xv.y, dot, 0, 0, 0);
                dot = __builtin_amdgcn_mfma_f32_16x16x4f32(a[2], xv.z, dot, 0, 0, 0);
                dot = __builtin_amdgcn_mfma_f32_16x16x4f32(a[3], xv.w, dot, 0, 0, 0);
                float* row = dt + (16 * g + pl) * kCR;
                *reinterpret_cast<f32x4*>(row + 4 * qd) = dot;
                row[16 + qd] = fmaf(xv.x, xv.x, fmaf(xv.y, xv.y, fmaf(xv.z, xv.z, xv.w * xv.w)));
            }
            wave_sync();
            const bool valid = base + lane < n;
            const int inc = state_cluster(ws);
            const bool surv = valid && !(fl.prune && state_value(ws) <= t_thr[inc]);
            cn.c1 += valid && !surv ? 1u : 0u;
            int mv = -1;   // a moved point: new cluster | old cluster << 4
            bool listed = false;
            if (surv) {
                const float* row = dt + lane * kCR;
                const f32x4 pn = *reinterpret_cast<const f32x4*>(row + 16);
                const float x2 = ((pn.x + pn.y) + pn.z) + pn.w;
                // The expanded-form values, formed again from the tile for the
                // candidate mask (no register array held across the tile).
                auto vals = [&](int j, float (&v)[4]) __attribute__((always_inline)) {
                    const f32x4 dv = *reinterpret_cast<const f32x4*>(row + j);
                    const f32x4 cv = *reinterpret_cast<const f32x4*>(t_cn + j);
                    v[0] = j < k ? fmaf(-2.f, dv.x, x2 + cv.x) : INFINITY;
                    v[1] = j + 1 < k ? fmaf(-2.f, dv.y, x2 + cv.y) : INFINITY;
                    v[2] = j + 2 < k ? fmaf(-2.f, dv.z, x2 + cv.z) : INFINITY;
                    v[3] = j + 3 < k ? fmaf(-2.f, dv.w, x2 + cv.w) : INFINITY;
                };
                float vmin = INFINITY;
#pragma unroll
                for (int j = 0; j < KC; j += 4) {
                    float v[4];
                    vals(j, v);
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        if (j + r < KC) vmin = fminf(vmin, v[r]);
                }
                const float R = sqrtf(x2) * (1.0f + 0x1p-20f) + fl.cnmax;
                const float E = (kExpGamma * R * R + 4.f * R * fl.ecmax + 2.f * fl.ecmax * fl.ecmax) * kUp;
                const float lim = vmin + 2.f * E;
                uint32_t cm = 0;
#pragma unroll
                for (int j = 0; j < KC; j += 4) {
                    float v[4];
                    vals(j, v);
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        if (j + r < KC) cm |= (v[r] <= lim ? 1u : 0u) << (j + r);
                }
                cm &= (1u << k) - 1u;   // (an infinite minimum would admit the slots past k)
                if (__popc(cm) == 1) {
                    const int b = __builtin_ctz(cm);
                    const float ub = sqrt_up(fmaxf(vmin + E, 0.f)) * kUp;
                    cn.comp += fl.prune ? mti_count<KC>(t_h, fmaf(-2.f, row[inc], x2 + t_cn[inc]), inc, b, ub, E)
                                        : (uint32_t)k;
                    F.w[base + lane] = settle_state(ub, t_ddn[b], b);
                    if (b != inc) {
                        cn.changed += 1;
                        const int cp = lane & (kCopies - 1);
                        atomicAdd(&t_cnt[cp * t_kp + b], 1u);
                        atomicAdd(&t_cnt[cp * t_kp + inc], 0xFFFFFFFFu);
                        mv = b | inc << 4;
                    }
                } else {
                    listed = true;
                }
            }
            const uint64_t lm = __ballot(listed);
            if (listed) {
                const int e = nl + lanes_below(lm);
                rl[e] = (int)(base + lane);
                ra[e] = inc;
            }
            nl += __popcll(lm);
            // The moved rows out of their old clusters' sums and into the new
            // ones': the lanes that hold a moved row's chunks put them in its
            // row of the tile (its products are spent), then four lanes per row.
            const uint64_t mm = __ballot(mv >= 0);
            if (mm) {
                if (mv >= 0) bt[lanes_below(mm)] = lane | mv << 6;
                wave_sync();
#pragma unroll
                for (int g = 0; g < 4; ++g)
                    if ((mm >> (16 * g + pl)) & 1ull)
                        *reinterpret_cast<f32x4*>(dt + (16 * g + pl) * kCR + 4 * qd) = xb[g];
                wave_sync();
                move_rows(T, dt, bt, __popcll(mm), lane, P.qscale);
            }
            wave_sync();   // the tile is read before the next one is written
        };
        // The stream stops (its two tiles in flight discarded) when the next two
        // tiles could overflow the list; the list is settled with no tile held,
        // and the stream restarts at the next tile.
        int64_t tl = (int64_t)kIncWaves * blockIdx.x + w;
        while (tl < ntiles) {
            prefetch(xA, sA, tl);
            prefetch(xB, sB, tl + nw);
            for (; tl < ntiles;) {
                tile_body(xA, sA, tl);
                prefetch(xA, sA, tl + 2 * nw);
                if (tl + nw < ntiles) {
                    tile_body(xB, sB, tl + nw);
                    prefetch(xB, sB, tl + 3 * nw);
                }
                tl += 2 * nw;
                if (nl > rcap - 128) break;
            }
            for (int e0 = 0; e0 < nl; e0 += 64) {
                take_batch(64 + e0, min(nl - e0, 64));
                scan_batch();
            }
            nl = 0;
        }
        flush_block(P, F, T, cn, true, t);
        return;
    }

    int queued = 0;      // wave-uniform
    uint32_t c1w = 0;    // wave-uniform: points Clause 1 kept
    auto tile_body = [&](int base, const uint4 s4) __attribute__((always_inline)) {
        const uint32_t ws[4] = {s4.x, s4.y, s4.z, s4.w};
        const int p0 = base + 4 * lane;
        const int lim = (int)min((int64_t)256, n - base);   // points of the sub-tile before n
        float thr[4];   // the four thresholds requested together (padding states read cluster 0)
#pragma unroll
        for (int e = 0; e < 4; ++e) thr[e] = T.thr[state_cluster(ws[e])];
        int pos = queued;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const bool valid = 4 * lane + e < lim;
            const int a = state_cluster(ws[e]);
            const bool surv = valid && !(fl.prune && state_value(ws[e]) <= thr[e]);
            const uint64_t bm = __ballot(surv);
            if (surv) {
                const int e_pos = pos + lanes_below(bm);
                wq_p[e_pos] = p0 + e;
                wq_a[e_pos] = a;
            }
            pos += __popcll(bm);
        }
        // Clause 1 kept every valid point that was not queued (a wave count).
        c1w += (uint32_t)(min(max(lim, 0), 256) - (pos - queued));
        queued = pos;
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();   // queue entries visible to the whole wave
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    };
    // Sub-tiles, each followed by the batch point: while a full batch is
    // queued (at the end: any entry), scan the batch in flight and take the
    // newest entries as the next one; at the end the last batch is scanned
    // too.  One call site each keeps the scan code in one copy.  The next
    // wave tile is taken at the first sub-tile and its states requested at
    // the last.
    int sub = 0, wt_next = 0;
    for (;;) {
        const bool more = wt < wt_hi;
        if (more) {
            const uint4 s4 = sn[0];
            sn[0] = sn[1];   // the next sub-tile's states move to the front
            sn[1] = sn[2];
            sn[2] = sn[3];
            const int base = wt * kIncWaveTile + 256 * sub;
            if (sub == 0) wt_next = grab();
            if (sub == 3) {
                wt = wt_next;
                if (wt < wt_hi) load_states(wt);
            }
            sub = (sub + 1) & 3;
            tile_body(base, s4);
        }
        for (;;) {
            const bool take = more ? queued >= 64 : queued > 0;
            if (bcnt > 0 && (take || !more)) scan_batch();
            if (!take) break;
            const int c = queued < 64 ? queued : 64;
            queued -= c;
            take_batch(queued, c);
        }
        if (!more) break;
    }
    cn.c1 = lane == 0 ? c1w : 0u;
    flush_block(P, F, T, cn, true, t);
}

// End of step t as its own launch (one block): after a streaming step, and
// after an incremental step whose results are needed before the next step
// (then the next step starts unfused).
__global__ __launch_bounds__(kTp) void k_small_finish(Dev P_, Fused F, int t, int delta) {
    if (t == 0 && F.amax) {   // the first step scanned X: the final scales from its word
        if (threadIdx.x == 0) put_scales(P_.st, sum_exp(F.amax), __uint_as_float(F.amax[kAmaxC]), P_.n, P_.d);
        __syncthreads();
    }
    const Dev P = with_scales(P_);
    if (!P.st->active) return;   // step t did not run (the run had stopped)
    const float em = eos_finish(P, F, t, eos_load(P, F, t, delta != 0), true, km_smem, nullptr, nullptr);
    if (threadIdx.x == 0) step_books(P, F, t, em);
}

// Assignments from the point states.
__global__ __launch_bounds__(256) void k_small_unpack(const uint32_t* __restrict__ w, int64_t n,
                                                      int32_t* __restrict__ a) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
        a[i] = (int32_t)(w[i] & 15u);
}

// ---------------------------------------------------------------------------
// Host-side launchers and configuration.

bool small_applies(int64_t n, int d, int k, bool aligned) {
    // int32 point indices, also over the state array's padding
    return aligned && d == 16 && k <= kSmallMaxK && n <= (int64_t)INT_MAX - kIncTile;
}

// Distance slots of the survivor scan for k centroids: k rounded up to even.
#define KM_SMALL_KCS(X) X(2) X(4) X(6) X(8) X(10) X(12) X(14) X(16)

static int small_kc(int k) { return (k + 1) / 2 * 2; }

const void* small_kernel_symbol(int k) {
    switch (small_kc(k)) {
#define KM_SYM(KC_) \
    case KC_: return reinterpret_cast<const void*>(&k_small<KC_>);
        KM_SMALL_KCS(KM_SYM)
#undef KM_SYM
        default: return nullptr;
    }
}

const void* inc_kernel_symbol(int k, bool dense) {
    switch (small_kc(k)) {
#define KM_SYM(KC_) \
    case KC_: return dense ? reinterpret_cast<const void*>(&k_inc<KC_, true>) : reinterpret_cast<const void*>(&k_inc<KC_, false>);
        KM_SMALL_KCS(KM_SYM)
#undef KM_SYM
        default: return nullptr;
    }
}

int small_lds_bytes(int k) { return small_lds(k, true).bytes; }

int first_lds_bytes(int k) { return small_lds(k, false, false).bytes; }

const void* first_kernel_symbol(int k) {
    switch (small_kc(k)) {
#define KM_SYM(KC_) \
    case KC_: return reinterpret_cast<const void*>(&k_first<KC_>);
        KM_SMALL_KCS(KM_SYM)
#undef KM_SYM
        default: return nullptr;
    }
}

hipError_t launch_first(const Dev& dv, const Fused& F, int grid, int lds_bytes, int t, hipStream_t s) {
    switch (small_kc(dv.k)) {
#define KM_LAUNCH(KC_) \
    case KC_: hipLaunchKernelGGL((k_first<KC_>), dim3(grid), dim3(kTp), lds_bytes, s, dv, F, t); break;
        KM_SMALL_KCS(KM_LAUNCH)
#undef KM_LAUNCH
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

int inc_lds_bytes(int) { return small_lds(kSmallMaxK, false).bytes; }

int small_finish_lds_bytes(int k) { return finish_lds(16, k); }

hipError_t launch_small(const Dev& dv, const Fused& F, int lds_bytes, int t, hipStream_t s) {
    switch (small_kc(dv.k)) {
#define KM_LAUNCH(KC_)                                                                          \
    case KC_: hipLaunchKernelGGL((k_small<KC_>), dim3(dv.G), dim3(kTp), lds_bytes, s, dv, F, t); break;
        KM_SMALL_KCS(KM_LAUNCH)
#undef KM_LAUNCH
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_inc(const Dev& dv, const Fused& F, int grid, int lds_bytes, int t, int fused, bool dense,
                      hipStream_t s) {
    switch (small_kc(dv.k)) {
#define KM_LAUNCH(KC_)                                                                                          \
    case KC_:                                                                                                   \
        if (dense)                                                                                              \
            hipLaunchKernelGGL((k_inc<KC_, true>), dim3(grid), dim3(kIncThreads), lds_bytes, s, dv, F, t, fused);  \
        else                                                                                                    \
            hipLaunchKernelGGL((k_inc<KC_, false>), dim3(grid), dim3(kIncThreads), lds_bytes, s, dv, F, t, fused); \
        break;
        KM_SMALL_KCS(KM_LAUNCH)
#undef KM_LAUNCH
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}


hipError_t launch_first_fix(const Dev& dv, const Fused& F, int grid, hipStream_t s) {
    if (!F.amax || grid < 1 || dv.d != kD || dv.k > kSmallMaxK) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k_first_fix, dim3(grid), dim3(256), 0, s, dv, F);
    return hipGetLastError();
}

hipError_t launch_small_finish(const Dev& dv, const Fused& F, int t, int delta, hipStream_t s) {
    hipLaunchKernelGGL(k_small_finish, dim3(1), dim3(kTp), finish_lds(dv.d, dv.k), s, dv, F, t, delta);
    return hipGetLastError();
}

hipError_t launch_small_unpack(const Fused& F, int64_t n, int32_t* assign_out, hipStream_t s) {
    int64_t blocks = (n + 255) / 256;
    if (blocks > 8192) blocks = 8192;
    hipLaunchKernelGGL(k_small_unpack, dim3((unsigned)blocks), dim3(256), 0, s, F.w, n, assign_out);
    return hipGetLastError();
}

}  // namespace km
