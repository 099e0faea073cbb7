// Internal declarations shared by the kernels (km_kernels.hip) and the C-ABI
// host code (km_capi.hip).  Not installed; the public interface is
// include/kmeans_mti.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace km {

// Float64 rounding constant 1.5 * 2^52: for |v| < 2^51, fma(x, scale, kMagic)
// rounds x*scale to the nearest integer q and stores it in the low mantissa
// bits, so bits(result) = kMagicBits + q.  This gives an exact integer image
// of each input in two instructions, and sums of images are exact.
constexpr double kMagic = 6755399441055744.0;
constexpr uint64_t kMagicBits = 0x4338000000000000ull;

constexpr int kHistCap = 4096;   // per-iteration records kept (ring)
constexpr int kNumStat = 5;      // per-block counters appended to each partial row

// Partial-row layout (uint64 words): [0, k*d) coordinate sums (cluster-major),
// [k*d, k*d + k) member counts, then the counters below.
enum StatCol { kStChanged = 0, kStComputed = 1, kStClause1 = 2, kStRecheck = 3, kStInertia = 4 };

struct IterRec {
    int64_t changed, computed, clause1, rechecks;
    double inertia;   // NaN unless inertia is collected
};

// Device-resident loop state.  Written only by the kernels named per field.
struct IterState {
    int32_t t;            // steps completed (update kernel)
    int32_t done;         // stop test met (update kernel); read by the next step
    int32_t active;       // 1 if the current step runs (assignment kernel)
    int32_t converged;    // stopped on the tol test (update kernel)
    int32_t max_iters;    // stop after this many steps (host, at init)
    int32_t pad_;
    double tol_n;         // stop when changed < tol_n; negative: never (host)
    int64_t changed_last; // update kernel
    int64_t tot_computed, tot_clause1, tot_rechecks;   // update kernel
    double inertia_last;  // update kernel
    float ec_max;         // max_j ||c32_j - c64_j|| (centroid-table kernel)
    float pad2_;
    // Fixed-point scales (set-up kernel k_set_scales, from the largest |x|):
    // 2^S, 2^-S of the coordinate sums and the same for the inertia sum.
    double qscale, qinv, iscale, iinv;
    // Nullable: a pinned, coherent host word that the end of every step sets
    // to the steps ended, negated once the stop test is met (a run's host
    // loop polls it instead of copying the flag).
    int32_t* host;
};

// Everything the kernels need, passed by value.
struct Dev {
    const float* X;
    int64_t n;
    int32_t d, k;
    int32_t* a;           // n assignments
    float* u;             // n upper bounds
    double* C64;          // k*d master centroids
    float* C32;           // k*d float32 copy used for distances
    float* ec;            // k: ||c32_j - c64_j|| rounded up
    float* h;             // k*k: half centroid distances rounded down
    float* s;             // k: min_{j != i} h[i][j] rounded down (+inf if k == 1)
    float* f;             // k: drift ||c_j^t - c_j^{t-1}|| rounded up
    float* cn2;           // k: ||c32_j||^2 (matrix-core path)
    float* lb;            // Elkan only: k x n lower bounds (centroid-major), offset by the cumulative drift
    double* dhi;          // Elkan and incremental path: k cumulative drifts, rounded up (else null)
    double* dlo;          // Elkan and incremental path: k cumulative drifts, rounded down
    float* dupf;          // Elkan and incremental path: k cumulative drifts, rounded up to float32
    float* ddnf;          // incremental path: k cumulative drifts, rounded down to float32 (else null)
    uint32_t* w;          // incremental path: point states (cluster and bound, below), padded
    uint64_t* sums;       // incremental path: k*d + k exact sums and counts, carried across steps (else null)
    float* hm;            // incremental path: k x 4, min over centroid block cb of h[a][j] (h[a][a] = 0), else null
    uint64_t* part;       // G x L per-block partial rows
    uint64_t* total;      // L reduced row (zero between iterations)
    IterState* st;
    IterRec* rec;
    int32_t G;            // assignment blocks = partial rows
    int32_t L;            // partial row length
    double qscale, qinv;  // 2^S, 2^-S: fixed-point scale of coordinate sums (copied from st by each kernel)
    double iscale, iinv;  // fixed-point scale of the inertia sum (likewise)
    float gamma;          // relative error bound of a float32 squared distance, d-dependent
    uint32_t flags;
};

inline int row_len(int d, int k) { return k * d + k + kNumStat; }

// Global-memory path (centroids or per-cluster sums too large for LDS): dense
// matrix-core distances for the Clause-1 survivors, then per-cluster sums
// through a counting sort of the points by cluster.
constexpr int kLgM = 128;            // survivors per block tile (matrix-core columns)
constexpr int kLgN = 256;            // centroids per block tile (matrix-core rows)
constexpr int kLgK = 16;             // dimensions per streamed chunk
constexpr int kLgStages = 3;         // LDS ring stages (chunks loaded ahead: kLgStages - 1)
constexpr int kLgStageBytes = (kLgN + kLgM) * 4 * kLgK;   // one chunk of the centroid and survivor tiles
constexpr int kLgChunkRows = 256;    // rows per segment-sum chunk
constexpr int kLgBoundThreads = 1024;                 // threads per block of the bound pass
constexpr int kLgBoundWaves = kLgBoundThreads / 64;
constexpr int kLgBoundRounds = 4;                     // rounds of kLgBoundThreads points per block
constexpr int kLgBoundSpan = kLgBoundThreads * kLgBoundRounds;
constexpr int kLgTableSplit = 4;     // block columns (centroid ranges) of the tiled centroid table
constexpr int kLgMaxD = 4096;        // largest d of the global-memory path

// Split rows (the matrix-core operands of the global path): every float32
// value x is held as hi = bf16(x) and lo = bf16(x - hi), both rounded to
// nearest.  Row r, chunk c (dimensions 16c .. 16c + 15, zero past d) takes 16
// words: hi of dimensions 16c .. +7, hi of 16c + 8 .. +15, lo of 16c .. +7, lo
// of 16c + 8 .. +15 (two bf16 per word, the lower dimension in the low half).
inline int split_chunks(int d) { return (d + kLgK - 1) / kLgK; }

// Best centroid of one range of a survivor decided over all centroids.
struct FullPart {
    double D;
    int32_t j, rk;
};
constexpr int kFullCap = 4096;       // survivors per step whose decision is split over blocks
constexpr int kFullSplit = 8;        // blocks (centroid ranges) per split decision

struct Large {
    int32_t* surv;        // n: survivor point indices of the current step
    uint32_t* nsurv;      // survivor count
    uint32_t* cnt;        // Gs x k per-block cluster counts
    uint32_t* off;        // Gs x k per-block write offsets
    uint32_t* base;       // k + 1 cluster starts in perm
    uint32_t* cbase;      // k + 1 first segment chunk of each cluster
    int32_t* perm;        // n point indices grouped by cluster
    uint64_t* cpart;      // NCmax x d chunk partial sums (fixed point)
    uint64_t* ciq;        // NCmax chunk inertia partials (fixed point)
    uint32_t* xs;         // n split rows of X (set-up)
    float* x2;            // n: float32 squared norms of the rows of X (set-up)
    float* sx2;           // n: x2 of the survivors, in list order
    int32_t* fq;          // n: survivors (list entries) decided over all centroids
    uint32_t* nfull;      // their count
    FullPart* fpart;      // kFullCap x kFullSplit: the ranges' bests of the split decisions
    uint32_t* fcnt;       // kFullCap: ranges done per split survivor (reset by the combining block)
    int4* mq;             // n: survivors with 2-3 candidates (list entry, candidates, -1 for none)
    uint32_t* nmq;        // their count
    int4* mv;             // mvcap moves of the step: point, old cluster, new cluster
    uint32_t* nmv;        // their count (nsurv, nfull, nmq, nmv: zeroed by the centroid-table pass)
    int32_t mvcap;        // at most this many moves: incremental sums, else full sums
    uint32_t* cs;         // nct * kLgN split rows of the float32 centroids (rows >= k zero)
    float* cn2p;          // nct * kLgN: their float32 squared norms (rows >= k: +inf)
    float* smin;          // kLgTableSplit x k: column minima of the half-distance table (reduced to s)
    uint2* cand;          // n x nct x 2 x 4: per survivor, centroid tile and half of it, the four
                          // smallest expanded distances (float bits) with their centroids
    int32_t nch;          // chunks per split row
    int32_t nct;          // centroid tiles
    int32_t Gs;           // blocks of the histogram / scatter passes
    int32_t NCmax;        // n / kLgChunkRows + k
    int64_t span;         // points per histogram / scatter block (contiguous)
    int32_t Gm;           // resident blocks of the matrix-core kernel
    int32_t Gr;           // blocks of the refinement pass
};

// LDS bytes of the global-memory matrix-core kernel: the ring of streamed
// chunks and, by item parity, the centroid tile's and the survivors' squared
// norms and every wave's survivor rows.
__host__ __device__ inline int large_mfma_lds() {
    return kLgStages * kLgStageBytes + 2 * 4 * (kLgN + kLgM) + 2 * 4 * 256;
}

// Padded LDS row stride of the X tile: 16-byte aligned rows, offset by 4
// floats so that 16-byte row reads of consecutive lanes spread over banks.
__host__ __device__ inline int xs_stride(int d) { return ((d + 3) / 4) * 4 + 4; }

// Dynamic LDS layout of the assignment kernel for tile size tp.
struct AssignLds {
    int off_acc, off_cnt, off_c, off_f, off_s, off_ec, off_cn, off_h, off_x, off_sa, off_su, off_sd,
        off_sq, off_misc, off_ca, bytes;
};

// The matrix-core variants with four 32-centroid blocks run blocks of 512
// threads (two waves per SIMD) and read their centroid operands from LDS
// instead of registers.
__host__ __device__ inline bool assign_wide(int variant) { return variant % 16 == 4; }
// LDS bytes of those operands: 4 blocks x d/2 k-steps x 64 lanes.
__host__ __device__ inline int wide_ca_bytes(int d) { return 4 * (d / 2) * 64 * 4; }

// The vector survivor scans keep the half-distance table in LDS up to this k.
constexpr int kHLdsMaxK = 64;
// Whether the assignment kernel with KB (the variant's low 4 bits) keeps the
// half-distance table in LDS; the host sizes the LDS image with the same rule.
__host__ __device__ inline bool assign_h_lds(int kb, int k) { return (kb == 0 || kb == 8) && k <= kHLdsMaxK; }

// Centroid count rounded up to the 32-row blocks of the matrix-core path,
// whose variants use 1, 2 or 4 blocks (k <= 32, <= 64, <= 128).
__host__ __device__ inline int k_pad32(int k) {
    const int p = (k + 31) / 32 * 32;
    return p > 64 && p < 128 ? 128 : p;
}

__host__ __device__ inline AssignLds assign_lds(int d, int k, int tp, bool h_lds, bool wide = false) {
    AssignLds L;
    int o = 0;
    auto take = [&](int bytes, int align) {
        o = (o + align - 1) / align * align;
        int r = o;
        o += bytes;
        return r;
    };
    L.off_acc = take(8 * k * d, 16);
    L.off_cnt = take(4 * k, 16);
    L.off_c = take(4 * k * d, 16);
    L.off_f = take(4 * k, 16);
    L.off_s = take(4 * k, 16);
    L.off_ec = take(4 * k, 16);
    L.off_cn = take(4 * k_pad32(k), 16);
    L.off_h = take(h_lds ? 4 * k * k : 0, 16);
    L.off_x = take(4 * tp * xs_stride(d), 16);
    L.off_sa = take(4 * tp, 16);
    L.off_su = take(4 * tp, 16);
    L.off_sd = take(4 * tp, 16);
    L.off_sq = take(4 * tp, 16);
    L.off_misc = take(64, 16);   // two survivor counters (int) at 0, kNumStat uint64 counters at 16
    L.off_ca = take(wide ? wide_ca_bytes(d) : 0, 16);
    L.bytes = (o + 15) / 16 * 16;
    return L;
}

// Streaming path for small k and d = 16 (km_small.hip): the streaming kernel
// (every row of X read) or the incremental kernel (only the Clause-1
// survivors' rows read); the end of each step (sums, update, centroid table)
// runs in the next incremental kernel or in one block of its own.
constexpr int kSmallTile = 256;   // threads per block; points per tile of the streaming kernel
constexpr int kSmallMaxK = 16;    // the cluster index fits in the 4 low bits of the point state
constexpr int kSmallCopies = 4;   // copies of the LDS sums (spread rows over banks and addresses)
constexpr int kSmallRowStride = 20;   // padded LDS row stride (floats) of centroid and queued rows
constexpr int kSmallAccRow = 17;      // LDS stride (uint64) of one cluster's 16 fixed-point sums

// Accumulation rows of a streaming step: block b adds its partial row into
// row b % kSmallRows of the step's slot with device atomics; the end of the
// step sums them, and a later step's block 0 clears the slot for reuse.
constexpr int kSmallRows = 16;

// Incremental kernel: each block of kIncWaves waves (two blocks per CU at
// four waves per SIMD, so that the end of the previous step, which every
// block forms itself, is formed only twice per CU) owns an equal share of
// the tiles of kIncWaveTile points, which its waves take one at a time (16
// points per lane, four 16-byte state loads issued together), in four
// sub-tiles of 256.  The state array is padded to whole kIncTile.
constexpr int kIncWaves = 8;
// Incremental steps 1 .. kIncDenseSteps stream every row (the dense form)
// instead of gathering the survivors': right after the first step most
// points survive Clause 1 and nearly every 128-byte line of X holds a
// survivor's row.
constexpr int kIncDenseSteps = 1;
// The stream path's first step takes the largest |x| itself (no set-up scan
// of X) from this many values of X on.
constexpr int64_t kFuseScanMin = int64_t(1) << 20;
constexpr int kIncThreads = 64 * kIncWaves;
constexpr int kIncWaveTile = 1024;
constexpr int kIncTile = 4 * kIncWaveTile;

// Survivor queues in LDS.  A batch of kSmallTile survivors is scanned as soon
// as that many are queued, so a queue holds at most kSmallTile - 1 plus one
// tile's points.
constexpr int kSmallQ = 2 * kSmallTile;          // streaming kernel: rows staged with the entries
// Incremental kernel: one queue per wave (point index and cluster); a wave
// takes a batch of 64 as soon as that many are queued, and one sub-tile adds
// at most 256.
constexpr int kIncWaveQ = 64 + 256;
constexpr int kIncQ = kIncWaves * kIncWaveQ;

// Point state of the streaming path: one 32-bit word per point.  Bits 3..0
// hold the assigned cluster; the word with those bits cleared is a float32
// value v such that v + (cumulative drift of that cluster) is an upper bound
// on the point's distance to its centroid.  The drift of every later update
// is then added by the reader, so a point whose bound needs no tightening is
// never written.
struct Fused {
    // Buffers that one launch both reads and writes are kept in slots by step
    // index t (steps counted from 0): an incremental step finishes the step
    // before it in the same launch, so the step's inputs and outputs differ.
    uint64_t* rows;       // 3 slots x kSmallRows x L: slot t % 3 receives step t's sums (zero before)
    uint64_t* stat;       // 3 slots x kNumStat: step t's counters (device atomics of every block)
    uint64_t* sum;        // 2 slots x (k*d + k): exact sums and counts after step t, slot t % 2
    double* c64;          // 2 slots x k*d: float64 centroids used by step t (C^t), slot t % 2
    uint32_t* w;          // point states, n rounded up to kIncTile (padding zero)
    double* dhi;          // 2 slots x k: cumulative drift after t updates (D^t), rounded up, slot t % 2
    double* dlo;          // 2 slots x k: the same rounded down
    float* dup;           // k: the latest D rounded up to float32
    float* ddn;           // k: the latest D rounded down to float32
    // Set-up magnitude words when the first step scans X itself (the largest
    // |x| is written by that step), else null.
    uint32_t* amax = nullptr;
};

__host__ __device__ inline int slot3(int t) { return ((t % 3) + 3) % 3; }
__host__ __device__ inline int slot2(int t) { return t & 1; }

struct SmallLds {
    int off_c, off_h, off_s, off_ec, off_du, off_dd, off_cn, off_acc, off_cnt, off_qr, off_qp, off_qa, off_misc,
        off_c64, bytes;
    int csu, kp;          // stride (uint64) of one copy of the sums; of one copy of the counts
    int copies;           // copies of the sums and counts
};

// Dynamic LDS layout of the streaming (staged = true: queued rows kept in
// LDS) and incremental (staged = false: one batch of gathered rows) kernels.
__host__ __device__ inline SmallLds small_lds(int k, bool staged, bool queue = true) {
    SmallLds L;
    int o = 0;
    auto take = [&](int bytes, int align) {
        o = (o + align - 1) / align * align;
        int r = o;
        o += bytes;
        return r;
    };
    const int q = staged ? kSmallQ : kIncQ;
    // Cluster rows of kSmallAccRow uint64 (16 sums and one pad word), so that
    // the same coordinate of different clusters falls on different banks;
    // odd: the copies start on different banks.
    L.csu = kSmallAccRow * k + 1;
    L.kp = k + 1;
    L.off_c = take(4 * k * kSmallRowStride, 16);
    L.off_h = take(4 * k * kSmallMaxK, 16);   // rows padded to kSmallMaxK (16-byte row loads)
    L.off_s = take(4 * k, 16);
    L.off_ec = take(4 * k, 16);
    L.off_du = take(4 * k, 16);
    L.off_dd = take(4 * k, 16);
    L.off_cn = take(4 * k, 16);
    // (the first step, whose rows all go to the sums, spreads them over twice
    // as many copies)
    L.copies = queue ? kSmallCopies : 2 * kSmallCopies;
    L.off_acc = take(8 * L.copies * L.csu, 16);
    L.off_cnt = take(4 * L.copies * L.kp, 16);
    // Queued rows (streaming kernel) or one gathered batch (incremental kernel).
    // Without a queue (the matrix-core first step): per wave of the block, 64
    // rows of products and partial norms and 64 cluster words.
    L.off_qr = take(queue ? 4 * (staged ? kSmallQ : 64 * kIncWaves) * kSmallRowStride
                          : 4 * (kSmallTile / 64) * (64 * kSmallRowStride + 64),
                    16);
    L.off_qp = take(queue ? 4 * q : 0, 16);
    L.off_qa = take(queue ? 4 * q : 0, 16);
    L.off_misc = take(64, 16);   // three queue counters (int) at 0, kNumStat uint64 counters at 16
    // Incremental kernel: the float64 centroids of near-tie decisions.
    L.off_c64 = take(staged || !queue ? 0 : 8 * k * 16, 16);
    L.bytes = (o + 15) / 16 * 16;
    return L;
}

// LDS bytes of the end-of-step computation (new centroids in float64, the
// rounding errors of their float32 copies).
__host__ __device__ inline int finish_lds(int d, int k) { return 8 * k * d + 4 * k; }

bool small_applies(int64_t n, int d, int k, bool aligned);
const void* small_kernel_symbol(int k);
const void* inc_kernel_symbol(int k, bool dense);
int small_lds_bytes(int k);
int inc_lds_bytes(int k);
int small_finish_lds_bytes(int k);
// Step t of the streaming kernel (dv.C64 = the slot of C^t).
hipError_t launch_small(const Dev& dv, const Fused& F, int lds_bytes, int t, hipStream_t s);
// The first step without statistics on the matrix cores (k_first): LDS bytes,
// kernel symbol (occupancy query) and launch on `grid` blocks of kSmallTile.
int first_lds_bytes(int k);
const void* first_kernel_symbol(int k);
hipError_t launch_first(const Dev& dv, const Fused& F, int grid, int lds_bytes, int t, hipStream_t s);
// After a first step that scanned X itself (F.amax set): the correction of
// its sums when X exceeded the sample's bound (exits at once otherwise).
hipError_t launch_first_fix(const Dev& dv, const Fused& F, int grid, hipStream_t s);
// Step t of the incremental kernel.  fused: the end of step t - 1 (an
// incremental step of the same grid) has not run; every block computes it
// first and block 0 stores it.  Else dv.C64 = the slot of C^t.  dense: every
// row is streamed (the dense form) instead of the survivors' gathered.
hipError_t launch_inc(const Dev& dv, const Fused& F, int grid, int lds_bytes, int t, int fused, bool dense,
                      hipStream_t s);
// End of step t (one block).  delta: the rows hold the moves of an
// incremental step (added to the sums of step t - 1), else the full sums of
// a streaming step (they replace them).
hipError_t launch_small_finish(const Dev& dv, const Fused& F, int t, int delta, hipStream_t s);
// assign_out[i] = cluster of point i from the point states.
hipError_t launch_small_unpack(const Fused& F, int64_t n, int32_t* assign_out, hipStream_t s);

// Global-memory path launchers (km_large.hip).  gb: blocks of the bound pass.
hipError_t launch_large_assign(const Dev& dv, const Large& lg, int gb, hipStream_t s);
hipError_t launch_large_reduce(const Dev& dv, const Large& lg, hipStream_t s);
hipError_t launch_large_table(const Dev& dv, const Large& lg, int force, hipStream_t s);
// Split rows (and, with norms, float32 squared norms) of X, once at set-up.
hipError_t launch_large_split_x(const Dev& dv, const Large& lg, int cus, hipStream_t s);
int large_table_lds(int d);
const void* large_mfma_symbol();   // the matrix-core kernel
// Raises the dynamic-LDS limits of the global-memory path's kernels.
hipError_t large_set_attributes(int k, int d);

// Kernel launchers (km_kernels.hip).  Each returns the launch status.
// Set-up magnitude words (out[kAmax*], zero before): the largest |value| of a
// (na floats; na = 0 when the first step scans X itself), of b (nb floats)
// and of a fixed sample of the n x d rows of x (kAbsSampleChunks chunks of
// about 1024 values), as float bits (atomic max; NaN ignored, an infinite
// value counted as the largest float), and whether a or b holds a
// non-finite value.
hipError_t launch_absmax(const float* a, int64_t na, const float* b, int64_t nb, const float* x, int64_t n,
                         int32_t d, int cus, uint32_t* out, hipStream_t s);

// Buffers cleared and the loop state written by one set-up launch.
struct ZeroRanges {
    static constexpr int kMax = 16;
    void* p[kMax];        // 16-byte aligned
    uint64_t bytes[kMax]; // multiples of 4
    int32_t n;
    int32_t max_iters;    // loop state written to *st (when st is not null)
    double tol_n;
    IterState* st;
    int32_t* host;        // its progress word (nullable)
    bool overflow;        // more than kMax ranges were added (the launch refuses)
    void add(void* q, uint64_t b) {
        if (n >= kMax) {
            overflow = true;
            return;
        }
        p[n] = q;
        bytes[n] = b;
        ++n;
    }
};
hipError_t launch_init_buffers(const ZeroRanges& z, int cus, hipStream_t s);
// Fixed-point scales into st from the largest |x| and |c0| (float bits in
// absmax[0] and absmax[2]; unit = 1: spherical k-means, centroids of norm 1).
hipError_t launch_set_scales(IterState* st, const uint32_t* absmax, int64_t n, int32_t d, int unit, hipStream_t s);
hipError_t launch_set_centroids(const float* C0, double* C64, float* C32, float* ec, int64_t kd,
                                int32_t k, hipStream_t s);
// Spherical k-means: rows of X projected to the unit sphere into Xn; unit
// centroids from C0 (*zero set for a zero row).
hipError_t launch_normalize_rows(const float* X, int64_t n, int32_t d, float* Xn, hipStream_t s);
hipError_t launch_set_centroids_unit(const float* C0, double* C64, float* C32, float* ec, int32_t k, int32_t d,
                                     int32_t* zero, hipStream_t s);
hipError_t launch_assign(const Dev& dv, int variant, int tp, int lds_bytes, hipStream_t s);
hipError_t launch_reduce(const Dev& dv, hipStream_t s);
hipError_t launch_update(const Dev& dv, hipStream_t s);
hipError_t launch_centroid_table(const Dev& dv, int force, hipStream_t s);

// Assignment-kernel variant for (d, k): 16 * D + KB, where D is the
// compile-time dimension (16, 32; 0 = generic, any d) and KB the number of
// 32-centroid blocks of the matrix-core survivor path (0 = vector path,
// 8 = Elkan's lower-bound scan on the vector units).
// The specialised dimensions read X with 16-byte loads and need a 16-byte
// aligned X; vector_only selects KB = 0.
int assign_variant(int d, int k, bool aligned, bool vector_only, bool elkan);
// Kernel symbol of an assignment-kernel variant (for occupancy queries).
const void* assign_kernel_symbol(int variant);


// Incremental matrix-core step (km_incmm.hip), d = 16 or 32, k <= 128: the
// point states are streamed (4 bytes per point), only the Clause-1
// survivors' rows are gathered, and the sums move the rows of the points
// whose cluster changed (the running sums are carried in Dev::sums).
// Point state: bits 6..0 the cluster, the word with those bits cleared a
// float32 value v (rounded up) with v + D_a an upper bound on the point's
// distance to its centroid, D_a the cumulative drift of its cluster.
constexpr int kIMWaves = 8;          // waves per block
constexpr int kIMBatch = 32;         // survivors per matrix-core batch
constexpr int kIMSub = 64;           // points per Clause-1 sub-step of a wave (one per lane)
constexpr int kIMTile = 4 * kIMSub;  // points a wave takes at once; the state array is padded to it
constexpr int kIMQcap = kIMBatch + kIMSub;   // entries of one survivor queue
constexpr int kIMMaxK = 128;

// Survivor queues of a wave: one per set of 32-centroid blocks a survivor
// needs (KB <= 2: 1 or 3 sets), or one per block of its cluster (KB = 4).
__host__ __device__ constexpr int inc_mm_queues(int KB) { return KB == 4 ? 4 : (1 << KB) - 1; }

struct IncMMLds {
    int off_c, off_ca, off_cn, off_thr, off_ec, off_ddn, off_dup, off_hm, off_nb, off_acc, off_cnt, off_misc, off_q,
        off_x, bytes;
};

// Every offset depends on D and KB only (constants of each kernel variant).
__host__ __device__ inline IncMMLds inc_mm_lds(int D, int KB) {
    IncMMLds L;
    int o = 0;
    auto take = [&](int bytes) {
        o = (o + 15) / 16 * 16;
        int r = o;
        o += bytes;
        return r;
    };
    const int kp = 32 * KB;
    L.off_c = take(4 * kp * D);                          // float32 centroid rows
    L.off_ca = take(KB == 4 ? 4 * KB * (D / 2) * 64 : 0); // matrix-core operands (KB = 4)
    L.off_cn = take(4 * kp);                             // squared centroid norms
    L.off_thr = take(4 * kIMMaxK);                       // Clause-1 thresholds
    L.off_ec = take(4 * kIMMaxK);
    L.off_ddn = take(4 * kIMMaxK);
    L.off_dup = take(4 * kIMMaxK);
    L.off_hm = take(4 * kIMMaxK * 4);                    // min half-distance from a cluster to each block
    L.off_nb = take(4 * kp);                             // -|c|^2 / 2 of each centroid (-huge for padding)
    L.off_acc = take(8 * kp * (D + 1));                  // fixed-point sums of the moves (rows of D + 1)
    L.off_cnt = take(4 * kp);
    L.off_misc = take(64);                               // tile counter at 0, kNumStat uint64 counters at 16
    L.off_q = take(kIMWaves * 2 * inc_mm_queues(KB) * kIMQcap * 4);   // per wave: queues of (point, state)
    L.off_x = take(kIMWaves * kIMBatch * (D + 4) * 4);   // per wave: the batch's rows (+ 4 spare words)
    L.bytes = (o + 15) / 16 * 16;
    return L;
}

bool inc_mm_applies(int64_t n, int d, int k, bool aligned);
int inc_mm_kb(int k);
const void* inc_mm_symbol(int d, int k);
// One step (first: no bounds yet, every point is scanned).
hipError_t launch_inc_mm(const Dev& dv, int grid, int lds_bytes, int first, hipStream_t s);
// assign_out[i] = cluster of point i from the point states.
hipError_t launch_inc_mm_unpack(const Dev& dv, int32_t* assign_out, hipStream_t s);

// k-means++ seeding (km_pp.hip).  Points are processed in chunks of
// kPPChunk rows, one workgroup per chunk; the block weight sums are per chunk.
constexpr int kPPChunk = 2048;

struct PPArgs {
    const float* X;       // n x d rows
    int64_t n;
    int32_t d, k;
    float* C;             // k x d seed rows (output)
    int64_t* idx;         // k seed indices
    const double* u;      // k uniforms in [0, 1)
    double* D2;           // n: squared distance to the nearest seed so far
    int32_t* A;           // n: index of that seed (pruning only)
    uint64_t* bs;         // G: block weight sums of the next draw
    uint64_t* Mb;         // k: bits of max D2 after the pass with seed t
    double* dcc;          // k: lower bounds of ||c_a - c_new||^2 (pruning only)
    uint64_t* cnt;        // 2k: distances computed and rows improved per pass, or null
    int32_t G;            // chunks = ceil(n / kPPChunk)
    int32_t L;            // smallest L with n <= 2^L
    int32_t prune;        // 1: triangle-inequality skip test
};

// Kernel launches of one seeding.
int pp_launches(int k, int d, bool prune);
// Enqueues the whole seeding.  i0 = first seed index.  ev (nullable):
// pp_launches + 1 events, recorded before the first launch and after every
// launch; kind[j] (with ev) = 0 for the first pass, 1 for a later pass and 2
// for the other kernels, per launch j.
// vw: row loads, 0 scalar, 1 16-byte (d % 4 == 0, 16-byte aligned rows), 2 the
// same with whole 128-byte lines per step (d % 32 == 0).
hipError_t launch_pp_seed(const PPArgs& P, int64_t i0, int vw, hipEvent_t* ev, int8_t* kind, hipStream_t s);

}  // namespace km
