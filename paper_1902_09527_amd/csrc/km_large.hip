// Global-memory path of the MTI k-means hot path for gfx950 (MI355X), used
// when the centroids or the per-cluster sums do not fit in LDS (large k*d,
// e.g. k = 1000, d = 256).  One iteration (one ||Lloyd's MM step, paper
// section III-B) is:
//   k_bound_large       drift-updated bound and Clause 1 (section III-C) for
//                       every point; survivors compacted into a global list;
//   k_mfma_large        distances of the survivors to all centroids on the
//                       matrix cores (128-survivor x 128-centroid work items,
//                       split-bf16 products over 16-dimension chunks streamed
//                       into LDS by direct loads, expanded form): the four
//                       smallest per survivor and centroid tile;
//   k_refine_large      per survivor, the candidates within the expanded
//                       form's error bound; a lone candidate settles it;
//   k_multi_large,
//   k_full_large        two or three candidates: direct form and the
//                       float64 near-tie rule; four or more: float64 over
//                       all centroids;
//   k_hist_large        per-block cluster counts of the new assignment;
//   k_scan_large_cols,
//   k_scan_large_clusters  cluster starts and per-block write offsets;
//   k_scatter_large     point indices grouped by cluster (counting sort);
//   k_segsum_large      exact fixed-point sums over chunks of each cluster;
//   k_chunk_reduce_large  per-cluster sums, counts and the inertia into the
//                       reduced row read by k_update;
//   k_centroid_table_tiled  half centroid distances for the next step;
//   k_split_rows        split operand rows of the new centroids with their
//                       squared norms and the per-centroid minimum s of the
//                       table (and, once at set-up, split rows of X).
// The order of points inside a cluster segment is not fixed, but every sum
// is an exact integer sum, so results are bitwise reproducible.
#include <float.h>
#include <limits.h>
#include <math.h>

#include "kmeans_mti.h"
#include "km_device.h"
#include "km_internal.h"

namespace km {

namespace {

constexpr int kTiTile = 16;   // centroid rows per block of the tiled centroid table
constexpr int kTiSplit = kLgTableSplit;
constexpr int kRefineFlush = 128;   // LDS entries of the refinement pass that trigger a flush

// Insert (v, j) into an ascending 4-list ordered by value, then index.
__device__ inline void top4_insert(float (&L)[4], int (&J)[4], float v, int j) {
    if (!(v < L[3] || (v == L[3] && j < J[3]))) return;
    L[3] = v;
    J[3] = j;
#pragma unroll
    for (int q = 3; q > 0; --q) {
        const bool sw = L[q] < L[q - 1] || (L[q] == L[q - 1] && J[q] < J[q - 1]);
        if (sw) {
            const float tv = L[q];
            L[q] = L[q - 1];
            L[q - 1] = tv;
            const int tj = J[q];
            J[q] = J[q - 1];
            J[q - 1] = tj;
        }
    }
}

// Adds each of n counters (summed over the block) to its slot of the step's
// statistics, one atomic per counter and block (per-wave atomics on the same
// words serialize).  Every thread of the block calls it.
template <int N>
__device__ __forceinline__ void add_stats_block(uint64_t* total, const int (&slot)[N], uint64_t (&v)[N]) {
    __shared__ uint64_t part[N][16];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, nw = blockDim.x >> 6;
#pragma unroll
    for (int c = 0; c < N; ++c) {
        v[c] = wave_sum_u64(v[c]);
        if (lane == 0) part[c][wave] = v[c];
    }
    __syncthreads();
    if (threadIdx.x < N) {
        uint64_t s = 0;
        for (int w = 0; w < nw; ++w) s += part[threadIdx.x][w];
        if (s) atomicAdd(reinterpret_cast<unsigned long long*>(total + slot[threadIdx.x]), (unsigned long long)s);
    }
}

// The step's per-cluster sums come from its moves (added to the running
// sums kept by k_update) when few points moved; otherwise from the counting
// sort and exact segment sums.  The first step, and steps that gather the
// inertia, always take the full sums.
__device__ __forceinline__ bool large_incremental(const Dev& P, const Large& Lg) {
    return P.st->t > 0 && !(P.flags & KM_FLAG_STATS) && *Lg.nmv <= (uint32_t)Lg.mvcap;
}

}  // namespace

// ---------------------------------------------------------------------------
// Bound update and Clause 1 for every point; survivors to the global list.

__global__ __launch_bounds__(kLgBoundThreads) void k_bound_large(Dev P, Large Lg) {
    IterState* st = P.st;
    if (st->done) {
        if (blockIdx.x == 0 && threadIdx.x == 0) st->active = 0;
        return;
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) st->active = 1;
    const bool first = st->t == 0;
    const bool prune = !(P.flags & KM_FLAG_NO_PRUNE);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    __shared__ uint32_t cnt[kLgBoundRounds * kLgBoundWaves], base[kLgBoundRounds * kLgBoundWaves];
    // Block b owns points [b kLgBoundSpan, (b + 1) kLgBoundSpan): the flags
    // of its rounds stay in a bit mask, the block's survivors take one atomic
    // on the list counter (few, large blocks: atomics on one counter are
    // serialized), then every survivor its place (block order, then point
    // order).
    const int64_t lo = (int64_t)blockIdx.x * kLgBoundSpan, hi = min(P.n, lo + kLgBoundSpan);
    uint64_t c1 = 0;
    uint32_t mask = 0;
#pragma unroll
    for (int r = 0; r < kLgBoundRounds; ++r) {
        const int64_t i = lo + kLgBoundThreads * r + tid;
        bool surv = false;
        if (i < hi) {
            if (first) {
                surv = true;
            } else {
                const int a = P.a[i];
                const float u = (P.u[i] + P.f[a]) * kUp;
                if (!prune || u > P.s[a]) {
                    surv = true;
                } else {
                    c1 += 1;
                    P.u[i] = u;
                }
            }
        }
        mask |= (surv ? 1u : 0u) << r;
        const uint64_t m = __ballot(surv);
        if (lane == 0) cnt[kLgBoundWaves * r + wave] = (uint32_t)__popcll(m);
    }
    __syncthreads();
    if (tid == 0) {
        uint32_t tot = 0;
        for (int q = 0; q < kLgBoundRounds * kLgBoundWaves; ++q) {
            base[q] = tot;
            tot += cnt[q];
        }
        const uint32_t b0 = tot ? atomicAdd(Lg.nsurv, tot) : 0u;
        for (int q = 0; q < kLgBoundRounds * kLgBoundWaves; ++q) base[q] += b0;
    }
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kLgBoundRounds; ++r) {
        const bool surv = (mask >> r) & 1u;
        const uint64_t m = __ballot(surv);
        if (surv) {
            const int64_t i = lo + kLgBoundThreads * r + tid;
            const uint32_t pos = base[kLgBoundWaves * r + wave] + (uint32_t)__popcll(m & ((1ull << lane) - 1ull));
            Lg.surv[pos] = (int32_t)i;
            Lg.sx2[pos] = Lg.x2[i];
        }
    }
    {
        const int slot[1] = {P.k * P.d + P.k + kStClause1};
        uint64_t v[1] = {c1};
        add_stats_block<1>(P.total, slot, v);
    }
}

// ---------------------------------------------------------------------------
// Split rows: hi = bf16(x), lo = bf16(x - hi) (both rounded to nearest; x - hi
// is exact in float32), in the chunk layout of the matrix-core operands, and
// the float32 squared norm of every row (each lane sums its dimensions in
// order, then a fixed butterfly over the wave: deterministic).  Rows from
// valid to rows are padding: zero operands, norm +inf.  One wave per row.

__global__ __launch_bounds__(256) void k_split_rows(const float* __restrict__ src, int64_t rows, int64_t valid, int d,
                                                    int nch, uint32_t* __restrict__ dst, float* __restrict__ norms,
                                                    const IterState* st, int force, const float* __restrict__ smin,
                                                    float* __restrict__ s_out) {
    if (st && !force && !st->active) return;
    const int lane = threadIdx.x & 63;
    const int64_t wstride = (int64_t)gridDim.x * (blockDim.x >> 6);
    for (int64_t r = (int64_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6); r < rows; r += wstride) {
        const bool pad = r >= valid;
        const float* x = src + (pad ? 0 : r) * d;
        uint32_t* o = dst + r * nch * 16;
        float sq = 0.f;
        for (int g = lane; g < 2 * nch; g += 64) {   // 8-dimension group g: chunk g / 2, half g % 2
            const int m0 = 8 * g;
            float v[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) v[e] = !pad && m0 + e < d ? x[m0 + e] : 0.f;
            uint32_t hw[4], lw[4];
#pragma unroll
            for (int p = 0; p < 4; ++p) {
                float ra, rb;
                hw[p] = split_hi(v[2 * p], v[2 * p + 1], ra, rb);
                lw[p] = split_lo(ra, rb);
                sq = fmaf(v[2 * p], v[2 * p], sq);
                sq = fmaf(v[2 * p + 1], v[2 * p + 1], sq);
            }
            uint32_t* oc = o + (g >> 1) * 16 + 4 * (g & 1);
            *reinterpret_cast<uint4*>(oc) = make_uint4(hw[0], hw[1], hw[2], hw[3]);
            *reinterpret_cast<uint4*>(oc + 8) = make_uint4(lw[0], lw[1], lw[2], lw[3]);
        }
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) sq += __shfl_xor(sq, off);
        if (lane == 0) {
            norms[r] = pad ? INFINITY : sq;
            if (smin && !pad) {   // min over j != r of the half distances: the table's column minima
                float m = INFINITY;
                for (int y = 0; y < kTiSplit; ++y) m = fminf(m, smin[(int64_t)y * valid + r]);
                s_out[r] = m;
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Dense survivor distances on the matrix cores.  A work item is one tile of
// kLgM = 128 survivors against one tile of kLgN = 256 centroids; wave
// (wr, wc) of the block owns centroid rows 128 wr .. +127 and survivor
// columns 64 wc .. +63, eight 32x32 float32 accumulators.  Each product x.c
// is formed from the split operands as hi.hi + hi.lo + lo.hi: three bf16
// products on v_mfma_f32_32x32x16_bf16 (16 dimensions each) in place of
// eight float32 ones, with the dropped lo.lo term and the accumulation
// inside the error bound used by the refinement pass.
//
// The 16-dimension chunks of a block's items form one stream that runs
// kLgStages - 1 chunks ahead of the products, across item boundaries (the
// next item's first chunks load during the current item's selection).  They
// go from the split rows straight into a ring of kLgStages LDS stages by
// global_load_lds_dwordx4 (no registers held); a stage is two tiles (256
// and 128 rows x 64 bytes) in 1 KB groups of 16 rows, the four 16-byte
// pieces of each row permuted by lg_swz so that the operand reads of eight
// (and of sixteen) consecutive lanes fall on distinct banks.  Loads return
// in order, so chunk g has landed once at most the loads issued after it
// are outstanding.  Loads in flight per CU are bounded by LDS, so the tile
// is wide: 24 products per wave and chunk for 24 KB.
//
// Work items are ordered so that the nct items of a survivor tile carry
// indices congruent modulo 8: with a resident grid whose size is a multiple
// of 8, they run at the same time on one XCD and its L2 serves the survivor
// rows to all of them (each row leaves HBM about once per step).
//
// Selection: each expanded distance |x|^2 + |c|^2 - 2 x.c is clamped at 0
// (the true distance is >= 0, so the error bound still holds) and packed
// with its centroid into one ordered 32-bit key: the float's bits with the
// low 8 bits (6 within a lane's list) replaced by the centroid's place in
// the item, which lowers the value by less than 2^-15 of itself.  A lane
// keeps, per survivor column, the four smallest keys by min and med3
// (branch-free); the two half-waves' lists of a column are merged by a lane
// swap, and each wave writes the four smallest (value, centroid) pairs of
// its 128 centroids to the candidate buffer.

__device__ __forceinline__ int lg_swz(int rho) { return ((rho >> 2) & 3) ^ (((rho >> 1) & 1) << 1); }

__device__ __forceinline__ uint32_t med3u(uint32_t a, uint32_t b, uint32_t c) {
    uint32_t r;
    asm("v_med3_u32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
    return r;
}

// Insert key v into the ascending 4-list L.
__device__ __forceinline__ void key4_insert(uint32_t (&L)[4], uint32_t v) {
    const uint32_t l0 = min(L[0], v), l1 = med3u(L[0], L[1], v), l2 = med3u(L[1], L[2], v),
                   l3 = med3u(L[2], L[3], v);
    L[0] = l0;
    L[1] = l1;
    L[2] = l2;
    L[3] = l3;
}

// Sort 4 keys ascending (five compare-exchanges).
__device__ __forceinline__ void sort4(uint32_t (&L)[4]) {
    auto cx = [&](int i, int j) __attribute__((always_inline)) {
        const uint32_t a = L[i], b = L[j];
        L[i] = min(a, b);
        L[j] = max(a, b);
    };
    cx(0, 1);
    cx(2, 3);
    cx(0, 2);
    cx(1, 3);
    cx(1, 2);
}

typedef __attribute__((address_space(3))) void* lds_ptr;

__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void k_mfma_large(Dev P, Large Lg) {
    IterState* st = P.st;
    if (!st->active) return;
    const int ns = (int)*Lg.nsurv;
    const int nch = Lg.nch, nct = Lg.nct;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, col = lane & 31, half = lane >> 5;
    const int wr = wave >> 1, wc = wave & 1;
    extern __shared__ __align__(16) unsigned char smem[];
    // [2][kLgN + kLgM] by item parity: |c|^2 of the centroid tile, then |x|^2 of the survivors.
    float* nrm = reinterpret_cast<float*>(smem + kLgStages * kLgStageBytes);
    int32_t* meta = reinterpret_cast<int32_t*>(nrm + 2 * (kLgN + kLgM));   // [2][4 waves][64]: survivor rows

    const int nst = (ns + kLgM - 1) / kLgM;
    const int per_round = 8 * nct;
    const int64_t nitems = (int64_t)((nst + 7) / 8) * per_round;
    const int G = gridDim.x;
    auto tile_of = [&](int64_t w, int& s0, int& n0) __attribute__((always_inline)) {
        const int64_t r = w / per_round;
        const int rem = (int)(w - r * per_round);
        s0 = (int)(r * 8 + (rem & 7)) * kLgM;
        n0 = (rem >> 3) * kLgN;
    };
    auto next_valid = [&](int64_t w) __attribute__((always_inline)) {
        for (; w < nitems; w += G) {
            int s0, n0;
            tile_of(w, s0, n0);
            if (s0 < ns) break;
        }
        return w;
    };

    // DMA role of this lane in a 16-row group: row rho, LDS slot lane, piece
    // (lane % 4) ^ lg_swz(rho) of the row's chunk.  This wave streams
    // centroid rows 64 wave .. +63 (groups 4 wave .. 4 wave + 3) and
    // survivor rows 32 wave .. +31 (groups 2 wave, 2 wave + 1).
    const int rho = lane >> 2, piece = (lane & 3) ^ lg_swz(rho);
    const int sr0 = 32 * wave + rho;
    // Operand reads of lane (col, half): row col of a 32-row block, pieces
    // half (hi) and 2 + half (lo), at these offsets in its 1 KB group.
    const int rr = col & 15;
    const int offh = 16 * (4 * rr + (half ^ lg_swz(rr))), offl = 16 * (4 * rr + ((2 + half) ^ lg_swz(rr)));
    const int ga = (8 * wr + (col >> 4)) * 1024, gb = kLgN * 64 + (4 * wc + (col >> 4)) * 1024;
    const int64_t rowb = (int64_t)nch * 64;   // bytes per split row
    const unsigned char* csb = reinterpret_cast<const unsigned char*>(Lg.cs) + 16 * piece;
    const unsigned char* xsb = reinterpret_cast<const unsigned char*>(Lg.xs) + 16 * piece;
    const float* __restrict__ cn2p = Lg.cn2p;
    const float* __restrict__ sx2 = Lg.sx2;
    const int32_t* __restrict__ surv = Lg.surv;
    // Item metadata goes to LDS by direct loads too (nothing loaded is held
    // in registers across the loop): the survivor rows of this wave's two
    // row groups (lane l: row 32 wave + l % 32; rows past the list repeat
    // the first), the 256 centroid squared norms (64 per wave) and the 128
    // survivor squared norms (waves 0-1; survivors past the list read the
    // first).
    auto load_meta = [&](int s0, int par) __attribute__((always_inline)) {
        const int r = 32 * wave + (lane & 31);
        __builtin_amdgcn_global_load_lds(surv + s0 + (s0 + r < ns ? r : 0), (lds_ptr)(meta + par * 256 + wave * 64),
                                         4, 0, 0);
    };
    auto load_norms = [&](int s0, int n0, int par) __attribute__((always_inline)) {
        float* dst = nrm + par * (kLgN + kLgM) + 64 * wave;
        __builtin_amdgcn_global_load_lds(cn2p + n0 + tid, (lds_ptr)(dst), 4, 0, 0);
        if (wave < 2) {
            const int sl = tid;
            __builtin_amdgcn_global_load_lds(sx2 + s0 + (s0 + sl < ns ? sl : 0), (lds_ptr)(dst + kLgN), 4, 0, 0);
        }
    };

    // Issue cursor: item wi, its next chunk ci, its parity ipar; wn the item
    // after it.
    int64_t wi = next_valid(blockIdx.x);
    if (wi >= nitems) return;
    int is0, in0;
    tile_of(wi, is0, in0);
    int64_t wn = next_valid(wi + G);
    const unsigned char *pa, *pb0, *pb1;
    {
        const int rows = min(kLgM, ns - is0);
        const int q0 = surv[is0 + (sr0 < rows ? sr0 : 0)], q1 = surv[is0 + (sr0 + 16 < rows ? sr0 + 16 : 0)];
        pa = csb + (int64_t)(in0 + 64 * wave + rho) * rowb;
        pb0 = xsb + (int64_t)q0 * rowb;
        pb1 = xsb + (int64_t)q1 * rowb;
    }
    int ipar = 0;
    load_norms(is0, in0, 0);
    if (wn < nitems) {
        int s1, n1;
        tile_of(wn, s1, n1);
        load_meta(s1, 1);
    }
    int ci = 0;
    bool more = true;
    int64_t issued = 0;
    auto issue_one = [&]() __attribute__((always_inline)) {
        if (ci == nch) {   // the issue cursor enters the next item (its survivor rows landed long ago)
            ci = 0;
            wi = wn;
            ipar ^= 1;
            tile_of(wi, is0, in0);
            const int* mrow = meta + ipar * 256 + wave * 64;
            const int q0 = mrow[rho], q1 = mrow[16 + rho];
            pa = csb + (int64_t)(in0 + 64 * wave + rho) * rowb;
            pb0 = xsb + (int64_t)q0 * rowb;
            pb1 = xsb + (int64_t)q1 * rowb;
            load_norms(is0, in0, ipar);
            wn = next_valid(wn + G);
            if (wn < nitems) {
                int s1, n1;
                tile_of(wn, s1, n1);
                load_meta(s1, ipar ^ 1);
            }
        }
        unsigned char* base = smem + (int)(issued % kLgStages) * kLgStageBytes;
        const int64_t o = (int64_t)ci * 64;
#pragma unroll
        for (int t = 0; t < 4; ++t)
            __builtin_amdgcn_global_load_lds(pa + 16 * t * rowb + o, (lds_ptr)(base + (4 * wave + t) * 1024), 16, 0, 0);
        __builtin_amdgcn_global_load_lds(pb0 + o, (lds_ptr)(base + kLgN * 64 + 2 * wave * 1024), 16, 0, 0);
        __builtin_amdgcn_global_load_lds(pb1 + o, (lds_ptr)(base + kLgN * 64 + (2 * wave + 1) * 1024), 16, 0, 0);
        ++issued;
        if (++ci == nch && wn >= nitems) more = false;
    };
    // Compute cursor: item wcur (tile cs0, cn0), chunk cc, parity par.
    int64_t wcur = wi;
    int cs0 = is0, cn0 = in0, cc = 0, par = 0;
    const int ahead = min(kLgStages - 1, nch);
    for (int e = 0; e < ahead && more; ++e) issue_one();

    f32x16 acc[4][2];
#pragma unroll
    for (int a = 0; a < 4; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int e = 0; e < 16; ++e) acc[a][b][e] = 0.f;
    for (int64_t g = 0; g < issued; ++g) {
        // Chunk g has landed once at most the chunks issued after it (six
        // loads each per wave) are outstanding (with it every older load:
        // the item's norms and the next item's survivor rows); the barrier
        // then makes every wave's part visible and frees the stage of chunk
        // g - 1 for the load issued next.
        if (issued - 1 - g >= 1)
            asm volatile("s_waitcnt vmcnt(6) lgkmcnt(0)\n\ts_barrier" ::: "memory");
        else
            asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)\n\ts_barrier" ::: "memory");
        if (more) issue_one();
        const unsigned char* S = smem + (int)(g % kLgStages) * kLgStageBytes;
        bf16x8 ah[4], al[4], bh[2], bl[2];
#pragma unroll
        for (int a = 0; a < 4; ++a) {
            ah[a] = *reinterpret_cast<const bf16x8*>(S + ga + 2048 * a + offh);
            al[a] = *reinterpret_cast<const bf16x8*>(S + ga + 2048 * a + offl);
        }
#pragma unroll
        for (int b = 0; b < 2; ++b) {
            bh[b] = *reinterpret_cast<const bf16x8*>(S + gb + 2048 * b + offh);
            bl[b] = *reinterpret_cast<const bf16x8*>(S + gb + 2048 * b + offl);
        }
#pragma unroll
        for (int a = 0; a < 4; ++a)
#pragma unroll
            for (int b = 0; b < 2; ++b)
                acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah[a], bh[b], acc[a][b], 0, 0, 0);
#pragma unroll
        for (int a = 0; a < 4; ++a)
#pragma unroll
            for (int b = 0; b < 2; ++b)
                acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ah[a], bl[b], acc[a][b], 0, 0, 0);
#pragma unroll
        for (int a = 0; a < 4; ++a)
#pragma unroll
            for (int b = 0; b < 2; ++b)
                acc[a][b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(al[a], bh[b], acc[a][b], 0, 0, 0);
        if (++cc < nch) continue;

        // Item done.  Register e of accumulator [a][cb]: centroid cn0 + 128 wr
        // + 32 a + 8 (e / 4) + 4 half + e % 4, survivor column 64 wc + 32 cb +
        // col; its place in the lane's list: 16 a + 4 (e / 4) + e % 4.
        const float* nr = nrm + par * (kLgN + kLgM);
        uint32_t KP[2][4];
#pragma unroll
        for (int cb = 0; cb < 2; ++cb) {
            uint32_t K[4] = {0xffffffffu, 0xffffffffu, 0xffffffffu, 0xffffffffu};
            const float xa = nr[kLgN + 64 * wc + 32 * cb + col];
#pragma unroll
            for (int a = 0; a < 4; ++a)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const f32x4 cn = *reinterpret_cast<const f32x4*>(nr + 128 * wr + 32 * a + 8 * q + 4 * half);
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const float v = fmaxf(fmaf(-2.f, acc[a][cb][4 * q + e], xa + cn[e]), 0.f);
                        key4_insert(K, (__float_as_uint(v) & ~63u) | (uint32_t)(16 * a + 4 * q + e));
                    }
                }
            // Place in the item: 128 wr + 32 a + 8 q + 4 half + e.  Clearing
            // two more value bits can reorder the list: sort it again.
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const uint32_t lo = K[q] & 63u;
                const uint32_t place = 128 * wr + 4 * half + (lo & 3u) + 8 * ((lo >> 2) & 3u) + 32 * (lo >> 4);
                KP[cb][q] = (K[q] & ~255u) | place;
            }
            sort4(KP[cb]);
        }
        // Half-wave h keeps column 32 h + col and merges in the other half's
        // list of it (a lane swap; no LDS store may follow the ring's loads
        // without waiting for them).
        uint32_t mine[4], other[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            mine[q] = half ? KP[1][q] : KP[0][q];
            other[q] = __shfl_xor(half ? KP[0][q] : KP[1][q], 32);
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) key4_insert(mine, other[q]);
        const int rows = min(kLgM, ns - cs0);
        const int sc = 64 * wc + 32 * half + col;
        if (sc < rows) {
            uint32_t o[8];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                o[2 * q] = mine[q] & ~255u;
                o[2 * q + 1] = (uint32_t)cn0 + (mine[q] & 255u);
            }
            uint4* dst = reinterpret_cast<uint4*>(Lg.cand + (((int64_t)(cs0 + sc) * nct + cn0 / kLgN) * 2 + wr) * 4);
            dst[0] = make_uint4(o[0], o[1], o[2], o[3]);
            dst[1] = make_uint4(o[4], o[5], o[6], o[7]);
        }
        // Next item of the compute cursor.
        cc = 0;
        par ^= 1;
        wcur = next_valid(wcur + G);
        if (wcur < nitems) tile_of(wcur, cs0, cn0);
#pragma unroll
        for (int a = 0; a < 4; ++a)
#pragma unroll
            for (int b = 0; b < 2; ++b)
#pragma unroll
                for (int e = 0; e < 16; ++e) acc[a][b][e] = 0.f;
    }
}

// ---------------------------------------------------------------------------
// Refinement of every survivor by a thread pair (each merging half of its
// candidate lists: four per centroid tile and half of it): only centroids
// within twice the expanded form's error bound of the smallest can be the
// nearest.  A lone candidate is the assignment, its bound taken from the
// expanded value; two or three go to k_multi_large (direct form, float64
// near-tie rule); a survivor whose four smallest all lie inside the bound
// (more may lie outside the lists) goes to k_full_large, which decides it in
// float64 over all centroids.
//
// Error bound of an expanded value (x and c the float32 row and centroid):
//   - |x|^2, |c|^2, the float32 roundings: (d + 8) 2^-24 R^2 with
//     R = |x| + max |c| (the float32 model of the other paths);
//   - the split product: dropping lo.lo and the residuals of the two
//     roundings costs at most 3.04 2^-16 |x_m| |c_m| per dimension;
//   - the bf16 products are exact in float32 and each instruction adds 16
//     of them to its accumulator; assuming an error of at most 18 units of
//     2^-23 relative to |C| + sum |p| per instruction (true of sequential
//     float32 additions, rounded or truncated, and of one alignment of all
//     17 addends to the largest), the 3 ceil(d/16) instructions of a
//     product contribute at most 6.9 d' 2^-24 sum_m |x_m| |c_m|, d' = 16
//     ceil(d / 16);
//   - the packed key lowers a value by less than 2^-15 of itself (<= R^2);
//   so a value is within gexp R^2 + 2 (778 + 6.9 d') 2^-24 |x| max |c| +
//   2^-15 R^2 of the distance, plus an absolute 2^-100 (1 + R) for bf16
//   values below the normal range.  Rows with |x|^2 or R out of range
//   (non-finite data) are decided in float64 over all centroids.

__global__ __launch_bounds__(256) void k_refine_large(Dev P, Large Lg) {
    IterState* st = P.st;
    if (!st->active) return;
    const int k = P.k, d = P.d, nct = Lg.nct;
    const bool first = st->t == 0;
    const uint32_t ns = *Lg.nsurv;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    __shared__ float red[4];
    float m2 = 0.f;
    for (int j = tid; j < k; j += blockDim.x) {
        const float v = P.cn2[j];
        m2 = fmaxf(m2, v <= FLT_MAX ? v : INFINITY);   // a non-finite centroid: every row in float64
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) m2 = fmaxf(m2, __shfl_xor(m2, off));
    if (lane == 0) red[wave] = m2;
    __syncthreads();
    const float cnmax = sqrtf(fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]))) * kUp;
    const float ecm = st->ec_max;
    const float gexp = (float)(d + 8) * 0x1p-24f + 0x1p-15f;
    const float gsp2 = 2.f * (778.f + 6.9f * (float)(16 * Lg.nch)) * 0x1p-24f * (1.f + 0x1p-10f);
    uint64_t my_changed = 0, my_comp = 0, my_rc = 0;
    const int part = tid & 1;
    // Queued survivors and moves gather in LDS and go to the global lists
    // with one atomic per flush of up to 2 kRefineFlush entries (a global
    // counter per wave would take one atomic per 64 survivors).
    __shared__ int4 qb[2 * kRefineFlush], mb[2 * kRefineFlush];
    __shared__ uint32_t nqb, nmb, gq, gm;
    if (tid == 0) {
        nqb = 0;
        nmb = 0;
    }
    __syncthreads();
    auto flush = [&](bool all) __attribute__((always_inline)) {
        __syncthreads();
        const uint32_t cq = nqb, cm = nmb;
        const bool fq = cq >= (all ? 1u : (uint32_t)kRefineFlush), fm = cm >= (all ? 1u : (uint32_t)kRefineFlush);
        if (tid == 0) {
            if (fq) gq = atomicAdd(Lg.nmq, cq);
            if (fm) gm = atomicAdd(Lg.nmv, cm);
        }
        __syncthreads();
        if (fq)
            for (uint32_t e = tid; e < cq; e += blockDim.x) Lg.mq[gq + e] = qb[e];
        if (fm)
            for (uint32_t e = tid; e < cm; e += blockDim.x)
                if (gm + e < (uint32_t)Lg.mvcap) Lg.mv[gm + e] = mb[e];
        __syncthreads();
        if (tid == 0) {
            if (fq) nqb = 0;
            if (fm) nmb = 0;
        }
        __syncthreads();
    };

    const bool rec_moves = !first && !(P.flags & KM_FLAG_STATS);
    for (int64_t c0 = (int64_t)blockIdx.x * 128; c0 < (int64_t)ns; c0 += (int64_t)gridDim.x * 128) {
        const int64_t c = c0 + (tid >> 1);
        int4 mvr = make_int4(0, 0, 0, 0), mqr = make_int4(0, 0, 0, 0);
        bool moved = false, queued = false;
        if (c < (int64_t)ns) {   // both threads of a pair
        float T[4];
        int TJ[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            T[q] = INFINITY;
            TJ[q] = INT_MAX;
        }
        // The pair reads half of the 8 nct candidates each, then each merges
        // in the other's four: the same list in both (a total order).
        const uint4* cl = reinterpret_cast<const uint4*>(Lg.cand + c * nct * 8) + part * 2 * nct;
        for (int q = 0; q < 2 * nct; ++q) {
            const uint4 v = cl[q];
            top4_insert(T, TJ, __uint_as_float(v.x), (int)v.y);
            top4_insert(T, TJ, __uint_as_float(v.z), (int)v.w);
        }
        {
            float OT[4];
            int OJ[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                OT[q] = __shfl_xor(T[q], 1);
                OJ[q] = __shfl_xor(TJ[q], 1);
            }
#pragma unroll
            for (int q = 0; q < 4; ++q) top4_insert(T, TJ, OT[q], OJ[q]);
        }
        const int64_t i = Lg.surv[c];
        const int inc = first ? -1 : P.a[i];
        const float x2 = Lg.sx2[c];
        const float xn = sqrtf(fmaxf(x2, 0.f)) * kUp;
        const float R = xn + cnmax;
        const float e1 = gexp * R * R + gsp2 * xn * cnmax + 4.f * R * ecm + 2.f * ecm * ecm + 0x1p-100f * (1.f + R);
        const float thr = T[0] + 2.f * e1;
        // Only centroids whose expanded distance lies within thr of the
        // smallest can be the nearest: any other one is certified farther
        // than the smallest's centroid.
        const bool full = T[3] <= thr || !(x2 <= 0x1p120f) || !(R <= 0x1p60f);
        if (full) {
            if (part == 0) {
                Lg.fq[atomicAdd(Lg.nfull, 1u)] = (int32_t)c;
                my_comp += (uint64_t)k;
                my_rc += 1;
            }
        } else {
        int nq = 0;
        while (nq < 3 && T[nq] <= thr && TJ[nq] < k) ++nq;   // uniform in the pair
        // One candidate is the nearest centroid (every other one is certified
        // farther): as on the LDS paths, its bound then comes from its
        // expanded value and the error bound, without the direct form (kept
        // when statistics are gathered).  Otherwise the survivor and its
        // candidates go to k_multi_large.
        if (nq == 1 && !(P.flags & KM_FLAG_STATS)) {
            const int b = TJ[0];
            const float ub = __builtin_amdgcn_sqrtf(fmaxf(T[0] + e1, 0.f)) * (1.0f + 0x1p-20f) * kUp;
            if (part == 0) {
                if (b != inc) {
                    P.a[i] = b;
                    my_changed += 1;
                    moved = true;
                    mvr = make_int4((int)i, inc, b, 0);
                }
                P.u[i] = ub;
                my_comp += (uint64_t)k;
            }
        } else if (part == 0) {
            queued = true;
            mqr = make_int4((int)c, TJ[0], nq > 1 ? TJ[1] : -1, nq > 2 ? TJ[2] : -1);
            my_comp += (uint64_t)k;
        }
        }   // not full
        }   // c < ns
        // At most 128 entries per round, so a buffer of 2 kRefineFlush holds
        // a round on top of fewer than kRefineFlush waiting entries.
        if (queued) qb[atomicAdd(&nqb, 1u)] = mqr;
        if (moved && rec_moves) mb[atomicAdd(&nmb, 1u)] = mvr;
        flush(false);
    }
    flush(true);
    {
        const int base = k * d + k;
        const int slot[3] = {base + kStChanged, base + kStComputed, base + kStRecheck};
        uint64_t v[3] = {my_changed, my_comp, my_rc};
        add_stats_block<3>(P.total, slot, v);
    }
}

// ---------------------------------------------------------------------------
// Survivors with two or three candidates inside the bound, one wave each:
// the candidates' direct-form float32 distances (lanes over the dimensions,
// coalesced rows, a fixed butterfly: the float32 error bound holds for any
// summation order), the nearest with the incumbent winning ties, and when
// the two smallest lie within the float32 band the float64 decision with
// the oracle's rule (smaller distance, then the incumbent, then the lower
// index).  With statistics every survivor comes here (direct-form bounds).

__global__ __launch_bounds__(256) void k_multi_large(Dev P, Large Lg) {
    IterState* st = P.st;
    if (!st->active) return;
    const int k = P.k, d = P.d, lane = threadIdx.x & 63;
    const bool first = st->t == 0;
    const bool rec_moves = !first && !(P.flags & KM_FLAG_STATS);
    const float gamma = P.gamma, ecm = st->ec_max;
    const uint32_t nq_all = *Lg.nmq;
    const bool vec = (d & 3) == 0;
    uint64_t my_changed = 0, my_rc = 0;
    for (uint32_t q = blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6); q < nq_all;
         q += gridDim.x * (blockDim.x >> 6)) {
        const int4 e = Lg.mq[q];
        const int js[3] = {e.y, e.z, e.w};
        const int nq = e.w >= 0 ? 3 : (e.z >= 0 ? 2 : 1);
        const int64_t i = Lg.surv[e.x];
        const float* xr = P.X + i * d;
        const int inc = first ? -1 : P.a[i];
        auto dist32 = [&](int j) __attribute__((always_inline)) {
            const float* cr = P.C32 + (int64_t)j * d;
            float acc = 0.f;
            if (vec) {
                for (int m = 4 * lane; m < d; m += 256) {
                    const f32x4 xv = *reinterpret_cast<const f32x4*>(xr + m);
                    const f32x4 cv = *reinterpret_cast<const f32x4*>(cr + m);
                    const float t0 = xv.x - cv.x, t1 = xv.y - cv.y, t2 = xv.z - cv.z, t3 = xv.w - cv.w;
                    acc = fmaf(t0, t0, acc);
                    acc = fmaf(t1, t1, acc);
                    acc = fmaf(t2, t2, acc);
                    acc = fmaf(t3, t3, acc);
                }
            } else {
                for (int m = lane; m < d; m += 64) {
                    const float t = xr[m] - cr[m];
                    acc = fmaf(t, t, acc);
                }
            }
#pragma unroll
            for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
            return acc;
        };
        auto dist64 = [&](int j) __attribute__((always_inline)) {
            const double* cr = P.C64 + (int64_t)j * d;
            double acc = 0.0;
            for (int m = lane; m < d; m += 64) {
                const double t = (double)xr[m] - cr[m];
                acc = fma(t, t, acc);
            }
#pragma unroll
            for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
            return acc;
        };
        float d1 = INFINITY, d2 = INFINITY;
        int rk1 = INT_MAX, j1 = 0;
        for (int t = 0; t < nq; ++t) {
            const int j = js[t];
            const float Dd = dist32(j);
            const int rk = j == inc ? -1 : j;
            if (Dd < d1 || (Dd == d1 && rk < rk1)) {
                d2 = d1;
                d1 = Dd;
                rk1 = rk;
                j1 = j;
            } else if (Dd < d2) {
                d2 = Dd;
            }
        }
        bool re = false;
        if (d2 != INFINITY) {
            const float band = 2.f * gamma * (d1 + d2) + 4.f * (sqrtf(d1) + sqrtf(d2)) * ecm + 8.f * ecm * ecm;
            re = d2 - d1 <= band;
        }
        int b = j1;
        float ub = upper_bound(d1, P.ec[j1], gamma);
        if (re) {
            double Dbb = INFINITY;
            int bb = -1, kb = INT_MAX;
            for (int t = 0; t < nq; ++t) {
                const int j = js[t];
                const double Dj = dist64(j);
                const int rk = j == inc ? -1 : j;
                if (Dj < Dbb || (Dj == Dbb && rk < kb)) {
                    Dbb = Dj;
                    bb = j;
                    kb = rk;
                }
            }
            b = bb < 0 ? 0 : bb;
            ub = f32_up(sqrt(Dbb) * (1.0 + 0x1p-40));
        }
        if (lane == 0) {
            if (b != inc) {
                P.a[i] = b;
                my_changed += 1;
                if (rec_moves) {
                    const uint32_t qm = atomicAdd(Lg.nmv, 1u);
                    if (qm < (uint32_t)Lg.mvcap) Lg.mv[qm] = make_int4((int)i, inc, b, 0);
                }
            }
            P.u[i] = ub;
            my_rc += re ? 1 : 0;
        }
    }
    {
        const int base = k * d + k;
        const int slot[2] = {base + kStChanged, base + kStRecheck};
        uint64_t v[2] = {my_changed, my_rc};
        add_stats_block<2>(P.total, slot, v);
    }
}

// ---------------------------------------------------------------------------
// Float64 decision over all centroids for the queued survivors.  The first
// kFullCap of them are split over kFullSplit blocks, each taking a range of
// centroids (the row in LDS as float64, one centroid per thread, its
// distance summed over the dimensions in order) and writing its best under
// the oracle's rule (smaller distance, then the incumbent, then the lower
// index); the block that finishes a survivor last (a counter per survivor
// behind a fence) combines the ranges and writes the decision.  Survivors
// past kFullCap take one block over all centroids.

__global__ __launch_bounds__(256) void k_full_large(Dev P, Large Lg) {
    IterState* st = P.st;
    if (!st->active) return;
    const int k = P.k, d = P.d;
    const bool first = st->t == 0;
    const bool rec_moves = !first && !(P.flags & KM_FLAG_STATS);
    const uint32_t nf = *Lg.nfull;
    const uint32_t nsplit = min(nf, (uint32_t)kFullCap);
    const int kr = (k + kFullSplit - 1) / kFullSplit;
    extern __shared__ __align__(16) unsigned char smem[];
    double* xd = reinterpret_cast<double*>(smem);   // [d]
    __shared__ double rD[256];
    __shared__ int rJ[256], rK[256];
    __shared__ uint32_t last;
    const int tid = threadIdx.x;
    uint64_t my_changed = 0;
    auto decide = [&](int64_t i, int inc, double D, int bj) __attribute__((always_inline)) {
        const int b = bj < 0 ? 0 : bj;
        if (b != inc) {
            P.a[i] = b;
            my_changed += 1;
            if (rec_moves) {
                const uint32_t qm = atomicAdd(Lg.nmv, 1u);
                if (qm < (uint32_t)Lg.mvcap) Lg.mv[qm] = make_int4((int)i, inc, b, 0);
            }
        }
        P.u[i] = f32_up(sqrt(D) * (1.0 + 0x1p-40));
    };
    const uint32_t items = nsplit * kFullSplit + (nf - nsplit);
    for (uint32_t it = blockIdx.x; it < items; it += gridDim.x) {
        const bool split = it < nsplit * kFullSplit;
        const uint32_t q = split ? it / kFullSplit : nsplit + (it - nsplit * kFullSplit);
        const int part = split ? (int)(it % kFullSplit) : 0;
        const int j0 = split ? part * kr : 0, j1 = split ? min(k, j0 + kr) : k;
        const int64_t i = Lg.surv[Lg.fq[q]];
        __syncthreads();   // the previous item's row and reduction are consumed
        for (int m = tid; m < d; m += blockDim.x) xd[m] = (double)P.X[i * d + m];
        __syncthreads();
        const int inc = first ? -1 : P.a[i];
        double Db = INFINITY;
        int bb = -1, kb = INT_MAX;
        for (int j = j0 + tid; j < j1; j += blockDim.x) {
            const double* cr = P.C64 + (int64_t)j * d;
            double acc = 0.0;
            for (int m = 0; m < d; ++m) {
                const double t = xd[m] - cr[m];
                acc = fma(t, t, acc);
            }
            const int rk = j == inc ? -1 : j;
            if (acc < Db || (acc == Db && rk < kb)) {
                Db = acc;
                bb = j;
                kb = rk;
            }
        }
        rD[tid] = Db;
        rJ[tid] = bb;
        rK[tid] = kb;
        __syncthreads();
        for (int w = 128; w > 0; w >>= 1) {
            if (tid < w) {
                const double D2 = rD[tid + w];
                const int k2 = rK[tid + w];
                if (D2 < rD[tid] || (D2 == rD[tid] && k2 < rK[tid])) {
                    rD[tid] = D2;
                    rJ[tid] = rJ[tid + w];
                    rK[tid] = k2;
                }
            }
            __syncthreads();
        }
        if (!split) {
            if (tid == 0) decide(i, inc, rD[0], rJ[0]);
            continue;
        }
        if (tid == 0) {
            FullPart* fp = Lg.fpart + (int64_t)q * kFullSplit;
            fp[part] = FullPart{rD[0], rJ[0], rK[0]};
            __threadfence();
            last = atomicAdd(&Lg.fcnt[q], 1u);
        }
        __syncthreads();
        if (tid == 0 && last == kFullSplit - 1) {   // every range is in: combine
            __threadfence();
            const volatile FullPart* fp = Lg.fpart + (int64_t)q * kFullSplit;
            double D = INFINITY;
            int bj = -1, bk = INT_MAX;
            for (int r = 0; r < kFullSplit; ++r) {
                const double D2 = fp[r].D;
                const int k2 = fp[r].rk;
                if (D2 < D || (D2 == D && k2 < bk)) {
                    D = D2;
                    bj = fp[r].j;
                    bk = k2;
                }
            }
            Lg.fcnt[q] = 0;   // ready for the next step
            decide(i, inc, D, bj);
        }
    }
    if (threadIdx.x == 0 && my_changed) {
        unsigned long long* sc = reinterpret_cast<unsigned long long*>(P.total + (int64_t)k * d + k);
        atomicAdd(&sc[kStChanged], (unsigned long long)my_changed);
    }
}

// ---------------------------------------------------------------------------
// Counting sort of the points by their new cluster.

__global__ __launch_bounds__(256) void k_hist_large(Dev P, Large Lg) {
    if (!P.st->active || large_incremental(P, Lg)) return;
    extern __shared__ __align__(16) unsigned char smem[];
    uint32_t* h = reinterpret_cast<uint32_t*>(smem);
    const int k = P.k;
    for (int j = threadIdx.x; j < k; j += blockDim.x) h[j] = 0;
    __syncthreads();
    const int64_t lo = (int64_t)blockIdx.x * Lg.span;
    const int64_t hi = min(P.n, lo + Lg.span);
    for (int64_t i = lo + threadIdx.x; i < hi; i += blockDim.x) atomicAdd(&h[P.a[i]], 1u);
    __syncthreads();
    for (int j = threadIdx.x; j < k; j += blockDim.x) Lg.cnt[(int64_t)blockIdx.x * k + j] = h[j];
}

// Per cluster j: exclusive prefix of the block counts (write offsets
// relative to the cluster start) and the cluster size into base[j].
__global__ __launch_bounds__(256) void k_scan_large_cols(Dev P, Large Lg) {
    if (!P.st->active || large_incremental(P, Lg)) return;
    const int j = blockIdx.x * blockDim.x + threadIdx.x;
    if (j >= P.k) return;
    uint32_t run = 0;
    for (int g = 0; g < Lg.Gs; ++g) {
        const int64_t o = (int64_t)g * P.k + j;
        const uint32_t c = Lg.cnt[o];
        Lg.off[o] = run;
        run += c;
    }
    Lg.base[j] = run;
}

// One block: cluster starts (exclusive scan of the sizes) and the first
// segment chunk of every cluster.  base[k] = n, cbase[k] = chunk count.
__global__ __launch_bounds__(1024) void k_scan_large_clusters(Dev P, Large Lg) {
    if (!P.st->active || large_incremental(P, Lg)) return;
    const int k = P.k, t = threadIdx.x, T = blockDim.x;
    __shared__ uint32_t ps[1024], pc[1024];
    const int per = (k + T - 1) / T, j0 = t * per, j1 = min(k, j0 + per);
    uint32_t s = 0, sc = 0;
    for (int j = j0; j < j1; ++j) {
        const uint32_t sz = Lg.base[j];
        s += sz;
        sc += (sz + kLgChunkRows - 1) / kLgChunkRows;
    }
    ps[t] = s;
    pc[t] = sc;
    __syncthreads();
    for (int w = 1; w < T; w <<= 1) {   // inclusive Hillis-Steele scan
        const uint32_t a = t >= w ? ps[t - w] : 0, b = t >= w ? pc[t - w] : 0;
        __syncthreads();
        ps[t] += a;
        pc[t] += b;
        __syncthreads();
    }
    uint32_t run = ps[t] - s, crun = pc[t] - sc;
    for (int j = j0; j < j1; ++j) {
        const uint32_t sz = Lg.base[j];
        Lg.base[j] = run;
        Lg.cbase[j] = crun;
        run += sz;
        crun += (sz + kLgChunkRows - 1) / kLgChunkRows;
    }
    if (t == T - 1) {
        Lg.base[k] = ps[T - 1];
        Lg.cbase[k] = pc[T - 1];
    }
}

__global__ __launch_bounds__(256) void k_scatter_large(Dev P, Large Lg) {
    if (!P.st->active || large_incremental(P, Lg)) return;
    extern __shared__ __align__(16) unsigned char smem[];
    uint32_t* pos = reinterpret_cast<uint32_t*>(smem);
    const int k = P.k;
    for (int j = threadIdx.x; j < k; j += blockDim.x)
        pos[j] = Lg.base[j] + Lg.off[(int64_t)blockIdx.x * k + j];
    __syncthreads();
    const int64_t lo = (int64_t)blockIdx.x * Lg.span;
    const int64_t hi = min(P.n, lo + Lg.span);
    for (int64_t i = lo + threadIdx.x; i < hi; i += blockDim.x)
        Lg.perm[atomicAdd(&pos[P.a[i]], 1u)] = (int32_t)i;
}

// One block per chunk of <= kLgChunkRows points of one cluster: exact
// fixed-point coordinate sums (and, with KM_FLAG_STATS, the squared
// distances to the cluster's current centroid, element by element).
__global__ __launch_bounds__(256) void k_segsum_large(Dev P_, Large Lg) {
    const Dev P = with_scales(P_);
    if (!P.st->active || large_incremental(P, Lg)) return;
    const int c = blockIdx.x;
    const int k = P.k, d = P.d;
    if (c >= (int)Lg.cbase[k]) return;
    int lo = 0, hi = k;   // cluster j with cbase[j] <= c < cbase[j + 1]
    while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if ((int)Lg.cbase[mid] <= c) lo = mid;
        else hi = mid;
    }
    const int j = lo;
    const uint32_t r0 = Lg.base[j] + (uint32_t)(c - (int)Lg.cbase[j]) * kLgChunkRows;
    const uint32_t r1 = min(Lg.base[j + 1], r0 + kLgChunkRows);
    const bool want_inertia = (P.flags & KM_FLAG_STATS) != 0;
    uint64_t iq = 0;
    for (int m = threadIdx.x; m < d; m += blockDim.x) {
        const float cj = P.C32[(int64_t)j * d + m];
        uint64_t acc = 0;
        for (uint32_t r = r0; r < r1; ++r) {
            const float x = P.X[(int64_t)Lg.perm[r] * d + m];
            acc += fixed_bits((double)x, P.qscale);
            if (want_inertia) {
                const float t = x - cj;
                iq += fixed_bits((double)(t * t), P.iscale) - kMagicBits;
            }
        }
        Lg.cpart[(int64_t)c * d + m] = acc;
    }
    if (want_inertia) {
        __shared__ uint64_t rs[4];
        iq = wave_sum_u64(iq);
        if ((threadIdx.x & 63) == 0) rs[threadIdx.x >> 6] = iq;
        __syncthreads();
        if (threadIdx.x == 0) Lg.ciq[c] = rs[0] + rs[1] + rs[2] + rs[3];
    }
}

// Per-cluster sums (over the cluster's chunks) and counts into the reduced
// row, less the running sums that k_update adds back; block 0 also adds the
// inertia partials.
__global__ __launch_bounds__(256) void k_chunk_reduce_large(Dev P, Large Lg) {
    if (!P.st->active || large_incremental(P, Lg)) return;
    const int k = P.k, d = P.d;
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (e < (int64_t)k * d) {
        const int j = (int)(e / d), m = (int)(e - (int64_t)j * d);
        uint64_t acc = 0;
        for (uint32_t cc = Lg.cbase[j]; cc < Lg.cbase[j + 1]; ++cc) acc += Lg.cpart[(int64_t)cc * d + m];
        P.total[e] = acc - P.sums[e];
        if (m == 0) {
            const int64_t o = (int64_t)k * d + j;
            P.total[o] = (uint64_t)(Lg.base[j + 1] - Lg.base[j]) - P.sums[o];
        }
    }
    if (blockIdx.x == 0 && (P.flags & KM_FLAG_STATS)) {
        __shared__ uint64_t rs[4];
        uint64_t s = 0;
        const uint32_t nc = Lg.cbase[k];
        for (uint32_t cc = threadIdx.x; cc < nc; cc += blockDim.x) s += Lg.ciq[cc];
        s = wave_sum_u64(s);
        if ((threadIdx.x & 63) == 0) rs[threadIdx.x >> 6] = s;
        __syncthreads();
        if (threadIdx.x == 0) P.total[(int64_t)k * d + k + kStInertia] = rs[0] + rs[1] + rs[2] + rs[3];
    }
}

// Incremental sums: every move takes its row's exact fixed-point image out
// of the old cluster's sum and into the new one's (wrap-around integers, so
// the result equals the full sum bit for bit); one wave per move.
__global__ __launch_bounds__(256) void k_moves_large(Dev P_, Large Lg) {
    const Dev P = with_scales(P_);
    if (!P.st->active || !large_incremental(P, Lg)) return;
    const int k = P.k, d = P.d, lane = threadIdx.x & 63;
    const uint32_t nm = *Lg.nmv;
    unsigned long long* T = reinterpret_cast<unsigned long long*>(P.total);
    for (uint32_t q = blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6); q < nm;
         q += gridDim.x * (blockDim.x >> 6)) {
        const int4 mv = Lg.mv[q];
        const float* xr = P.X + (int64_t)mv.x * d;
        for (int m = lane; m < d; m += 64) {
            const uint64_t img = fixed_bits((double)xr[m], P.qscale);
            atomicAdd(&T[(int64_t)mv.y * d + m], (unsigned long long)(0ull - img));
            atomicAdd(&T[(int64_t)mv.z * d + m], (unsigned long long)img);
        }
        if (lane == 0) {
            atomicAdd(&T[(int64_t)k * d + mv.y], ~0ull);
            atomicAdd(&T[(int64_t)k * d + mv.z], 1ull);
        }
    }
}

// ---------------------------------------------------------------------------
// Centroid table for large k*d: a block stages kTiTile float64 rows in LDS
// and streams every centroid once against them.

__global__ __launch_bounds__(256) void k_centroid_table_tiled(Dev P, Large Lg, int force) {
    if (!force && !P.st->active) return;
    if (blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0) {   // the next step's lists start empty
        *Lg.nsurv = 0;
        *Lg.nfull = 0;
        *Lg.nmq = 0;
        *Lg.nmv = 0;
    }
    const int k = P.k, d = P.d;
    const int i0 = blockIdx.x * kTiTile, ni = min(kTiTile, k - i0);
    // Block column y takes centroids j in [y k / kTiSplit, (y + 1) k / kTiSplit).
    const int j0 = (int)((int64_t)blockIdx.y * k / kTiSplit), j1 = (int)((int64_t)(blockIdx.y + 1) * k / kTiSplit);
    extern __shared__ __align__(16) unsigned char smem[];
    double* ci = reinterpret_cast<double*>(smem);                  // [kTiTile][d]
    float* mins = reinterpret_cast<float*>(ci + kTiTile * d);      // [kTiTile][256]
    for (int e = threadIdx.x; e < kTiTile * d; e += blockDim.x) {
        const int r = e / d;
        ci[e] = r < ni ? P.C64[(int64_t)(i0 + r) * d + (e - r * d)] : 0.0;
    }
    __syncthreads();
    float mn[kTiTile];
#pragma unroll
    for (int r = 0; r < kTiTile; ++r) mn[r] = INFINITY;
    for (int j = j0 + threadIdx.x; j < j1; j += blockDim.x) {
        const double* cj = P.C64 + (int64_t)j * d;
        double acc[kTiTile];
#pragma unroll
        for (int r = 0; r < kTiTile; ++r) acc[r] = 0.0;
        for (int m = 0; m < d; ++m) {
            const double v = cj[m];
#pragma unroll
            for (int r = 0; r < kTiTile; ++r) {
                const double t = ci[r * d + m] - v;
                acc[r] = fma(t, t, acc[r]);
            }
        }
#pragma unroll
        for (int r = 0; r < kTiTile; ++r) {
            if (r >= ni) continue;
            const int i = i0 + r;
            float hv = 0.f;
            if (j != i) {
                hv = f32_down(0.5 * sqrt(acc[r]) * (1.0 - 0x1p-40));
                mn[r] = fminf(mn[r], hv);
            }
            P.h[(int64_t)i * k + j] = hv;
        }
    }
#pragma unroll
    for (int r = 0; r < kTiTile; ++r) mins[r * 256 + threadIdx.x] = mn[r];
    __syncthreads();
    if (threadIdx.x < ni) {   // this column's minimum; k_split_rows forms s from the columns
        const int r = threadIdx.x, i = i0 + r;
        float m = INFINITY;
        for (int q = 0; q < (int)blockDim.x; ++q) m = fminf(m, mins[r * 256 + q]);
        Lg.smin[(int64_t)blockIdx.y * k + i] = m;
        if (blockIdx.y == 0) {
            const float* c32 = P.C32 + (int64_t)i * d;
            double n2 = 0.0;
            for (int q = 0; q < d; ++q) n2 = fma((double)c32[q], (double)c32[q], n2);
            P.cn2[i] = (float)n2;
        }
    }
    if (blockIdx.x == 0 && blockIdx.y == 0) {
        float em = 0.f;
        for (int j = threadIdx.x; j < k; j += blockDim.x) em = fmaxf(em, P.ec[j]);
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) em = fmaxf(em, __shfl_xor(em, off));
        __syncthreads();
        if ((threadIdx.x & 63) == 0) mins[threadIdx.x >> 6] = em;
        __syncthreads();
        if (threadIdx.x == 0)
            P.st->ec_max = fmaxf(fmaxf(mins[0], mins[1]), fmaxf(mins[2], mins[3]));
    }
}

// ---------------------------------------------------------------------------
// Launchers

const void* large_mfma_symbol() { return reinterpret_cast<const void*>(&k_mfma_large); }

// Assignment group: Clause 1 and the matrix-core candidates.  The candidates'
// refinement opens the reduction group (its timing slot).
hipError_t launch_large_assign(const Dev& dv, const Large& lg, int gb, hipStream_t s) {
    hipLaunchKernelGGL(k_bound_large, dim3(gb), dim3(kLgBoundThreads), 0, s, dv, lg);
    hipLaunchKernelGGL(k_mfma_large, dim3(lg.Gm), dim3(256), large_mfma_lds(), s, dv, lg);
    return hipGetLastError();
}

hipError_t launch_large_split_x(const Dev& dv, const Large& lg, int cus, hipStream_t s) {
    int64_t g = (dv.n + 3) / 4;
    if (g > (int64_t)cus * 16) g = (int64_t)cus * 16;
    hipLaunchKernelGGL(k_split_rows, dim3((unsigned)g), dim3(256), 0, s, dv.X, dv.n, dv.n, dv.d, lg.nch, lg.xs,
                       lg.x2, static_cast<const IterState*>(nullptr), 1, static_cast<const float*>(nullptr),
                       static_cast<float*>(nullptr));
    return hipGetLastError();
}

hipError_t launch_large_reduce(const Dev& dv, const Large& lg, hipStream_t s) {
    hipLaunchKernelGGL(k_refine_large, dim3(lg.Gr), dim3(256), 0, s, dv, lg);
    hipLaunchKernelGGL(k_multi_large, dim3(lg.Gr), dim3(256), 0, s, dv, lg);
    hipLaunchKernelGGL(k_full_large, dim3(lg.Gr), dim3(256), 8 * dv.d, s, dv, lg);
    const int hl = 4 * dv.k;
    hipLaunchKernelGGL(k_hist_large, dim3(lg.Gs), dim3(256), hl, s, dv, lg);
    hipLaunchKernelGGL(k_scan_large_cols, dim3((dv.k + 255) / 256), dim3(256), 0, s, dv, lg);
    hipLaunchKernelGGL(k_scan_large_clusters, dim3(1), dim3(1024), 0, s, dv, lg);
    hipLaunchKernelGGL(k_scatter_large, dim3(lg.Gs), dim3(256), hl, s, dv, lg);
    hipLaunchKernelGGL(k_segsum_large, dim3(lg.NCmax), dim3(256), 0, s, dv, lg);
    const int64_t kd = (int64_t)dv.k * dv.d;
    hipLaunchKernelGGL(k_chunk_reduce_large, dim3((unsigned)((kd + 255) / 256)), dim3(256), 0, s, dv, lg);
    hipLaunchKernelGGL(k_moves_large, dim3(lg.Gr), dim3(256), 0, s, dv, lg);
    return hipGetLastError();
}

int large_table_lds(int d) { return 8 * kTiTile * d + 4 * kTiTile * 256; }

hipError_t large_set_attributes(int k, int d) {
    hipError_t e;
    const auto attr = hipFuncAttributeMaxDynamicSharedMemorySize;
    if ((e = hipFuncSetAttribute(large_mfma_symbol(), attr, large_mfma_lds())) != hipSuccess) return e;
    if ((e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_full_large), attr, 8 * d)) != hipSuccess)
        return e;
    if ((e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_hist_large), attr, 4 * k)) != hipSuccess)
        return e;
    if ((e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_scatter_large), attr, 4 * k)) != hipSuccess)
        return e;
    return hipFuncSetAttribute(reinterpret_cast<const void*>(&k_centroid_table_tiled), attr,
                               large_table_lds(d));
}

hipError_t launch_large_table(const Dev& dv, const Large& lg, int force, hipStream_t s) {
    hipLaunchKernelGGL(k_centroid_table_tiled, dim3((dv.k + kTiTile - 1) / kTiTile, kTiSplit), dim3(256),
                       large_table_lds(dv.d), s, dv, lg, force);
    const int64_t kp = (int64_t)lg.nct * kLgN;   // padded to whole centroid tiles
    hipLaunchKernelGGL(k_split_rows, dim3((unsigned)((kp + 3) / 4)), dim3(256), 0, s, static_cast<const float*>(dv.C32),
                       kp, (int64_t)dv.k, dv.d, lg.nch, lg.cs, lg.cn2p, static_cast<const IterState*>(dv.st), force,
                       static_cast<const float*>(lg.smin), dv.s);
    return hipGetLastError();
}

}  // namespace km
