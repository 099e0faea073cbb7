// Incremental MTI step on the matrix cores, d = 16 or 32 and k <= 128: the
// paper's skipping of the data of the points Clause 1 keeps (section III-C:
// no row of such a point is read) on the path where the survivors'
// distances are a dense product X . C^T.
//
// Point state.  One 32-bit word per point: the cluster in bits 6..0 and, in
// the rest, a float32 value v (rounded up to 128 units in the last place)
// with v + D_a an upper bound on the point's distance to its centroid, D_a
// the cumulative drift of the cluster (the bound of section III-C,
// u^t = u^{t0} + f^{t0+1} + ... + f^t, kept relative to D so that a point
// that keeps its bound is never written).
//
// Per block: every wave takes tiles of kIMTile points from a block counter
// (work stealing within the block) and for each point
//   1. applies Clause 1 to its state (v <= thr(a), thr(a) the largest float
//      with thr + D_a <= s(a));
//   2. queues a survivor by the 32-centroid blocks it needs (k <= 64: its
//      own block and every block Clause 2 does not skip for it, one queue
//      per set) or by the block of its cluster (k > 64);
// and whenever a queue holds kIMBatch survivors, gathers their rows
// (16-byte loads, requested one batch ahead of their use), stages them in its
// own LDS rows and settles them:
//   - a 32-centroid block is skipped when Clause 2 holds for the whole batch:
//     every survivor's bound is at most half the distance from its
//     incumbent to each centroid of the block (the incumbent's own block is
//     never skipped, its half-distance to itself being zero);
//   - the other blocks' distances come from matrix-core tiles in the
//     expanded form |x|^2 - 2 (x.c - |c|^2 / 2), x.c as three bf16 products
//     of split operands (hi = bf16(v), lo = bf16(v - hi): hi.hi + hi.lo +
//     lo.hi, v_mfma_f32_32x32x16_bf16); every centroid within twice the
//     expanded form's error bound (the split and accumulation terms
//     included) of the smallest is a candidate, a single
//     candidate is the nearest centroid (its bound from the expanded value
//     plus the error bound), several are decided in the direct form and a
//     near tie again in float64 against the master centroids;
//   - a point whose cluster changed moves its row between the block's
//     fixed-point sums (exact integers: added to the new cluster, subtracted
//     from the old one).
// The first step has no bounds: every point is a survivor, every block is
// evaluated and every row is added to its cluster.  The block's sums of the
// moves go to its partial row; the reduction adds them and the update adds
// the total to the running sums (Dev::sums), which are therefore the exact
// sums a full read forms.
#include <float.h>
#include <limits.h>
#include <math.h>

#include "kmeans_mti.h"
#include "km_device.h"
#include "km_internal.h"

namespace km {

extern __shared__ __align__(16) unsigned char km_smem[];

namespace {

constexpr int kW = kIMWaves;
constexpr int kB = kIMBatch;
constexpr int kQ = kIMQcap;

// State word: v rounded up to a multiple of 128 units in the last place (for
// v >= 0 the bit pattern grows, for v < 0 the magnitude shrinks), the cluster
// in the cleared bits.
__device__ __forceinline__ uint32_t pack7(float v, int a) {
    uint32_t b = __float_as_uint(v);
    if (!(b >> 31)) b += 127u;
    return (b & ~127u) | (uint32_t)a;
}
__device__ __forceinline__ int st_cluster(uint32_t w) { return (int)(w & 127u); }
__device__ __forceinline__ float st_value(uint32_t w) { return __uint_as_float(w & ~127u); }

__device__ __forceinline__ float sqrt_up(float v) { return __builtin_amdgcn_sqrtf(v) * (1.0f + 0x1p-20f); }

template <int D, int KB>
__global__ __launch_bounds__(kW * 64) __attribute__((amdgpu_waves_per_eu(2))) void k_inc_mm(Dev P_, int first) {
    const Dev P = with_scales(P_);
    IterState* st = P.st;
    if (st->done) {
        if (blockIdx.x == 0 && threadIdx.x == 0) st->active = 0;
        return;
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) st->active = 1;
    constexpr int kHalf = D / 2;              // dimensions of a lane's half of a row
    constexpr int NS = D / 16;                // 16-dimension matrix-core k-steps
    constexpr int XS = D + 4;                // staged row stride (floats): D values, then point and state
    constexpr int CPR = D / 4;               // 16-byte chunks per row
    constexpr int RPL = 64 / CPR;            // rows per wave-wide load
    constexpr int kLoads = kB / RPL;         // loads per lane per batch
    constexpr bool WIDE = KB == 4;           // centroid operands in LDS
    constexpr int KP = 32 * KB;

    const int k = P.k, tid = threadIdx.x, lane = tid & 63;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int col = lane & 31, half = lane >> 5;
    const bool prune = !(P.flags & KM_FLAG_NO_PRUNE) && !first;
    const float ecmax = st->ec_max, gamma = P.gamma;
    const IncMMLds lay = inc_mm_lds(D, KB);
    float* Cs = reinterpret_cast<float*>(km_smem + lay.off_c);
    float* ca = reinterpret_cast<float*>(km_smem + lay.off_ca);
    float* cn2s = reinterpret_cast<float*>(km_smem + lay.off_cn);
    float* thr = reinterpret_cast<float*>(km_smem + lay.off_thr);
    float* ecs = reinterpret_cast<float*>(km_smem + lay.off_ec);
    float* ddn = reinterpret_cast<float*>(km_smem + lay.off_ddn);
    float* dup = reinterpret_cast<float*>(km_smem + lay.off_dup);
    float* hm = reinterpret_cast<float*>(km_smem + lay.off_hm);
    uint64_t* acc = reinterpret_cast<uint64_t*>(km_smem + lay.off_acc);
    int* cnt = reinterpret_cast<int*>(km_smem + lay.off_cnt);
    int* tcount = reinterpret_cast<int*>(km_smem + lay.off_misc);
    uint64_t* bst = reinterpret_cast<uint64_t*>(km_smem + lay.off_misc + 16);
    constexpr int NQ = inc_mm_queues(KB);
    int* qp = reinterpret_cast<int*>(km_smem + lay.off_q) + w * (2 * NQ * kQ);   // this wave's queues: points
    uint32_t* qw = reinterpret_cast<uint32_t*>(qp + NQ * kQ);                      // and their states
    float* nb = reinterpret_cast<float*>(km_smem + lay.off_nb);
    float* wg = reinterpret_cast<float*>(km_smem + lay.off_x) + w * kB * XS;       // its staged rows

    // Tables of the step.
    constexpr int AR = D + 1;   // LDS stride (uint64) of a cluster's sums: one pad word spreads clusters over banks
    for (int i = tid; i < KP * D; i += kW * 64) Cs[i] = i < k * D ? P.C32[i] : 0.f;
    for (int i = tid; i < KP * AR; i += kW * 64) acc[i] = 0;
    for (int i = tid; i < KP; i += kW * 64) {
        cn2s[i] = i < k ? P.cn2[i] : INFINITY;
        // -|c|^2 / 2 (exact halving) enters the matrix-core product as one
        // more dimension; padding centroids get a value no point reaches.
        nb[i] = i < k ? -0.5f * P.cn2[i] : -0x1p100f;
        cnt[i] = 0;
    }
    for (int i = tid; i < k; i += kW * 64) {
        thr[i] = first ? 0.f : clause1_thr(P.s[i], P.dhi[i]);
        ecs[i] = P.ec[i];
        ddn[i] = P.ddnf[i];
        dup[i] = P.dupf[i];
    }
    // hm[4a + cb]: the smallest half-distance from centroid a to a centroid
    // of block cb (zero for a's own block), from the centroid table.
    for (int i = tid; i < 4 * k; i += kW * 64) hm[i] = P.hm[i];
    if (tid < kNumStat) bst[tid] = 0;
    if (tid == 0) *tcount = 0;
    // Matrix-core A operands, split (hi, lo): at k-step s lane l feeds
    // centroid row 32*cb + l%32, dimensions 16 s + 8 (l/32) .. + 7.
    auto centroid_split = [&](int cb, int s, int l, uint4& hi, uint4& lo) __attribute__((always_inline)) {
        const int j = cb * 32 + (l & 31);
        float v[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = j < k ? P.C32[(int64_t)j * D + 16 * s + 8 * (l >> 5) + i] : 0.f;
        uint32_t h[4], o[4];
#pragma unroll
        for (int p = 0; p < 4; ++p) {
            float ra, rb;
            h[p] = split_hi(v[2 * p], v[2 * p + 1], ra, rb);
            o[p] = split_lo(ra, rb);
        }
        hi = make_uint4(h[0], h[1], h[2], h[3]);
        lo = make_uint4(o[0], o[1], o[2], o[3]);
    };
    uint4* cau = reinterpret_cast<uint4*>(ca);   // WIDE: [cb][s][hi, lo][lane]
    uint4 chi[WIDE ? 1 : KB][WIDE ? 1 : NS], clo[WIDE ? 1 : KB][WIDE ? 1 : NS];
    if constexpr (WIDE) {
        for (int i = tid; i < KB * NS * 64; i += kW * 64) {
            const int l = i & 63, s2 = (i >> 6) % NS, cb = i / (64 * NS);
            uint4 hi, lo;
            centroid_split(cb, s2, l, hi, lo);
            cau[((cb * NS + s2) * 2) * 64 + l] = hi;
            cau[((cb * NS + s2) * 2 + 1) * 64 + l] = lo;
        }
    } else {
#pragma unroll
        for (int cb = 0; cb < KB; ++cb)
#pragma unroll
            for (int s2 = 0; s2 < NS; ++s2) centroid_split(cb, s2, lane, chi[cb][s2], clo[cb][s2]);
    }
    __syncthreads();
    float cnmax;
    {
        float m2 = 0.f;
        for (int i = 0; i < k; ++i) m2 = fmaxf(m2, cn2s[i]);
        cnmax = sqrtf(m2) * kUp * kUp;
    }
    // Error bound of an expanded value (x and c the float32 row and
    // centroid): (D + 8) 2^-24 R^2 (R = |x| + max |c|) for the float32 norms
    // and roundings; for the split product 3.04 2^-16 |x_m| |c_m| per
    // dimension (the dropped lo.lo and the two roundings' residuals) and, at
    // most 18 units of 2^-23 relative to |C| + sum |p| per instruction of 16
    // exact bf16 products, 6.9 D 2^-24 sum |x_m| |c_m| over the 3 D / 16
    // instructions of a dot (doubled in the squared distance); an absolute
    // 2^-100 (1 + R) for bf16 values below the normal range.
    constexpr float gexp = (float)(D + 8) * 0x1p-24f;
    constexpr float gsp2 = 2.f * (778.f + 6.9f * (float)D) * 0x1p-24f * (1.f + 0x1p-10f);

    uint32_t my_changed = 0, my_comp = 0, my_rc = 0, c1w = 0;

    // The batch in flight: its rows (load i of lane l holds chunk l % CPR of
    // entry RPL * i + l / CPR) and size; each entry's point and state are
    // parked in the spare words of its staged row.
    const f32x4* X4 = reinterpret_cast<const f32x4*>(P.X);
    f32x4 r[kLoads];
    int bcnt = 0;
    auto take_batch = [&](int qi, int e0, int c) __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < kLoads; ++i) {
            const int e = RPL * i + lane / CPR;
            const int64_t rp = e < c ? (int64_t)qp[qi * kQ + e0 + e] : 0;
            r[i] = __builtin_nontemporal_load(X4 + rp * CPR + lane % CPR);
        }
        if (lane < kB) {
            int* park = reinterpret_cast<int*>(wg + lane * XS + D);
            park[0] = lane < c ? qp[qi * kQ + e0 + lane] : 0;
            park[1] = lane < c ? (int)qw[qi * kQ + e0 + lane] : 0;
        }
        bcnt = c;
    };

    auto dim_of = [&](int q) { return 16 * (q >> 3) + 8 * half + (q & 7); };
    auto scan_batch = [&]() __attribute__((always_inline)) {
#pragma unroll
        for (int i = 0; i < kLoads; ++i)
            *reinterpret_cast<f32x4*>(wg + (RPL * i + lane / CPR) * XS + 4 * (lane % CPR)) = r[i];
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        const bool live = col < bcnt;
        const float* xr = wg + col * XS;
        const int* park = reinterpret_cast<const int*>(xr + D);
        const int p = park[0];
        const uint32_t wst = (uint32_t)park[1];
        const int inc = first ? -1 : st_cluster(wst);
        // The lane's half of the row: dimensions 16 s + 8 half .. + 7 of each
        // k-step s (xh[8 s + i]).
        float xh[kHalf];
#pragma unroll
        for (int q = 0; q < kHalf; q += 4) {
            const f32x4 v = *reinterpret_cast<const f32x4*>(xr + dim_of(q));
            xh[q] = v.x;
            xh[q + 1] = v.y;
            xh[q + 2] = v.z;
            xh[q + 3] = v.w;
        }
        float x2 = 0.f;
#pragma unroll
        for (int q = 0; q < kHalf; ++q) x2 = fmaf(xh[q], xh[q], x2);
        x2 += __shfl_xor(x2, 32);

        // Clause 2 per 32-centroid block over the whole batch, with each
        // survivor's drift-updated bound.
        bool eval[KB];
        int nreal = 0;   // real centroids of the evaluated blocks
        {
            const float u = live && inc >= 0 ? (st_value(wst) + dup[inc]) * kUp : 0.f;
#pragma unroll
            for (int cb = 0; cb < KB; ++cb) {
                const bool need = live && !(prune && u <= hm[4 * max(inc, 0) + cb]);
                eval[cb] = !prune || __ballot(need) != 0;
                if (eval[cb]) nreal += min(32, max(k - 32 * cb, 0));
            }
        }
        // dot'_j = x.c_j - |c_j|^2 / 2: x.c_j from the bf16 matrix cores
        // (hi.hi + hi.lo + lo.hi per k-step), then -|c_j|^2 / 2 added.  The
        // squared distance is |x|^2 - 2 dot'_j, so the nearest centroid has
        // the largest dot'.
        uint4 bhi[NS], blo[NS];
#pragma unroll
        for (int s2 = 0; s2 < NS; ++s2) {
            uint32_t h[4], o[4];
#pragma unroll
            for (int p = 0; p < 4; ++p) {
                float ra, rb;
                h[p] = split_hi(xh[8 * s2 + 2 * p], xh[8 * s2 + 2 * p + 1], ra, rb);
                o[p] = split_lo(ra, rb);
            }
            bhi[s2] = make_uint4(h[0], h[1], h[2], h[3]);
            blo[s2] = make_uint4(o[0], o[1], o[2], o[3]);
        }
        auto bf = [](uint4 u) { return __builtin_bit_cast(bf16x8, u); };
        f32x16 dot[KB];
#pragma unroll
        for (int cb = 0; cb < KB; ++cb) {
            if (eval[cb]) {   // uniform
                f32x16 pr = {};
#pragma unroll
                for (int s2 = 0; s2 < NS; ++s2) {
                    const uint4 ah = WIDE ? cau[((cb * NS + s2) * 2) * 64 + lane] : chi[WIDE ? 0 : cb][WIDE ? 0 : s2];
                    const uint4 al = WIDE ? cau[((cb * NS + s2) * 2 + 1) * 64 + lane] : clo[WIDE ? 0 : cb][WIDE ? 0 : s2];
                    pr = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bf(ah), bf(bhi[s2]), pr, 0, 0, 0);
                    pr = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bf(ah), bf(blo[s2]), pr, 0, 0, 0);
                    pr = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bf(al), bf(bhi[s2]), pr, 0, 0, 0);
                }
#pragma unroll
                for (int a4 = 0; a4 < 4; ++a4) {
                    const f32x4 nv = *reinterpret_cast<const f32x4*>(nb + cb * 32 + 8 * a4 + 4 * half);
                    dot[cb][4 * a4] = pr[4 * a4] + nv.x;
                    dot[cb][4 * a4 + 1] = pr[4 * a4 + 1] + nv.y;
                    dot[cb][4 * a4 + 2] = pr[4 * a4 + 2] + nv.z;
                    dot[cb][4 * a4 + 3] = pr[4 * a4 + 3] + nv.w;
                }
            } else {
#pragma unroll
                for (int e = 0; e < 16; ++e) dot[cb][e] = -INFINITY;
            }
        }
        // Register e of block cb holds centroid 32*cb + 8*(e/4) + 4*half + e%4.
        auto cent = [&](int cb, int e) { return cb * 32 + 8 * (e >> 2) + 4 * half + (e & 3); };
        float dmax = -INFINITY;
#pragma unroll
        for (int cb = 0; cb < KB; ++cb)
#pragma unroll
            for (int e = 0; e < 16; ++e) dmax = fmaxf(dmax, dot[cb][e]);
        dmax = fmaxf(dmax, __shfl_xor(dmax, 32));
        const float e1 = fmaf(-2.f, dmax, x2);   // the smallest squared distance, expanded form
        // Candidates: dot' within E of the largest (squared distances within
        // 2E of the smallest); every other evaluated centroid is certified
        // farther than the nearest.  A single candidate is counted and found
        // in the same pass.
        const float xn = sqrtf(fmaxf(x2, 0.f)) * (1.0f + 0x1p-20f);
        const float R = xn + cnmax;
        const float E = (gexp * R * R + gsp2 * xn * cnmax + 4.f * R * ecmax + 2.f * ecmax * ecmax +
                         0x1p-100f * (1.f + R)) * kUp;
        const float lim = dmax - E;
        int own = 0, jown = -1;
#pragma unroll
        for (int cb = 0; cb < KB; ++cb)
#pragma unroll
            for (int e = 0; e < 16; ++e) {
                const bool c = dot[cb][e] >= lim;
                own += c ? 1 : 0;
                jown = c ? cb * 32 + 8 * (e >> 2) + (e & 3) : jown;
            }
        jown = jown >= 0 ? jown + 4 * half : -1;
        const bool single = own + __shfl_xor(own, 32) == 1;
        const int jsingle = max(jown, __shfl_xor(jown, 32));
        uint64_t cmask = 0;
        if (!single) {   // the candidate mask (rarely needed)
#pragma unroll
            for (int cb = 0; cb < KB; ++cb)
#pragma unroll
                for (int e = 0; e < 16; ++e)
                    if (dot[cb][e] >= lim) cmask |= 1ull << (16 * cb + e);
        }
        const uint64_t cmask0 = cmask;
        // Several candidates: direct-form distances, each half over its own,
        // then the smaller (distance, incumbent first, lower index).
        float d1 = INFINITY, d2 = INFINITY;
        int rk1 = INT_MAX, j1 = 0;
        while (cmask) {
            const int bit = __builtin_ctzll(cmask);
            cmask &= cmask - 1;
            const int j = cent(bit >> 4, bit & 15);
            const float Dd = sqd_lds_fixed<D>(xr, Cs + j * D);
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
        {
            const float od1 = __shfl_xor(d1, 32), od2 = __shfl_xor(d2, 32);
            const int ork = __shfl_xor(rk1, 32), oj = __shfl_xor(j1, 32);
            if (od1 < d1 || (od1 == d1 && ork < rk1)) {
                d2 = fminf(d1, fminf(d2, od2));
                d1 = od1;
                j1 = oj;
            } else {
                d2 = fminf(d2, fminf(od1, od2));
            }
        }
        bool re = false;
        if (!single && d2 != INFINITY) {
            const float band = 2.f * gamma * (d1 + d2) + 4.f * (sqrtf(d1) + sqrtf(d2)) * ecmax + 8.f * ecmax * ecmax;
            re = live && d2 - d1 <= band;
        }
        double Dbb = INFINITY;
        int kb = INT_MAX, bb = -1;
        if (re) {   // near tie: float64 decision among the candidates
            uint64_t cm = cmask0;
            while (cm) {
                const int bit = __builtin_ctzll(cm);
                cm &= cm - 1;
                const int j = cent(bit >> 4, bit & 15);
                const double Dj = sqd64(xr, P.C64 + (int64_t)j * D, D);
                const int rk = j == inc ? -1 : j;
                if (Dj < Dbb || (Dj == Dbb && rk < kb)) {
                    Dbb = Dj;
                    kb = rk;
                    bb = j;
                }
            }
        }
        {
            const double oD = __shfl_xor(Dbb, 32);
            const int okb = __shfl_xor(kb, 32), obb = __shfl_xor(bb, 32);
            if (oD < Dbb || (oD == Dbb && okb < kb)) {
                Dbb = oD;
                kb = okb;
                bb = obb;
            }
        }
        int b = j1;
        float ub;
        if (single) {
            b = jsingle;
            ub = sqrt_up(fmaxf(e1 + E, 0.f)) * kUp;
        } else if (re) {
            b = bb < 0 ? 0 : bb;
            ub = f32_up(sqrt(Dbb) * (1.0 + 0x1p-40));
        } else {
            ub = upper_bound(d1, ecs[b], gamma);
        }
        if (live) {
            const bool moved = b != inc;
            if (half == 0) {
                const float rr = ub - ddn[b];   // v = ub - D_b, rounded up
                P.w[p] = pack7(rr + fabsf(rr) * 0x1p-22f, b);
                my_comp += (uint32_t)nreal;
                my_rc += re ? 1u : 0u;
                my_changed += moved ? 1u : 0u;
                if (moved) {
                    atomicAdd(&cnt[b], 1);
                    if (inc >= 0) atomicAdd(&cnt[inc], -1);
                }
            }
            if (moved) {   // each half moves its half of the row
#pragma unroll
                for (int q = 0; q < kHalf; ++q) {
                    const uint64_t v = fixed_bits((double)xh[q], P.qscale);
                    atomicAdd(reinterpret_cast<unsigned long long*>(acc + b * AR + dim_of(q)),
                              (unsigned long long)v);
                    if (inc >= 0)
                        lds_sub64(acc + inc * AR + dim_of(q), v);
                }
            }
        }
        bcnt = 0;
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();   // staged rows consumed before the next batch is staged
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    };

    // Queue lengths (wave-uniform).
    int qn[NQ];
#pragma unroll
    for (int qi = 0; qi < NQ; ++qi) qn[qi] = 0;
    // Settles the batch in flight and takes the next from the fullest queue
    // while one holds a whole batch (at the end: while any holds entries).
    auto batch_point = [&](bool drain) __attribute__((always_inline)) {
        for (;;) {
            int qsel = -1, best = drain ? 0 : kB - 1;
#pragma unroll
            for (int qi = 0; qi < NQ; ++qi)
                if (qn[qi] > best) {
                    best = qn[qi];
                    qsel = qi;
                }
            if (qsel < 0) {   // nothing to take: the batch in flight waits for the next point (or the end)
                if (drain && bcnt > 0) scan_batch();
                break;
            }
            if (bcnt > 0) scan_batch();
            const int c = min(best, kB);
#pragma unroll
            for (int qi = 0; qi < NQ; ++qi)
                if (qi == qsel) qn[qi] -= c;
            take_batch(qsel, best - c, c);   // the newest c entries
        }
    };

    const int64_t n = P.n;
    const int nwt = (int)((n + kIMTile - 1) / kIMTile);
    const int wt_lo = (int)((int64_t)blockIdx.x * nwt / gridDim.x);
    const int wt_hi = (int)((int64_t)(blockIdx.x + 1) * nwt / gridDim.x);
    int wt = wt_lo + w;
    while (wt < wt_hi) {
        const int base = wt * kIMTile;
        uint32_t sv[4];
#pragma unroll
        for (int c = 0; c < 4; ++c) sv[c] = P.w[base + kIMSub * c + lane];   // the state array is padded
        int nxt = 0;
        if (lane == 0) nxt = wt_lo + kW + atomicAdd(tcount, 1);
        nxt = __builtin_amdgcn_readfirstlane(nxt);
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const int p = base + kIMSub * c + lane;
            const bool valid = p < n;
            const uint32_t ws = sv[c];
            const int a = first ? 0 : st_cluster(ws);
            const bool surv = valid && (first || !prune || !(st_value(ws) <= thr[a]));
            const uint64_t kept = __ballot(valid && !surv);
            c1w += (uint32_t)__popcll(kept);
            // Queue: for KB <= 2 the set of blocks the survivor needs (its
            // own block and every block Clause 2 does not skip for it), so
            // that a batch skips the blocks none of its survivors needs; for
            // KB = 4 the block of its cluster.
            int key;
            if constexpr (KB == 4) {
                key = a >> 5;
            } else {
                int mask = (1 << KB) - 1;
                if (!first && prune) {
                    const float u = (st_value(ws) + dup[a]) * kUp;
                    mask = 0;
#pragma unroll
                    for (int cb = 0; cb < KB; ++cb)
                        mask |= (cb == (a >> 5) || !(u <= hm[4 * a + cb])) ? 1 << cb : 0;
                }
                key = mask - 1;
            }
#pragma unroll
            for (int qi = 0; qi < NQ; ++qi) {
                const bool mine = surv && key == qi;
                const uint64_t bm = __ballot(mine);
                if (mine) {
                    const int e = qn[qi] + lanes_below(bm);
                    qp[qi * kQ + e] = p;
                    qw[qi * kQ + e] = ws;
                }
                qn[qi] += __popcll(bm);
            }
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();   // queue entries visible to the whole wave
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
            batch_point(false);
        }
        wt = nxt;
    }
    batch_point(true);

    // Block counters, then the block's partial row (the moves).
    const uint64_t v0 = wave_sum_u64(my_changed), v1 = wave_sum_u64(my_comp), v3 = wave_sum_u64(my_rc);
    __syncthreads();
    if (lane == 0) {
        unsigned long long* bs = reinterpret_cast<unsigned long long*>(bst);
        atomicAdd(bs + kStChanged, (unsigned long long)v0);
        atomicAdd(bs + kStComputed, (unsigned long long)v1);
        atomicAdd(bs + kStClause1, (unsigned long long)c1w);
        atomicAdd(bs + kStRecheck, (unsigned long long)v3);
    }
    __syncthreads();
    uint64_t* row = P.part + (int64_t)blockIdx.x * P.L;
    for (int i = tid; i < k * D; i += kW * 64) row[i] = acc[(i / D) * AR + i % D];
    for (int i = tid; i < k; i += kW * 64) row[k * D + i] = (uint64_t)(int64_t)cnt[i];
    if (tid < kNumStat) row[k * D + k + tid] = bst[tid];
}

__global__ __launch_bounds__(256) void k_inc_mm_unpack(const uint32_t* __restrict__ w, int64_t n,
                                                       int32_t* __restrict__ a) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) a[i] = st_cluster(w[i]);
}

}  // namespace

bool inc_mm_applies(int64_t n, int d, int k, bool aligned) {
    // int32 point indices, also over the state array's padding
    return aligned && (d == 16 || d == 32) && k <= kIMMaxK && n <= (int64_t)INT_MAX - kIMTile;
}

int inc_mm_kb(int k) { return k <= 32 ? 1 : (k <= 64 ? 2 : 4); }

#define KM_IM_VARIANTS(X) X(16, 1) X(16, 2) X(16, 4) X(32, 1) X(32, 2) X(32, 4)

const void* inc_mm_symbol(int d, int k) {
    const int kb = inc_mm_kb(k);
#define KM_SYM(D_, KB_) \
    if (d == D_ && kb == KB_) return reinterpret_cast<const void*>(&k_inc_mm<D_, KB_>);
    KM_IM_VARIANTS(KM_SYM)
#undef KM_SYM
    return nullptr;
}

hipError_t launch_inc_mm(const Dev& dv, int grid, int lds_bytes, int first, hipStream_t s) {
    const int kb = inc_mm_kb(dv.k);
#define KM_LAUNCH(D_, KB_)                                                                               \
    if (dv.d == D_ && kb == KB_) {                                                                       \
        hipLaunchKernelGGL((k_inc_mm<D_, KB_>), dim3(grid), dim3(kW * 64), lds_bytes, s, dv, first); \
        return hipGetLastError();                                                                        \
    }
    KM_IM_VARIANTS(KM_LAUNCH)
#undef KM_LAUNCH
    return hipErrorInvalidValue;
}

hipError_t launch_inc_mm_unpack(const Dev& dv, int32_t* assign_out, hipStream_t s) {
    int64_t blocks = (dv.n + 255) / 256;
    if (blocks > 8192) blocks = 8192;
    hipLaunchKernelGGL(k_inc_mm_unpack, dim3((unsigned)blocks), dim3(256), 0, s, dv.w, dv.n, assign_out);
    return hipGetLastError();
}

}  // namespace km
