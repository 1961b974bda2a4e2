// Drift-based block selection (Secs. 4.2-4.3), one launch for every row of a
// layer: pooled map, drift scores, exact top-c, R budget-neutral restoration
// rounds with track-best, and compaction of the kept-block lists.
//
// Work layout. A workgroup holds 4 independent waves; each wave owns R query
// blocks ("rows") of one head, so loads of the head's pooled key/value tensors
// are shared by the R rows in registers and by the 4 waves through L1.
//  - Per-candidate quantities live "lane <-> key block": lane l, slot c holds key
//    block j = l + 64 c (CPL slots). Channel-major copies of the pooled tensors
//    make these passes coalesced.
//  - Per-row vectors (vbar, M vbar, g, M g) live "lane <-> channel" (D = 64 is
//    the wave width); values are broadcast with readlane.
//  - Every top-k is exact: a bitwise search for the k-th largest of
//    order-preserving 64-bit keys, using wave ballots and popcounts, ties broken
//    by the lower block index. No atomics, no data-dependent reduction order:
//    reruns are bit-identical.
// All arithmetic is float64: CDNA4 runs float64 FMA at the rate of unpacked
// float32, and it keeps the discrete decisions stable.
#include <math.h>

#include "ress_internal.h"

namespace ress {
namespace {

constexpr int kThreads = 256;

__device__ __forceinline__ double readlane_f64(double x, int l)
{
    const long long u = __double_as_longlong(x);
    const int lo = __builtin_amdgcn_readlane((int)u, l);
    const int hi = __builtin_amdgcn_readlane((int)(u >> 32), l);
    return __longlong_as_double(((long long)hi << 32) | (unsigned int)lo);
}

__device__ __forceinline__ double wave_sum(double x)
{
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o);
    return x;  // butterfly with commutative adds: identical in every lane
}

__device__ __forceinline__ double wave_max(double x)
{
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) x = fmax(x, __shfl_xor(x, o));
    return x;
}

// Order-preserving map of a double to uint64 (larger value -> larger key);
// -0 is folded onto +0 so that equal values get equal keys.
__device__ __forceinline__ unsigned long long order_key(double x)
{
    const unsigned long long u = (unsigned long long)__double_as_longlong(x + 0.0);
    return (u >> 63) ? ~u : (u | 0x8000000000000000ull);
}

// Exact top-k of the member slots by (key desc, block index asc). Returns this
// lane's chosen slots as a bit mask. Requires 0 <= k <= number of members.
template <int CPL>
__device__ unsigned long long topk_slots(const unsigned long long (&key)[CPL],
                                         unsigned long long memb, int k, unsigned long long lane_lt)
{
    if (k <= 0) return 0ull;
    unsigned long long thr = 0;  // invariant: #members with key >= thr is >= k
    bool exact = false;
    for (int b = 63; b >= 0; --b) {
        const unsigned long long cand = thr | (1ull << b);
        int cnt = 0;
#pragma unroll
        for (int c = 0; c < CPL; ++c) cnt += __popcll(__ballot(((memb >> c) & 1ull) && key[c] >= cand));
        if (cnt >= k) {
            thr = cand;
            if (cnt == k) {  // exactly k keys reach thr: they are the top k
                exact = true;
                break;
            }
        }
    }
    unsigned long long chosen = 0;
    if (exact) {
#pragma unroll
        for (int c = 0; c < CPL; ++c)
            if (((memb >> c) & 1ull) && key[c] >= thr) chosen |= 1ull << c;
        return chosen;
    }
    // thr is the k-th largest key; take all larger ones and the lowest-index ties.
    int gt = 0;
#pragma unroll
    for (int c = 0; c < CPL; ++c) gt += __popcll(__ballot(((memb >> c) & 1ull) && key[c] > thr));
    const int need = k - gt;
    int before = 0;
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
        const bool m = (memb >> c) & 1ull;
        const bool tie = m && key[c] == thr;
        const unsigned long long tb = __ballot(tie);
        const int rank = before + __popcll(tb & lane_lt);
        if (m && (key[c] > thr || (tie && rank < need))) chosen |= 1ull << c;
        before += __popcll(tb);
    }
    return chosen;
}

// Swap count of round r (Eq. 17): max(floor, floor(rho c 2^-(r+1))).
__device__ __forceinline__ int swaps_of_round(int c, double rho, int r, int swap_floor)
{
    const int m = (int)floor(rho * (double)c * ldexp(1.0, -(r + 1)));
    return m > swap_floor ? m : swap_floor;
}

// x = M_h y for a lane <-> channel vector y (M row-major, staged in LDS).
__device__ __forceinline__ double mat_vec(const float *Ms, double y, int lane)
{
    double acc = 0.0;
    for (int b = 0; b < kD; ++b) acc = fma((double)Ms[lane * (kD + 1) + b], readlane_f64(y, b), acc);
    return acc;
}

template <int CPL, int R>
__global__ void __launch_bounds__(kThreads) select_kernel(const SelectParams p)
{
    __shared__ float Ms[kD * (kD + 1)];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const unsigned long long lane_lt = (1ull << lane) - 1ull;
    const int groups = (p.n_qb + 4 * R - 1) / (4 * R);
    const int h = blockIdx.x / groups;
    const int row0 = (blockIdx.x % groups) * 4 * R + wave * R;
    {
        const float *Mh = p.gram + (size_t)h * kD * kD;
        for (int e = threadIdx.x; e < kD * kD; e += kThreads) Ms[(e >> 6) * (kD + 1) + (e & 63)] = Mh[e];
    }
    __syncthreads();
    if (row0 >= p.n_qb) return;

    const int nkb = p.n_kb, nqb = p.n_qb;
    const double eps = p.eps;
    const double *Kt = p.pooled.kbarT + (size_t)h * kD * nkb;
    const double *Vr = p.pooled.vbar + (size_t)h * nkb * kD;
    const double *Vt = p.pooled.vbarT + (size_t)h * kD * nkb;
    const double *Ut = p.pooled.uT + (size_t)h * kD * nkb;
    const double *Qb = p.pooled.qbar + (size_t)h * nqb * kD;
    const int c_h = p.budgets[h];
    const int n_p = p.first_forced;  // candidates are the key blocks j < first_forced

    int irow[R];
    bool live[R], dense[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        live[r] = row0 + r < nqb;
        irow[r] = live[r] ? row0 + r : nqb - 1;
        dense[r] = irow[r] >= p.first_dense_qb || c_h >= n_p;
    }
    unsigned long long memb = 0;  // candidate slots of this lane
#pragma unroll
    for (int c = 0; c < CPL; ++c)
        if (lane + 64 * c < n_p) memb |= 1ull << c;

    // Pooled logits Qbar_i . Kbar_j / sqrt(D) (Eq. 1).
    double acc[R][CPL], P[R][CPL], S2[R][CPL];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
        for (int c = 0; c < CPL; ++c) acc[r][c] = 0.0;
    for (int d = 0; d < kD; ++d) {
        double kd[CPL];
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
            const int j = lane + 64 * c;
            kd[c] = j < nkb ? Kt[(size_t)d * nkb + j] : 0.0;
        }
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const double qd = Qb[(size_t)irow[r] * kD + d];
#pragma unroll
            for (int c = 0; c < CPL; ++c) acc[r][c] = fma(qd, kd[c], acc[r][c]);
        }
    }
    // Softmax over all key blocks.
#pragma unroll
    for (int r = 0; r < R; ++r) {
        double mx = -INFINITY;
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
            acc[r][c] *= 0.125;  // 1/sqrt(64)
            if (lane + 64 * c < nkb) mx = fmax(mx, acc[r][c]);
        }
        mx = wave_max(mx);
        double z = 0.0;
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
            P[r][c] = lane + 64 * c < nkb ? exp(acc[r][c] - mx) : 0.0;
            z += P[r][c];
        }
        z = wave_sum(z);
#pragma unroll
        for (int c = 0; c < CPL; ++c) P[r][c] = P[r][c] / z;
        if (p.prob_out && live[r]) {
            double *po = p.prob_out + ((size_t)h * nqb + irow[r]) * nkb;
#pragma unroll
            for (int c = 0; c < CPL; ++c)
                if (lane + 64 * c < nkb) po[lane + 64 * c] = P[r][c];
        }
    }

    // Dense pooled output vbar_i = sum_j P_ij Vbar_j (lane <-> channel) and M vbar_i.
    double vb[R], wv[R];
#pragma unroll
    for (int r = 0; r < R; ++r) vb[r] = 0.0;
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
        const int lim = min(64, nkb - 64 * c);
        for (int l2 = 0; l2 < lim; ++l2) {
            const double vjd = Vr[(size_t)(64 * c + l2) * kD + lane];
#pragma unroll
            for (int r = 0; r < R; ++r) vb[r] = fma(readlane_f64(P[r][c], l2), vjd, vb[r]);
        }
    }
#pragma unroll
    for (int r = 0; r < R; ++r) wv[r] = mat_vec(Ms, vb[r], lane);

    // q_ij = e^T M e with e = vbar_i - Vbar_j, as e . (M vbar_i - M Vbar_j) (Eq. 9);
    // s_ij = P_ij sqrt(q_ij), key_ij = s_ij / max(1 - P_ij, eps) (Eqs. 6-7).
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
        for (int c = 0; c < CPL; ++c) acc[r][c] = 0.0;
    for (int d = 0; d < kD; ++d) {
        double vt[CPL], ut[CPL];
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
            const int j = lane + 64 * c;
            vt[c] = j < nkb ? Vt[(size_t)d * nkb + j] : 0.0;
            ut[c] = j < nkb ? Ut[(size_t)d * nkb + j] : 0.0;
        }
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const double vbd = readlane_f64(vb[r], d), wd = readlane_f64(wv[r], d);
#pragma unroll
            for (int c = 0; c < CPL; ++c) acc[r][c] = fma(vbd - vt[c], wd - ut[c], acc[r][c]);
        }
    }
#pragma unroll
    for (int r = 0; r < R; ++r) {
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
            const double q = acc[r][c];
            const double s = P[r][c] * sqrt(q > 0.0 ? q : 0.0);
            const double den = 1.0 - P[r][c];
            S2[r][c] = s * s;
            acc[r][c] = s / (den > eps ? den : eps);  // ranking key
        }
        if (p.key_out && live[r]) {
            double *ko = p.key_out + ((size_t)h * nqb + irow[r]) * nkb;
#pragma unroll
            for (int c = 0; c < CPL; ++c) {
                const int j = lane + 64 * c;
                if (j < nkb) ko[j] = j < n_p ? acc[r][c] : -1.0;
            }
        }
    }

    // Initial selection (Eq. 7) and the state of its drop set (Eqs. 10-12).
    unsigned long long inD[R], best[R];
    double K[R], G[R], J[R], J0[R], Jb[R], gd[R], hd[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        inD[r] = best[r] = 0ull;
        K[r] = 1.0;
        G[r] = J[r] = J0[r] = Jb[r] = gd[r] = hd[r] = 0.0;
        if (dense[r]) continue;
        unsigned long long ko[CPL];
#pragma unroll
        for (int c = 0; c < CPL; ++c) ko[c] = order_key(acc[r][c]);
        inD[r] = memb & ~topk_slots<CPL>(ko, memb, c_h, lane_lt);
        double mass = 0.0;
#pragma unroll
        for (int c = 0; c < CPL; ++c)
            if ((inD[r] >> c) & 1ull) mass += P[r][c];
        K[r] = 1.0 - wave_sum(mass);
        double g = 0.0;
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
            unsigned long long bm = __ballot((inD[r] >> c) & 1ull);
            while (bm) {
                const int b = __ffsll((long long)bm) - 1;
                bm &= bm - 1ull;
                const double pj = readlane_f64(P[r][c], b);
                g = fma(pj, vb[r] - Vr[(size_t)(64 * c + b) * kD + lane], g);
            }
        }
        gd[r] = g;
        hd[r] = mat_vec(Ms, g, lane);
        G[r] = wave_sum(g * hd[r]);
        const double Kh = K[r] > eps ? K[r] : eps;
        J[r] = J0[r] = Jb[r] = G[r] / (Kh * Kh);
        best[r] = inD[r];
    }

    // Budget-neutral restoration rounds (Eqs. 13-17) with track-best.
    const int nD = n_p - c_h, nS = c_h;
    for (int rr = 0; rr < p.rounds; ++rr) {
        int m = swaps_of_round(c_h, p.rho, rr, p.swap_floor);
        m = min(m, min(nD, nS));
        if (m <= 0) break;
        // e_k . (M g) for every candidate k of every row (shares the loads).
#pragma unroll
        for (int r = 0; r < R; ++r)
#pragma unroll
            for (int c = 0; c < CPL; ++c) acc[r][c] = 0.0;
        for (int d = 0; d < kD; ++d) {
            double vt[CPL];
#pragma unroll
            for (int c = 0; c < CPL; ++c) {
                const int j = lane + 64 * c;
                vt[c] = j < nkb ? Vt[(size_t)d * nkb + j] : 0.0;
            }
#pragma unroll
            for (int r = 0; r < R; ++r) {
                const double vbd = readlane_f64(vb[r], d), hdd = readlane_f64(hd[r], d);
#pragma unroll
                for (int c = 0; c < CPL; ++c) acc[r][c] = fma(vbd - vt[c], hdd, acc[r][c]);
            }
        }
#pragma unroll
        for (int r = 0; r < R; ++r) {
            if (dense[r]) continue;
            unsigned long long dj[CPL];
#pragma unroll
            for (int c = 0; c < CPL; ++c) {
                const double dkMg = P[r][c] * acc[r][c];
                double dG, u;
                if ((inD[r] >> c) & 1ull) {  // restore: Eq. 14
                    dG = -2.0 * dkMg + S2[r][c];
                    u = P[r][c];
                } else {  // drop: Eq. 15
                    dG = 2.0 * dkMg + S2[r][c];
                    u = -P[r][c];
                }
                const double Kn = K[r] + u;
                const double Knh = Kn > eps ? Kn : eps;
                dj[c] = order_key(J[r] - (G[r] + dG) / (Knh * Knh));  // Eq. 16
            }
            const unsigned long long rest = topk_slots<CPL>(dj, inD[r], m, lane_lt);
            const unsigned long long drop = topk_slots<CPL>(dj, memb & ~inD[r], m, lane_lt);
            double mr = 0.0, md = 0.0;
#pragma unroll
            for (int c = 0; c < CPL; ++c) {
                if ((rest >> c) & 1ull) mr += P[r][c];
                if ((drop >> c) & 1ull) md += P[r][c];
            }
            K[r] = (K[r] + wave_sum(mr)) - wave_sum(md);  // Eq. 13
            double g = gd[r];
#pragma unroll
            for (int c = 0; c < CPL; ++c) {
                unsigned long long bm = __ballot((rest >> c) & 1ull);
                while (bm) {
                    const int b = __ffsll((long long)bm) - 1;
                    bm &= bm - 1ull;
                    const double pj = readlane_f64(P[r][c], b);
                    g = fma(-pj, vb[r] - Vr[(size_t)(64 * c + b) * kD + lane], g);
                }
                bm = __ballot((drop >> c) & 1ull);
                while (bm) {
                    const int b = __ffsll((long long)bm) - 1;
                    bm &= bm - 1ull;
                    const double pj = readlane_f64(P[r][c], b);
                    g = fma(pj, vb[r] - Vr[(size_t)(64 * c + b) * kD + lane], g);
                }
            }
            gd[r] = g;
            inD[r] = (inD[r] & ~rest) | drop;
            hd[r] = mat_vec(Ms, g, lane);
            G[r] = wave_sum(g * hd[r]);
            const double Kh = K[r] > eps ? K[r] : eps;
            J[r] = G[r] / (Kh * Kh);
            if (J[r] < Jb[r]) {
                Jb[r] = J[r];
                best[r] = inD[r];
            }
        }
    }

    // Kept lists: (P \ D_best) u F in ascending block order, padded with -1.
#pragma unroll
    for (int r = 0; r < R; ++r) {
        if (!live[r]) continue;
        const size_t row = (size_t)h * nqb + irow[r];
        int32_t *out = p.kept_idx + row * nkb;
        int before = 0;
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
            const int j = lane + 64 * c;
            const bool kept = j < nkb && !((best[r] >> c) & 1ull);
            const unsigned long long km = __ballot(kept);
            if (kept) out[before + __popcll(km & lane_lt)] = j;
            before += __popcll(km);
        }
        for (int t = before + lane; t < nkb; t += 64) out[t] = -1;
        if (lane == 0) {
            p.kept_count[row] = before;
            if (p.drift) {
                p.drift[2 * row] = J0[r];
                p.drift[2 * row + 1] = Jb[r];
            }
        }
    }
}

template <int CPL, int R>
hipError_t launch_cfg(const SelectParams &p, hipStream_t s)
{
    const int groups = (p.n_qb + 4 * R - 1) / (4 * R);
    hipLaunchKernelGGL((select_kernel<CPL, R>), dim3((unsigned)(p.H * groups)), dim3(kThreads), 0, s, p);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_select(const SelectParams &p, hipStream_t s)
{
    if (p.H == 0 || p.n_qb == 0) return hipSuccess;
    const int n = p.n_kb;
    if (n <= 64) return launch_cfg<1, 4>(p, s);
    if (n <= 128) return launch_cfg<2, 4>(p, s);
    if (n <= 256) return launch_cfg<4, 4>(p, s);
    if (n <= 384) return launch_cfg<6, 4>(p, s);
    if (n <= 512) return launch_cfg<8, 2>(p, s);
    if (n <= 768) return launch_cfg<12, 2>(p, s);
    if (n <= 1088) return launch_cfg<17, 2>(p, s);
    if (n <= 1536) return launch_cfg<24, 1>(p, s);
    if (n <= 2048) return launch_cfg<32, 1>(p, s);
    if (n <= 3072) return launch_cfg<48, 1>(p, s);
    return launch_cfg<64, 1>(p, s);
}

}  // namespace ress
