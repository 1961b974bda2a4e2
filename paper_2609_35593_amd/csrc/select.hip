// Drift-based block selection (Secs. 4.2-4.3), one launch for every row of a
// layer: pooled map, drift scores, exact top-c, R budget-neutral restoration
// rounds with track-best, and compaction of the kept-block lists.
//
// Work layout. A workgroup holds 4 independent waves; each wave owns R query
// blocks ("rows") of one head, so every load of the head's pooled key/value
// tensors is used by the R rows in registers and by the 4 waves through L1.
//  - Per-candidate quantities live "lane <-> key block": lane l, slot c holds key
//    block j = l + 64 c (CPL slots).
//  - Per-row vectors (Qbar, vbar, S vbar with S the symmetric part of M, g, M g)
//    live "lane <-> channel"
//    (D = 64 is the wave width) and are broadcast to the candidate lanes through
//    the wave's LDS area, two doubles per read.
//  - Every top-k is exact: a bitwise search for the k-th largest of
//    order-preserving 64-bit keys, using wave ballots and popcounts, ties broken
//    by the lower block index. No atomics and no data-dependent reduction
//    order: reruns are bit-identical.
// All arithmetic is float64: CDNA4 runs float64 FMA at the rate of unpacked
// float32, and it keeps the discrete decisions stable.
#include <math.h>

#include "ress_internal.h"

namespace ress {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
// Word 3 of a raw buffer descriptor on gfx9-family chips (32-bit data format,
// no swizzle, no index stride): loads past num_records bytes return zero.
constexpr int kBufWord3 = 0x00020000;

// Buffer descriptor over one head's pooled tensor (n_kb x 64 doubles, either layout).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t pooled_rsrc(const double *base, int nkb)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<double *>(base), 0, kD * nkb * (int)sizeof(double),
                                             kBufWord3);
}

// Channel `lane` of row j (wave-uniform) of a row-major pooled tensor.
__device__ __forceinline__ double pooled_row(__amdgpu_buffer_rsrc_t rs, int j, int lane)
{
    return __builtin_bit_cast(double, __builtin_amdgcn_raw_buffer_load_b64(
                                          rs, (unsigned)lane * (unsigned)sizeof(double),
                                          __builtin_amdgcn_readfirstlane(j) * kD * (int)sizeof(double), 0));
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

// Exact top-k of the member slots by (key desc, block index asc). memb[c] is the
// wave-wide mask of member lanes of slot c. Returns this lane's chosen slots as
// a bit mask. Requires 0 <= k <= number of members.
template <int CPL>
__device__ unsigned long long topk_slots(const unsigned long long (&key)[CPL],
                                         const unsigned long long (&memb)[CPL], int k,
                                         unsigned long long lane_bit, unsigned long long lane_lt)
{
    if (k <= 0) return 0ull;
    unsigned long long thr = 0;  // invariant: #members with key >= thr is >= k
    bool exact = false;
    for (int b = 63; b >= 0; --b) {
        const unsigned long long cand = thr | (1ull << b);
        int cnt = 0;
#pragma unroll
        for (int c = 0; c < CPL; ++c) cnt += __popcll(__ballot(key[c] >= cand) & memb[c]);
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
            if ((memb[c] & lane_bit) && key[c] >= thr) chosen |= 1ull << c;
        return chosen;
    }
    // thr is the k-th largest key; take all larger ones and the lowest-index ties.
    int gt = 0;
#pragma unroll
    for (int c = 0; c < CPL; ++c) gt += __popcll(__ballot(key[c] > thr) & memb[c]);
    const int need = k - gt;
    int before = 0;
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
        const unsigned long long tb = __ballot(key[c] == thr) & memb[c];
        const int rank = before + __popcll(tb & lane_lt);
        if ((memb[c] & lane_bit) && (key[c] > thr || ((tb & lane_bit) && rank < need))) chosen |= 1ull << c;
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

// Per-wave LDS area (doubles): broadcast vectors vec[slot][R][64], one slot of
// block weights wts[R][64], and a swap list of up to 64 (block, weight) pairs plus
// padding to a multiple of 8. Every part starts on a 16-byte boundary.
template <int R>
struct WaveLds {
    static constexpr int kVecs = 3;  // 0: Qbar then vbar, 1: M vbar then M g, 2: g
    static constexpr int kSwaps = 72;
    static constexpr int kDoubles = kVecs * R * kD + R * 64 + kSwaps + kSwaps / 2;
    static_assert(kDoubles % 2 == 0, "16-byte aligned wave areas");
    double *base;
    __device__ double *vec(int slot, int r) const { return base + (slot * R + r) * kD; }
    __device__ double *wts(int r) const { return base + kVecs * R * kD + r * 64; }
    __device__ double *swap_w() const { return base + kVecs * R * kD + R * 64; }
    __device__ int *swap_j() const { return reinterpret_cast<int *>(base + kVecs * R * kD + R * 64 + kSwaps); }
};

// x_r = M y_r for the R rows, lane <-> output channel, M row-major in LDS (padded
// rows), y_r broadcast from LDS two channels at a time; with SYM, x_r = (M + M^T)/2
// y_r (the matrix whose quadratic form equals that of M, exact in float64 from
// float32 entries).
template <int R, bool SYM>
__device__ __forceinline__ void mat_vec(const float *Ms, double *const (&y)[R], double (&x)[R], int lane)
{
#pragma unroll
    for (int r = 0; r < R; ++r) x[r] = 0.0;
#pragma unroll 4
    for (int b = 0; b < kD; b += 2) {
        double m0 = (double)Ms[lane * (kD + 1) + b], m1 = (double)Ms[lane * (kD + 1) + b + 1];
        if (SYM) {
            m0 = 0.5 * (m0 + (double)Ms[b * (kD + 1) + lane]);
            m1 = 0.5 * (m1 + (double)Ms[(b + 1) * (kD + 1) + lane]);
        }
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const double2 yb = *reinterpret_cast<const double2 *>(y[r] + b);
            x[r] = fma(m1, yb.y, fma(m0, yb.x, x[r]));
        }
    }
}

// Pass over the head's key blocks, lane <-> channel, with per-row block weights
// w_r(j) held by the lane owning block j (slot c):
//   SUB: out_r = sum_j w_r(j) (x_r - Vbar_j)      (net drift g, Eq. 10)
//  !SUB: out_r = sum_j w_r(j) Vbar_j              (dense pooled output, Eq. 1)
// in ascending block order with eight rows of Vbar in flight; the weights of one
// slot (64 blocks) at a time are staged in the wave's LDS area.
template <int CPL, int R, bool SUB>
__device__ __forceinline__ void block_pass(const WaveLds<R> &lds, const double (&w)[R][CPL], const double (&x)[R],
                                           const double *__restrict__ Vr, int nkb, int lane, double (&out)[R])
{
    const __amdgpu_buffer_rsrc_t rsV = pooled_rsrc(Vr, nkb);
#pragma unroll
    for (int r = 0; r < R; ++r) out[r] = 0.0;
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int r = 0; r < R; ++r) lds.wts(r)[lane] = w[r][c];  // 0 past the last block
        __builtin_amdgcn_wave_barrier();
        const int lim = min(64, nkb - 64 * c);
        for (int l0 = 0; l0 < lim; l0 += 8) {
            double vj[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) vj[u] = pooled_row(rsV, 64 * c + min(l0 + u, lim - 1), lane);
#pragma unroll
            for (int r = 0; r < R; ++r) {
                const double *wr = lds.wts(r) + l0;
#pragma unroll
                for (int u = 0; u < 8; u += 2) {
                    const double2 pw = *reinterpret_cast<const double2 *>(wr + u);
                    if (SUB)
                        out[r] = fma(pw.y, x[r] - vj[u + 1], fma(pw.x, x[r] - vj[u], out[r]));
                    else
                        out[r] = fma(pw.y, vj[u + 1], fma(pw.x, vj[u], out[r]));
                }
            }
        }
    }
    __builtin_amdgcn_wave_barrier();
}

// Per-shape tuning, measured: the 32-view shape (6 slots, 2 rows) runs faster with
// three workgroups per CU (168 VGPRs); 17+ slots run faster with fewer channel
// loads unrolled (fewer registers held by loads in flight).
template <int CPL, int R>
constexpr int kMinBlocks = (CPL == 6 && R == 2) ? 3 : 1;
template <int CPL>
constexpr int kUnroll = CPL >= 17 ? 2 : 4;

// acc[r][c] = sum_d T[d][jc[c]] * x_r[d] over the 64 channels of a channel-major
// pooled tensor T (lane <-> key block), in ascending d with the same fused
// multiply-adds whichever loop order is used. SUB: sum_d (y_r[d] - T[d][jc[c]]) x_r[d].
// Few slots and rows: channels outermost, so the loads of every slot are in flight
// together; otherwise slots outermost (fewer registers held by loads; measured:
// the channel-outer order costs the 4-slot, 4-row shape its second wave per SIMD).
template <int CPL, int R, bool SUB>
__device__ __forceinline__ void column_dots(const double *__restrict__ T, const int (&jc)[CPL], int nkb,
                                            double *const (&x)[R], double *const (&y)[R], double (&acc)[R][CPL])
{
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
        for (int c = 0; c < CPL; ++c) acc[r][c] = 0.0;
    // Buffer loads: a per-lane 32-bit byte offset (the key block) and a wave-uniform
    // one (the channel row), range-checked by the hardware against the head's tensor.
    const __amdgpu_buffer_rsrc_t rs = pooled_rsrc(T, nkb);
    unsigned off[CPL];
#pragma unroll
    for (int c = 0; c < CPL; ++c) off[c] = (unsigned)jc[c] * (unsigned)sizeof(double);
    const int stride = nkb * (int)sizeof(double);
    auto at = [&](int d, int c) __attribute__((always_inline)) {
        return __builtin_bit_cast(double, __builtin_amdgcn_raw_buffer_load_b64(rs, off[c], d * stride, 0));
    };
    if constexpr (CPL <= 8 && CPL * R <= 12) {
#pragma unroll 1
        for (int d = 0; d < kD; d += 2) {
            double t0[CPL], t1[CPL];
#pragma unroll
            for (int c = 0; c < CPL; ++c) {
                t0[c] = at(d, c);
                t1[c] = at(d + 1, c);
            }
#pragma unroll
            for (int r = 0; r < R; ++r) {
                const double2 xd = *reinterpret_cast<const double2 *>(x[r] + d);
                double2 yd = {0.0, 0.0};
                if (SUB) yd = *reinterpret_cast<const double2 *>(y[r] + d);
#pragma unroll
                for (int c = 0; c < CPL; ++c) {
                    if (SUB)
                        acc[r][c] = fma(yd.y - t1[c], xd.y, fma(yd.x - t0[c], xd.x, acc[r][c]));
                    else
                        acc[r][c] = fma(xd.y, t1[c], fma(xd.x, t0[c], acc[r][c]));
                }
            }
        }
    } else {
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
#pragma unroll kUnroll<CPL>
            for (int d = 0; d < kD; d += 2) {
                const double t0 = at(d, c), t1 = at(d + 1, c);
#pragma unroll
                for (int r = 0; r < R; ++r) {
                    const double2 xd = *reinterpret_cast<const double2 *>(x[r] + d);
                    if (SUB) {
                        const double2 yd = *reinterpret_cast<const double2 *>(y[r] + d);
                        acc[r][c] = fma(yd.y - t1, xd.y, fma(yd.x - t0, xd.x, acc[r][c]));
                    } else {
                        acc[r][c] = fma(xd.y, t1, fma(xd.x, t0, acc[r][c]));
                    }
                }
            }
        }
    }
}

template <int CPL, int R, bool CDF>
__global__ void __launch_bounds__(kThreads, (kMinBlocks<CPL, R>)) select_kernel(const SelectParams p)
{
    __shared__ __align__(16) double smem[kWaves * WaveLds<R>::kDoubles];
    __shared__ float Ms[kD * (kD + 1)];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const unsigned long long lane_bit = 1ull << lane, lane_lt = lane_bit - 1ull;
    // Workgroups are numbered so that each of the 8 XCDs gets a contiguous range
    // of (head, row group) items: the rows of a head share one XCD's L2.
    const int groups = (p.n_qb + kWaves * R - 1) / (kWaves * R);
    const int item = (blockIdx.x & 7) * p.items_per_xcd + (blockIdx.x >> 3);
    if (item >= p.H * groups) return;
    const int h = item / groups;
    const int row0 = (item % groups) * kWaves * R + wave * R;
    {
        const float *Mh = p.gram + (size_t)h * kD * kD;
        for (int e = tid; e < kD * kD; e += kThreads) Ms[(e >> 6) * (kD + 1) + (e & 63)] = Mh[e];
    }
    __syncthreads();
    if (row0 >= p.n_qb) return;  // waves are independent from here on
    const WaveLds<R> lds{smem + wave * WaveLds<R>::kDoubles};

    const int nkb = p.n_kb, nqb = p.n_qb;
    const double eps = p.eps;
    const double *Kt = p.pooled.kbarT + (size_t)h * kD * nkb;
    const double *Vr = p.pooled.vbar + (size_t)h * nkb * kD;
    const double *Vt = p.pooled.vbarT + (size_t)h * kD * nkb;
    const double *cT = p.pooled.cT + (size_t)h * nkb;
    const int c_h = p.budgets[h];
    const int n_p = p.first_forced;  // candidates are the key blocks j < first_forced

    int irow[R];
    bool live[R], dense[R];
    double *vbv[R], *wvv[R], *gv[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        live[r] = row0 + r < nqb;
        irow[r] = live[r] ? row0 + r : nqb - 1;
        dense[r] = irow[r] >= p.first_dense_qb || c_h >= n_p;
        vbv[r] = lds.vec(0, r);
        wvv[r] = lds.vec(1, r);
        gv[r] = lds.vec(2, r);
        vbv[r][lane] = p.pooled.qbar[((size_t)h * nqb + irow[r]) * kD + lane];  // Qbar_i for now
    }
    int jc[CPL];  // this lane's key block per slot, clamped into range for loads
    bool valid[CPL];
    unsigned long long memb[CPL];  // wave masks of candidate lanes per slot
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
        const int j = lane + 64 * c;
        valid[c] = j < nkb;
        jc[c] = valid[c] ? j : nkb - 1;
        memb[c] = __ballot(j < n_p);
    }
    __builtin_amdgcn_wave_barrier();

    // Pooled logits Qbar_i . Kbar_j / sqrt(D) (Eq. 1).
    double acc[R][CPL], P[R][CPL], S2[R][CPL];
    column_dots<CPL, R, false>(Kt, jc, nkb, vbv, vbv, acc);
    // Softmax over all key blocks.
#pragma unroll
    for (int r = 0; r < R; ++r) {
        double mx = -INFINITY;
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
            acc[r][c] *= 0.125;  // 1/sqrt(64)
            if (valid[c]) mx = fmax(mx, acc[r][c]);
        }
        mx = wave_max(mx);
        double z = 0.0;
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
            P[r][c] = valid[c] ? exp(acc[r][c] - mx) : 0.0;
            z += P[r][c];
        }
        z = wave_sum(z);
#pragma unroll
        for (int c = 0; c < CPL; ++c) P[r][c] = P[r][c] / z;
        if (p.prob_out && live[r]) {
            double *po = p.prob_out + ((size_t)h * nqb + irow[r]) * nkb;
#pragma unroll
            for (int c = 0; c < CPL; ++c)
                if (valid[c]) po[lane + 64 * c] = P[r][c];
        }
    }

    // Dense pooled output vbar_i = sum_j P_ij Vbar_j, w_i = S vbar_i with S the
    // symmetric part of M (lane <-> channel), and vbar_i^T S vbar_i.
    double vsv[R];
    {
        double vb[R], wv[R];
        block_pass<CPL, R, false>(lds, P, vb, Vr, nkb, lane, vb);
#pragma unroll
        for (int r = 0; r < R; ++r) vbv[r][lane] = vb[r];
        __builtin_amdgcn_wave_barrier();
        mat_vec<R, true>(Ms, vbv, wv, lane);
#pragma unroll
        for (int r = 0; r < R; ++r) {
            wvv[r][lane] = wv[r];
            vsv[r] = wave_sum(vb[r] * wv[r]);
        }
        __builtin_amdgcn_wave_barrier();
    }

    // q_ij = e^T M e with e = vbar_i - Vbar_j (Eq. 9), expanded through the symmetric
    // part S of M (same quadratic form): q = vbar_i^T S vbar_i - 2 Vbar_j . w_i +
    // Vbar_j^T M Vbar_j, the last term per block from the pooling pass; one column of
    // Vbar per candidate. s_ij = P_ij sqrt(q_ij), key_ij = s_ij / max(1 - P_ij, eps)
    // (Eqs. 6-7).
    column_dots<CPL, R, false>(Vt, jc, nkb, wvv, wvv, acc);
#pragma unroll
    for (int r = 0; r < R; ++r) {
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
            const double q = fma(-2.0, acc[r][c], vsv[r] + cT[jc[c]]);
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
                if (valid[c]) ko[j] = j < n_p ? acc[r][c] : -1.0;
            }
        }
    }

    // Initial selection (Eq. 7), then the state of each drop set (Eqs. 10-12):
    // g = sum_{j in D} P_j (vbar - Vbar_j), K = 1 - sum_{j in D} P_j, G = g^T M g.
    // The criterion picks the ranking: the key (drift), P (probability) or the
    // negated key (drift maximisation from the start). A CDF cap (probability
    // only) shrinks the row's kept count to the shortest descending-P prefix
    // whose mass, forced blocks included, reaches cdf_tau.
    const int crit = p.criterion;
    const bool maximise = crit == RESS_CRITERION_DRIFT_MAX_SWAP || crit == RESS_CRITERION_DRIFT_MAX_FULL;
    unsigned long long inD[R], best[R];
    double K[R], G[R], J[R], J0[R], Jb[R];
    int crow[R];  // kept candidates of the row
#pragma unroll
    for (int r = 0; r < R; ++r) {
        inD[r] = 0ull;
        crow[r] = c_h;
        if (!dense[r]) {
            unsigned long long ko[CPL];
#pragma unroll
            for (int c = 0; c < CPL; ++c)
                ko[c] = order_key(crit == RESS_CRITERION_PROBABILITY ? P[r][c]
                                  : crit == RESS_CRITERION_DRIFT_MAX_FULL ? -acc[r][c] : acc[r][c]);
            if (CDF && crit == RESS_CRITERION_PROBABILITY && p.cdf_tau > 0.0) {
                // mass(n) = forced mass + the n largest candidate P: smallest n <= c_h
                // with mass(n) >= tau by bisection (mass is non-decreasing in n).
                double fm = 0.0;
#pragma unroll
                for (int c = 0; c < CPL; ++c) {
                    const int j = lane + 64 * c;
                    if (valid[c] && j >= n_p) fm += P[r][c];
                }
                fm = wave_sum(fm);
                auto mass = [&](int n) {
                    const unsigned long long sel = topk_slots<CPL>(ko, memb, n, lane_bit, lane_lt);
                    double m = 0.0;
#pragma unroll
                    for (int c = 0; c < CPL; ++c)
                        if ((sel >> c) & 1ull) m += P[r][c];
                    return fm + wave_sum(m);
                };
                int lo = 0, hi = c_h;
                if (mass(hi) >= p.cdf_tau) {
                    while (lo < hi) {
                        const int mid = (lo + hi) >> 1;
                        if (mass(mid) >= p.cdf_tau)
                            hi = mid;
                        else
                            lo = mid + 1;
                    }
                    const int floor2 = max(0, 2 - (nkb - n_p));
                    crow[r] = max(lo, min(floor2, n_p));
                }
            }
            const unsigned long long keep = topk_slots<CPL>(ko, memb, crow[r], lane_bit, lane_lt);
#pragma unroll
            for (int c = 0; c < CPL; ++c)
                if ((memb[c] & lane_bit) && !((keep >> c) & 1ull)) inD[r] |= 1ull << c;
        }
        double mass = 0.0;
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
            acc[r][c] = ((inD[r] >> c) & 1ull) ? P[r][c] : 0.0;  // weights of the g pass
            mass += acc[r][c];
        }
        K[r] = 1.0 - wave_sum(mass);
    }
    {
        double vb[R], g[R];
#pragma unroll
        for (int r = 0; r < R; ++r) vb[r] = vbv[r][lane];
        block_pass<CPL, R, true>(lds, acc, vb, Vr, nkb, lane, g);
#pragma unroll
        for (int r = 0; r < R; ++r) gv[r][lane] = g[r];
    }
    double *hv[R];  // M g reuses the slot of M vbar
#pragma unroll
    for (int r = 0; r < R; ++r) hv[r] = wvv[r];
    auto objective = [&]() {  // h = M g, G = g . h, J = G / max(K, eps)^2
        __builtin_amdgcn_wave_barrier();
        double hh[R];
        mat_vec<R, false>(Ms, gv, hh, lane);
#pragma unroll
        for (int r = 0; r < R; ++r) {
            hv[r][lane] = hh[r];
            G[r] = wave_sum(gv[r][lane] * hh[r]);
            const double Kh = K[r] > eps ? K[r] : eps;
            J[r] = G[r] / (Kh * Kh);
        }
        __builtin_amdgcn_wave_barrier();
    };
    objective();
#pragma unroll
    for (int r = 0; r < R; ++r) {
        J0[r] = Jb[r] = J[r];
        best[r] = inD[r];
    }

    // Budget-neutral restoration rounds (Eqs. 13-17) with track-best. The swap
    // count follows each row's kept count; rows whose count reached 0 are done.
    const __amdgpu_buffer_rsrc_t rsV = pooled_rsrc(Vr, nkb);
    double *swap_w = lds.swap_w();
    int *swap_j = lds.swap_j();
    for (int rr = 0; rr < p.rounds; ++rr) {
        int mrow[R], mmax = 0;
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int m = swaps_of_round(crow[r], p.rho, rr, p.swap_floor);
            mrow[r] = dense[r] ? 0 : min(m, min(n_p - crow[r], crow[r]));
            mmax = max(mmax, mrow[r]);
        }
        if (mmax <= 0) break;
        // e_k . (M g) for every candidate k of every row.
        column_dots<CPL, R, true>(Vt, jc, nkb, hv, vbv, acc);
        // Gains of every single restore / drop at the round-start state; the m best
        // of each kind are applied together, g and K following Eq. 13.
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int m = mrow[r];
            if (m <= 0) continue;
            unsigned long long dj[CPL], memD[CPL], memS[CPL];
#pragma unroll
            for (int c = 0; c < CPL; ++c) {
                const bool in = (inD[r] >> c) & 1ull;
                const double dkMg = P[r][c] * acc[r][c];
                const double dG = in ? -2.0 * dkMg + S2[r][c] : 2.0 * dkMg + S2[r][c];  // Eqs. 14-15
                const double Kn = K[r] + (in ? P[r][c] : -P[r][c]);
                const double Knh = Kn > eps ? Kn : eps;
                const double dJ = J[r] - (G[r] + dG) / (Knh * Knh);  // Eq. 16
                dj[c] = order_key(maximise ? -dJ : dJ);
                memD[c] = __ballot(in);
                memS[c] = memb[c] & ~memD[c];
            }
            const unsigned long long rest = topk_slots<CPL>(dj, memD, m, lane_bit, lane_lt);
            const unsigned long long drop = topk_slots<CPL>(dj, memS, m, lane_bit, lane_lt);
            inD[r] = (inD[r] & ~rest) | drop;
            double mr = 0.0, md = 0.0;
            double g = gv[r][lane];
            const double vbl = vbv[r][lane];
            // The swapped blocks of all slots, in slot order, are gathered into one list
            // (up to 64 entries) and applied 8 rows of Vbar at a time: restores
            // subtract d_k, drops add it. The list is padded to a multiple of 8 with
            // zero-weight entries of block 0, which leave g unchanged.
            int nbuf = 0;
            auto apply = [&]() __attribute__((always_inline)) {
                const int nr = (nbuf + 7) & ~7;
                if (lane < nr - nbuf) {
                    swap_j[nbuf + lane] = 0;
                    swap_w[nbuf + lane] = 0.0;
                }
                __builtin_amdgcn_wave_barrier();
                for (int t0 = 0; t0 < nr; t0 += 8) {
                    const int4 ja = *reinterpret_cast<const int4 *>(swap_j + t0);
                    const int4 jb = *reinterpret_cast<const int4 *>(swap_j + t0 + 4);
                    const int js[8] = {ja.x, ja.y, ja.z, ja.w, jb.x, jb.y, jb.z, jb.w};
                    double vj[8];
#pragma unroll
                    for (int u = 0; u < 8; ++u)
                        vj[u] = pooled_row(rsV, js[u], lane);
#pragma unroll
                    for (int u = 0; u < 8; u += 2) {
                        const double2 w = *reinterpret_cast<const double2 *>(swap_w + t0 + u);
                        g = fma(w.x, vbl - vj[u], g);
                        g = fma(w.y, vbl - vj[u + 1], g);
                    }
                }
                __builtin_amdgcn_wave_barrier();
                nbuf = 0;
            };
#pragma unroll
            for (int c = 0; c < CPL; ++c) {
                const bool is_rest = (rest >> c) & 1ull, is_drop = (drop >> c) & 1ull;
                const unsigned long long sm = __ballot(is_rest || is_drop);
                if (sm == 0ull) continue;
                const int n = __popcll(sm);
                if (nbuf + n > 64) apply();
                if (is_rest || is_drop) {
                    const int pos = nbuf + __popcll(sm & lane_lt);
                    swap_j[pos] = lane + 64 * c;
                    swap_w[pos] = is_drop ? P[r][c] : -P[r][c];
                }
                if (is_rest) mr += P[r][c];
                if (is_drop) md += P[r][c];
                nbuf += n;
            }
            if (nbuf > 0) apply();
            K[r] = (K[r] + wave_sum(mr)) - wave_sum(md);
            __builtin_amdgcn_wave_barrier();
            gv[r][lane] = g;
        }
        objective();
#pragma unroll
        for (int r = 0; r < R; ++r)
            if (!dense[r] && (maximise ? J[r] > Jb[r] : J[r] < Jb[r])) {
                Jb[r] = J[r];
                best[r] = inD[r];
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
            const bool kept = valid[c] && !((best[r] >> c) & 1ull);
            const unsigned long long km = __ballot(kept);
            if (kept) out[before + __popcll(km & lane_lt)] = lane + 64 * c;
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
    SelectParams q = p;
    const int groups = (p.n_qb + kWaves * R - 1) / (kWaves * R);
    q.items_per_xcd = (p.H * groups + 7) / 8;
    if (p.cdf_tau > 0.0)  // the CDF cap has its own instantiation (it adds registers)
        hipLaunchKernelGGL((select_kernel<CPL, R, true>), dim3((unsigned)(8 * q.items_per_xcd)), dim3(kThreads), 0, s, q);
    else
        hipLaunchKernelGGL((select_kernel<CPL, R, false>), dim3((unsigned)(8 * q.items_per_xcd)), dim3(kThreads), 0, s, q);
    return hipGetLastError();
}

// Rows per wave: the most rows, up to RMAX, that still give each of the chip's
// 256 compute units a workgroup. Measured: sharing every pooled-tensor load among
// more rows pays only while the grid fills the chip (8 views, 86 blocks: 4 rows
// per wave 0.20 ms, 1 row 0.12 ms; 16 views, 172 blocks: 4 rows 0.39 ms, 2 rows
// 0.22 ms; 32 views, 344 blocks: 2 rows 0.48 ms, 1 row 0.70 ms).
constexpr long long kCUs = 256;
template <int CPL, int RMAX>
hipError_t launch_rows(const SelectParams &p, hipStream_t s)
{
    auto workgroups = [&](int r) { return (long long)p.H * ((p.n_qb + kWaves * r - 1) / (kWaves * r)); };
    if constexpr (RMAX >= 4)
        if (workgroups(4) >= kCUs) return launch_cfg<CPL, 4>(p, s);
    if constexpr (RMAX >= 2)
        if (workgroups(2) >= kCUs) return launch_cfg<CPL, 2>(p, s);
    return launch_cfg<CPL, 1>(p, s);
}

}  // namespace

hipError_t launch_select(const SelectParams &p, hipStream_t s)
{
    if (p.H == 0 || p.n_qb == 0) return hipSuccess;
    const int n = p.n_kb;
    if (n <= 64) return launch_rows<1, 4>(p, s);
    if (n <= 128) return launch_rows<2, 4>(p, s);
    if (n <= 256) return launch_rows<4, 4>(p, s);
    if (n <= 384) return launch_rows<6, 2>(p, s);
    if (n <= 512) return launch_cfg<8, 1>(p, s);
    if (n <= 768) return launch_cfg<12, 1>(p, s);
    if (n <= 1088) return launch_cfg<17, 1>(p, s);
    if (n <= 1536) return launch_cfg<24, 1>(p, s);
    if (n <= 2048) return launch_cfg<32, 1>(p, s);
    if (n <= 3072) return launch_cfg<48, 1>(p, s);
    return launch_cfg<64, 1>(p, s);
}

}  // namespace ress
