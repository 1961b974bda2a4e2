// Drift-based block selection (Secs. 4.2-4.3), one launch for every row of a
// layer: pooled map, drift scores, exact top-c, R budget-neutral restoration
// rounds with track-best, and compaction of the kept-block lists.
//
// Work layout. A workgroup of NW waves owns NW x R query blocks ("rows") of one
// head; each wave owns R of them.
//  - Per-candidate quantities live "lane <-> key block": lane l, slot c holds key
//    block j = l + 64 c (CPL slots). Per-row vectors (Qbar, vbar, S vbar with S
//    the symmetric part of M, g, M g) live in the wave's LDS area, channel d at
//    index d.
//  - The contractions are float64 matrix products of the workgroup's rows
//    (padded to a multiple of 16) with the head's row-major pooled tensors, on
//    the matrix cores (16x16x4 float64 steps): over channels, the pooled logits
//    against Kbar and the drift scores (expanded as in Eq. 9; a row's block with
//    P > 1/2 gets e^T M e directly) and every round's gains against Vbar;
//    over key blocks, the dense pooled output vbar and the net drift g against
//    Vbar. The pooled tensor goes from L2 straight into the B operands (each lane
//    reads 16 contiguous bytes or more of one key block); the A operands are the
//    rows' LDS vectors, or their weights staged in LDS; result tiles pass through
//    the LDS staging area into the layout of the owning wave. Each output element
//    is one chain of matrix steps in a fixed order: reruns are bit-identical.
//  - Every top-k is exact: a bitwise search for the k-th largest of
//    order-preserving 64-bit keys, using wave ballots and popcounts, ties broken
//    by the lower block index. No atomics and no data-dependent reduction order.
// All arithmetic is float64 (the discrete decisions stay stable).
#include <math.h>

#include "ress_internal.h"

namespace ress {
namespace {

typedef double v4d __attribute__((ext_vector_type(4)));
typedef unsigned int v4u __attribute__((ext_vector_type(4)));

// Word 3 of a raw buffer descriptor on gfx9-family chips (32-bit data format,
// no swizzle, no index stride): loads past num_records bytes return zero.
constexpr int kBufWord3 = 0x00020000;

// Buffer descriptor over one head's row-major pooled tensor (nkb x 64 doubles).
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

// 16 bytes at byte offset `off` of a pooled tensor (zero past its end).
__device__ __forceinline__ double2 pooled_16(__amdgpu_buffer_rsrc_t rs, int off)
{
    return __builtin_bit_cast(double2, __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0));
}

// Wave reductions on registers only (no LDS permutes): DPP exchanges within 16
// lanes (lane i with i^1, i^2, then with 7-i within 8 and 15-i within 16, each
// step adding a symmetric pair, so every lane holds the same partial), then the
// gfx950 row swaps, whose two results added give x[l] + x[l^16] and
// x[l] + x[l^32] in every lane. Commutative adds in a fixed pattern: the result
// is identical in every lane and on every run.
template <int CTRL>
__device__ __forceinline__ double dpp_f64(double x)
{
    const unsigned long long u = (unsigned long long)__double_as_longlong(x);
    const int lo = __builtin_amdgcn_mov_dpp((int)(unsigned)u, CTRL, 0xf, 0xf, false);
    const int hi = __builtin_amdgcn_mov_dpp((int)(unsigned)(u >> 32), CTRL, 0xf, 0xf, false);
    return __longlong_as_double((long long)(((unsigned long long)(unsigned)hi << 32) | (unsigned)lo));
}

// Lane l's value and that of lane l^16 (ROW32: l^32), in an order that is the
// same for both lanes of the pair.
template <bool ROW32>
__device__ __forceinline__ void swap_pair(double x, double &d0, double &d1)
{
    const unsigned long long u = (unsigned long long)__double_as_longlong(x);
    const unsigned lo = (unsigned)u, hi = (unsigned)(u >> 32);
    const auto a = ROW32 ? __builtin_amdgcn_permlane32_swap(lo, lo, false, false)
                         : __builtin_amdgcn_permlane16_swap(lo, lo, false, false);
    const auto b = ROW32 ? __builtin_amdgcn_permlane32_swap(hi, hi, false, false)
                         : __builtin_amdgcn_permlane16_swap(hi, hi, false, false);
    d0 = __longlong_as_double((long long)(((unsigned long long)b[0] << 32) | a[0]));
    d1 = __longlong_as_double((long long)(((unsigned long long)b[1] << 32) | a[1]));
}

template <bool ROW32>
__device__ __forceinline__ double swap_sum(double x)
{
    double d0, d1;
    swap_pair<ROW32>(x, d0, d1);
    return d0 + d1;
}

__device__ __forceinline__ double wave_sum(double x)
{
    x += dpp_f64<0xB1>(x);   // quad_perm [1,0,3,2]: lane i^1
    x += dpp_f64<0x4E>(x);   // quad_perm [2,3,0,1]: lane i^2
    x += dpp_f64<0x141>(x);  // row_half_mirror: lane 7-i within 8
    x += dpp_f64<0x140>(x);  // row_mirror: lane 15-i within 16
    x = swap_sum<false>(x);  // + the partner 16-lane row
    return swap_sum<true>(x);  // + the other 32 lanes
}

// Two wave sums with their exchanges interleaved.
__device__ __forceinline__ void wave_sum2(double a, double b, double &sa, double &sb)
{
    a += dpp_f64<0xB1>(a);
    b += dpp_f64<0xB1>(b);
    a += dpp_f64<0x4E>(a);
    b += dpp_f64<0x4E>(b);
    a += dpp_f64<0x141>(a);
    b += dpp_f64<0x141>(b);
    a += dpp_f64<0x140>(a);
    b += dpp_f64<0x140>(b);
    a = swap_sum<false>(a);
    b = swap_sum<false>(b);
    sa = swap_sum<true>(a);
    sb = swap_sum<true>(b);
}

template <int CTRL>
__device__ __forceinline__ unsigned long long dpp_u64(unsigned long long u)
{
    const int lo = __builtin_amdgcn_mov_dpp((int)(unsigned)u, CTRL, 0xf, 0xf, false);
    const int hi = __builtin_amdgcn_mov_dpp((int)(unsigned)(u >> 32), CTRL, 0xf, 0xf, false);
    return ((unsigned long long)(unsigned)hi << 32) | (unsigned)lo;
}

template <bool ROW32>
__device__ __forceinline__ unsigned long long swap_max_u64(unsigned long long u)
{
    const unsigned lo = (unsigned)u, hi = (unsigned)(u >> 32);
    const auto a = ROW32 ? __builtin_amdgcn_permlane32_swap(lo, lo, false, false)
                         : __builtin_amdgcn_permlane16_swap(lo, lo, false, false);
    const auto b = ROW32 ? __builtin_amdgcn_permlane32_swap(hi, hi, false, false)
                         : __builtin_amdgcn_permlane16_swap(hi, hi, false, false);
    const unsigned long long d0 = ((unsigned long long)b[0] << 32) | a[0];
    const unsigned long long d1 = ((unsigned long long)b[1] << 32) | a[1];
    return d0 > d1 ? d0 : d1;
}

// Largest 64-bit unsigned value over the wave, in every lane.
__device__ __forceinline__ unsigned long long wave_max_u64(unsigned long long x)
{
    unsigned long long y = dpp_u64<0xB1>(x);
    x = y > x ? y : x;
    y = dpp_u64<0x4E>(x);
    x = y > x ? y : x;
    y = dpp_u64<0x141>(x);
    x = y > x ? y : x;
    y = dpp_u64<0x140>(x);
    x = y > x ? y : x;
    return swap_max_u64<true>(swap_max_u64<false>(x));
}

__device__ __forceinline__ double wave_max(double x)
{
    x = fmax(x, dpp_f64<0xB1>(x));
    x = fmax(x, dpp_f64<0x4E>(x));
    x = fmax(x, dpp_f64<0x141>(x));
    x = fmax(x, dpp_f64<0x140>(x));
    double d0, d1;
    swap_pair<false>(x, d0, d1);
    x = fmax(d0, d1);
    swap_pair<true>(x, d0, d1);
    return fmax(d0, d1);
}

__device__ __forceinline__ v4d mfma_f64(double a, double b, v4d c)
{
    return __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, c, 0, 0, 0);
}

// Order-preserving map of a double to uint64 (larger value -> larger key);
// -0 is folded onto +0 so that equal values get equal keys.
__device__ __forceinline__ unsigned long long order_key(double x)
{
    const unsigned long long u = (unsigned long long)__double_as_longlong(x + 0.0);
    return (u >> 63) ? ~u : (u | 0x8000000000000000ull);
}

// Bitwise search over member high words h[0..NS) (zero for non-members): the
// largest t such that at least k of them reach t with a zero low word below it,
// built bit by bit; found = exactly k reach it. The threshold, bit and counts are
// wave-uniform and the loop has a single exit, so that it runs on scalar
// registers and scalar branches.
template <int NS>
__device__ __forceinline__ unsigned int search_high(const unsigned int (&h)[NS], int k, int &found)
{
    unsigned int thi = 0, bit = 0x80000000u;
    do {
        const unsigned int cand = __builtin_amdgcn_readfirstlane(thi | bit);
        unsigned long long bl[NS];
#pragma unroll
        for (int c = 0; c < NS; ++c) bl[c] = __ballot(h[c] >= cand);
        int cnt = 0;
#pragma unroll
        for (int c = 0; c < NS; ++c) cnt += __popcll(bl[c]);
        thi = cnt >= k ? cand : thi;
        found = cnt == k;
        bit >>= 1;
    } while (!found && bit != 0u);
    return thi;
}

// The member high words packed into the first NS slots (zero past them) through
// the wave's scratch scr (this wave's LDS only), when at most 64 NS are members.
template <int CPL, int NS>
__device__ __forceinline__ void pack_high(const unsigned int (&hi)[CPL], unsigned long long mbits, int nmem,
                                          unsigned int *scr, unsigned long long lane_lt, int lane,
                                          unsigned int (&h)[NS])
{
    int base = 0;
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
        const bool m = (mbits >> c) & 1ull;
        const unsigned long long bl = __ballot(m);
        if (m) scr[base + __popcll(bl & lane_lt)] = hi[c];
        base += __popcll(bl);
    }
    __builtin_amdgcn_wave_barrier();
#pragma unroll
    for (int c = 0; c < NS; ++c) h[c] = 64 * c + lane < nmem ? scr[64 * c + lane] : 0u;
    __builtin_amdgcn_wave_barrier();
}

// Exact top-k of the member slots by (key desc, block index asc). Bit c of
// mbits marks this lane's slot c as a member. Non-member keys are replaced by 0,
// below every member key (an order key of a finite value is at least 1), so one
// ballot per slot counts members only. The k-th largest key is found bit by
// bit, high word first (search_high); when the members fit 2 or 4 slots and a
// scratch is given, that search runs on them packed (same threshold, fewer
// compares). Once the high word t of the k-th largest key is known, a key
// reaches a candidate (t, x) (x >= 1) exactly when the 32-bit value "all ones if
// its high word is above t, its low word if equal, zero if below" reaches x. The
// search stops as soon as exactly k keys reach the threshold. Returns this
// lane's chosen slots as a bit mask. Requires 0 <= k <= number of members.
template <int CPL>
__device__ __forceinline__ unsigned long long topk_slots(const unsigned long long (&key)[CPL],
                                                         unsigned long long mbits, int k, unsigned long long lane_lt,
                                                         unsigned int *scr = nullptr, int lane = 0)
{
    k = __builtin_amdgcn_readfirstlane(k);
    if (k <= 0) return 0ull;
    unsigned int hi[CPL], lo[CPL];
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
        const unsigned long long km = ((mbits >> c) & 1ull) ? key[c] : 0ull;
        hi[c] = (unsigned int)(km >> 32);
        lo[c] = (unsigned int)km;
    }
    int found = 0;
    unsigned int thi;
    int nmem = 64 * CPL;
    if (scr != nullptr && CPL > 2) {
        nmem = 0;
#pragma unroll
        for (int c = 0; c < CPL; ++c) nmem += __popcll(__ballot((mbits >> c) & 1ull));
    }
    if (CPL > 2 && nmem <= 128) {
        unsigned int h[2];
        pack_high<CPL, 2>(hi, mbits, nmem, scr, lane_lt, lane, h);
        thi = search_high<2>(h, k, found);
    } else if (CPL > 4 && nmem <= 256) {
        unsigned int h[4];
        pack_high<CPL, 4>(hi, mbits, nmem, scr, lane_lt, lane, h);
        thi = search_high<4>(h, k, found);
    } else {
        thi = search_high<CPL>(hi, k, found);
    }
    if (found) {  // exactly k keys reach (thi, 0): they are the top k
        unsigned long long chosen = 0;
#pragma unroll
        for (int c = 0; c < CPL; ++c)
            if (hi[c] >= thi) chosen |= 1ull << c;
        return chosen;
    }
    // Low word, against the high word thi of the k-th largest key.
    unsigned int l2[CPL];
#pragma unroll
    for (int c = 0; c < CPL; ++c) l2[c] = hi[c] > thi ? 0xffffffffu : (hi[c] == thi ? lo[c] : 0u);
    unsigned int tlo = 0, bit = 0x80000000u;
    do {
        const unsigned int cand = __builtin_amdgcn_readfirstlane(tlo | bit);
        unsigned long long bl[CPL];
#pragma unroll
        for (int c = 0; c < CPL; ++c) bl[c] = __ballot(l2[c] >= cand);
        int cnt = 0;
#pragma unroll
        for (int c = 0; c < CPL; ++c) cnt += __popcll(bl[c]);
        tlo = cnt >= k ? cand : tlo;
        found = cnt == k;
        bit >>= 1;
    } while (!found && bit != 0u);
    if (found) {
        unsigned long long chosen = 0;
#pragma unroll
        for (int c = 0; c < CPL; ++c)
            if (l2[c] >= tlo) chosen |= 1ull << c;
        return chosen;
    }
    // thr is the k-th largest key and is tied: take all larger keys and the
    // lowest-index ties.
    const unsigned long long thr = ((unsigned long long)thi << 32) | tlo;
    unsigned long long km[CPL];
#pragma unroll
    for (int c = 0; c < CPL; ++c) km[c] = ((unsigned long long)hi[c] << 32) | lo[c];
    int gt = 0;
#pragma unroll
    for (int c = 0; c < CPL; ++c) gt += __popcll(__ballot(km[c] > thr));
    const int need = k - gt;
    int before = 0;
    unsigned long long chosen = 0;
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
        const bool tie = km[c] == thr;
        const unsigned long long tb = __ballot(tie);
        const int rank = before + __popcll(tb & lane_lt);
        if (km[c] > thr || (tie && rank < need)) chosen |= 1ull << c;
        before += __popcll(tb);
    }
    return chosen;
}

// The same selection as topk_slots for small k, by k extractions of the largest
// remaining member key: per lane the largest over its slots (lowest slot on
// ties), then over the wave (wave_max_u64), then the lowest block index among
// the slots holding that key (slots in ascending order, lanes in ascending
// order within a slot, which is ascending block index).
template <int CPL>
__device__ __forceinline__ unsigned long long topk_small(const unsigned long long (&key)[CPL],
                                                         unsigned long long mbits, int k, int lane)
{
    unsigned long long left = mbits, chosen = 0;
    for (int t = 0; t < k; ++t) {
        unsigned long long best = 0;
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
            const unsigned long long v = ((left >> c) & 1ull) ? key[c] : 0ull;
            best = v > best ? v : best;
        }
        best = wave_max_u64(best);
        // best > 0: at least one member is left (k <= members)
        bool done = false;
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
            const unsigned long long at = __ballot(((left >> c) & 1ull) && key[c] == best);
            if (!done && at != 0ull) {
                if (lane == __builtin_ctzll(at)) {
                    left &= ~(1ull << c);
                    chosen |= 1ull << c;
                }
                done = true;
            }
        }
    }
    return chosen;
}

// Top-k of the member slots: extraction for k up to 2, bitwise search beyond
// (measured: extraction costs more than the search from k = 5 on); scr as for
// topk_slots.
template <int CPL>
__device__ __forceinline__ unsigned long long topk_any(const unsigned long long (&key)[CPL],
                                                       unsigned long long mbits, int k, int lane,
                                                       unsigned long long lane_lt, unsigned int *scr)
{
    return k <= 2 ? topk_small<CPL>(key, mbits, k, lane) : topk_slots<CPL>(key, mbits, k, lane_lt, scr, lane);
}

// Swap count of round r (Eq. 17): max(floor, floor(rho c 2^-(r+1))).
__device__ __forceinline__ int swaps_of_round(int c, double rho, int r, int swap_floor)
{
    const int m = (int)floor(rho * (double)c * ldexp(1.0, -(r + 1)));
    return m > swap_floor ? m : swap_floor;
}

// Per-wave LDS area (doubles): vectors vec[slot][R][64] and a swap list of up to
// 64 (block, weight) pairs plus padding to a multiple of 8. Every part starts on
// a 16-byte boundary.
template <int R>
struct WaveLds {
    static constexpr int kVecs = 3;  // 0: Qbar then vbar, 1: S vbar then M g, 2: g
    static constexpr int kSwaps = 72;
    static constexpr int kDoubles = kVecs * R * kD + kSwaps + kSwaps / 2;
    static_assert(kDoubles % 2 == 0, "16-byte aligned wave areas");
    double *base;
    __device__ double *vec(int slot, int r) const { return base + (slot * R + r) * kD; }
    __device__ double *swap_w() const { return base + kVecs * R * kD; }
    __device__ int *swap_j() const { return reinterpret_cast<int *>(base + kVecs * R * kD + kSwaps); }
};

// Sizes of a workgroup configuration: RW rows in MT 16-row tiles; the LDS
// staging area holds 16 MT rows of CHK slots (64 key blocks each) plus 2 doubles
// of padding per row (so that rows start on different 16-byte bank groups), as
// many slots as the LDS left by the wave areas and M_h allows.
template <int CPL, int R, int NW>
struct SelCfg {
    static constexpr int RW = NW * R;
    static constexpr int MT = (RW + 15) / 16;
    static constexpr int WD = WaveLds<R>::kDoubles;
    static constexpr int FIXED = NW * WD * 8 + kD * (kD + 1) * 4 + 256;
    static constexpr int chk()
    {
        int c = CPL;
        while (c > 1 && FIXED + 16 * MT * (c * 512 + 16) > 163840) --c;
        return c;
    }
    static constexpr int CHK = chk();
    static constexpr int SROW = CHK * 64 + 2;          // doubles per staging row
    static constexpr int NCH = (CPL + CHK - 1) / CHK;  // chunks of slots
    // Key-block splits of the weighted sums: 2 MT KS items, one per wave; the KS
    // partial tiles of a row sit side by side in its staging row.
    static constexpr int KS = (NW / (2 * MT)) < CHK ? (NW / (2 * MT)) : CHK;
    static_assert(KS >= 1, "one weighted-sum item per wave at most");
    static_assert(4 * MT <= NW, "one mat-vec item per wave at most");
};

template <int CPL, int R, int NW>
__global__ void __launch_bounds__(NW * 64, 1) select_kernel(const SelectParams p)
{
    using Cfg = SelCfg<CPL, R, NW>;
    constexpr int RW = Cfg::RW, MT = Cfg::MT, CHK = Cfg::CHK, SROW = Cfg::SROW, NCH = Cfg::NCH, KS = Cfg::KS;
    __shared__ __align__(16) double stage[16 * MT * SROW];
    __shared__ __align__(16) double wareas[NW * Cfg::WD];
    __shared__ float Ms[kD * (kD + 1)];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const unsigned long long lane_lt = (1ull << lane) - 1ull;
    // Workgroups are numbered so that each of the 8 XCDs gets a contiguous range
    // of (head, row group) items: the rows of a head share one XCD's L2.
    const int groups = (p.n_qb + RW - 1) / RW;
    const int item = (blockIdx.x & 7) * p.items_per_xcd + (blockIdx.x >> 3);
    if (item >= p.H * groups) return;  // the whole workgroup
    const int h = item / groups;
    const int row0 = (item % groups) * RW + wave * R;
    const int nkb = p.n_kb, nqb = p.n_qb;
    const int ntiles = (nkb + 15) >> 4;
    const __amdgpu_buffer_rsrc_t rsK = pooled_rsrc(p.pooled.kbar + (size_t)h * nkb * kD, nkb);
    const __amdgpu_buffer_rsrc_t rsV = pooled_rsrc(p.pooled.vbar + (size_t)h * nkb * kD, nkb);
    {
        const float *Mh = p.gram + (size_t)h * kD * kD;
        for (int e = tid; e < kD * kD; e += NW * 64) Ms[(e >> 6) * (kD + 1) + (e & 63)] = Mh[e];
    }
    // Vector `slot` of the workgroup's row m (in the area of the wave owning it).
    auto row_vec = [&](int slot, int m) -> double * {
        return wareas + (m / R) * Cfg::WD + (slot * R + m % R) * kD;
    };
    const int grp = lane >> 4, col = lane & 15;  // matrix-step lane coordinates
    const WaveLds<R> lds{wareas + wave * Cfg::WD};

    // acc[r][c] = sum_d X_m[d] T_j[d] for this wave's rows m and key blocks
    // j = lane + 64 c, with X_m vector `xs` of row m and T the head's pooled tensor
    // behind rs. Tiles of 16 key blocks go round the waves; for tile t, lane l holds
    // channels 16 (l / 16) .. +15 of key block 16 t + l % 16 (in step s the k index
    // l / 16 stands for channel 16 (l / 16) + s, in A as in B) and the tile is
    // multiplied with every 16-row tile of the workgroup (rows past RW repeat the
    // last one; their results are not read). Results reach the owners through the
    // staging area, CHK slots at a time.
    auto dot_pass = [&](int xs, __amdgpu_buffer_rsrc_t rs, double (&acc)[R][CPL]) __attribute__((always_inline)) {
        const double *arow[MT];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) arow[mt] = row_vec(xs, min(16 * mt + col, RW - 1)) + 16 * grp;
#pragma unroll
        for (int q = 0; q < NCH; ++q) {
            const int t0 = 4 * CHK * q, t1 = min(4 * CHK * (q + 1), ntiles);
            // Tile t belongs to wave t mod NW (loads past the tensor give zero).
            auto load_b = [&](int t, double (&b)[16]) __attribute__((always_inline)) {
                const int off = (16 * t + col) * kD * (int)sizeof(double) + grp * 128;
#pragma unroll
                for (int u = 0; u < 8; ++u) {
                    const double2 v = pooled_16(rs, off + 16 * u);
                    b[2 * u] = v.x;
                    b[2 * u + 1] = v.y;
                }
            };
            for (int t = t0 + (wave - t0 % NW + NW) % NW; t < t1; t += NW) {
                double b[16];
                load_b(t, b);
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) {
                    v4d c = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
                    for (int u = 0; u < 8; ++u) {
                        const double2 a = *reinterpret_cast<const double2 *>(arow[mt] + 2 * u);
                        c = mfma_f64(a.x, b[2 * u], c);
                        c = mfma_f64(a.y, b[2 * u + 1], c);
                    }
                    // c[v] = C[16 mt + 4 v + l / 16][16 t + l % 16]
                    double *dst = stage + (16 * mt + grp) * SROW + (16 * t - 64 * CHK * q) + col;
#pragma unroll
                    for (int v = 0; v < 4; ++v) dst[4 * v * SROW] = c[v];
                }
            }
            __syncthreads();
#pragma unroll
            for (int c = 0; c < CPL; ++c)
                if (c / CHK == q)
#pragma unroll
                    for (int r = 0; r < R; ++r) acc[r][c] = stage[(wave * R + r) * SROW + (c - CHK * q) * 64 + lane];
            __syncthreads();
        }
    };
    // out_m[d] = sum_j w_m(j) Vbar_j[d] for every row m of the workgroup, into vector
    // `os` of row m, with w_m(j) = w[r][c] of the owning wave (zero for key blocks
    // past n_kb). The owners stage their weights CHK slots at a time. Item
    // (mt, np, ks) of wave mt 2 KS + np KS + ks accumulates the 16 rows of tile mt
    // against channels 32 np + 2 n + e (n < 16, e = 0, 1) over the key-block
    // octets o = ks (mod KS): in each step the k index l / 16 stands for key block
    // 8 o + 2 (l / 16) + (0 or 1), so one 16-byte read gives the A values of two
    // steps and one 16-byte read of a key block's channel pair the B values of two
    // products. The KS partial tiles are then added in split order by the owners.
    auto wsum_pass = [&](const double (&w)[R][CPL], int os) __attribute__((always_inline)) {
        const bool mine = wave < 2 * MT * KS;
        const int it = mine ? wave : 0;
        const int ks = it % KS, np = (it / KS) & 1, mt = it / (2 * KS);
        v4d c0 = {0.0, 0.0, 0.0, 0.0}, c1 = c0;
        const double *arow = stage + (16 * mt + col) * SROW + 2 * grp;
        const int boff = (32 * np + 2 * col) * (int)sizeof(double);
#pragma unroll
        for (int q = 0; q < NCH; ++q) {
#pragma unroll
            for (int c = 0; c < CPL; ++c)
                if (c / CHK == q)
#pragma unroll
                    for (int r = 0; r < R; ++r) stage[(wave * R + r) * SROW + (c - CHK * q) * 64 + lane] = w[r][c];
            __syncthreads();
            const int kq = min(64 * CHK, nkb - 64 * CHK * q);  // key blocks of the chunk
            if (mine && kq > 0) {
                const int noct = (kq + 7) >> 3;
                const int key0 = 64 * CHK * q + 2 * grp;
#pragma unroll 4
                for (int o = ks; o < noct; o += KS) {
                    const double2 a = *reinterpret_cast<const double2 *>(arow + 8 * o);
                    const int key = key0 + 8 * o;
                    const double2 b0 = pooled_16(rsV, key * kD * (int)sizeof(double) + boff);
                    const double2 b1 = pooled_16(rsV, (key + 1) * kD * (int)sizeof(double) + boff);
                    c0 = mfma_f64(a.x, b0.x, c0);
                    c1 = mfma_f64(a.x, b0.y, c1);
                    c0 = mfma_f64(a.y, b1.x, c0);
                    c1 = mfma_f64(a.y, b1.y, c1);
                }
            }
            __syncthreads();
        }
        // c_e[v] = partial of row 16 mt + 4 v + l / 16, channel 32 np + 2 (l % 16) + e
        if (mine) {
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                double *o = stage + (16 * mt + 4 * v + grp) * SROW + ks * kD + 32 * np + 2 * col;
                *reinterpret_cast<double2 *>(o) = double2{c0[v], c1[v]};
            }
        }
        __syncthreads();
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const double *src = stage + (wave * R + r) * SROW + lane;
            double tot = src[0];
#pragma unroll
            for (int k2 = 1; k2 < KS; ++k2) tot += src[k2 * kD];
            lds.vec(os, r)[lane] = tot;
        }
        __syncthreads();
    };

    // x_m = A y_m for every row m of the workgroup (y: vector `ys`, x: vector `xs`)
    // with A = M_h, or with SYM its symmetric part (M + M^T) / 2 (the same quadratic
    // form; exact in float64 from float32 entries). Item (mt, nt) of 4 MT, on
    // wave mt 4 + nt: the 16 rows of tile mt against output channels 16 nt .. +15,
    // k <-> channel 16 (l / 16) + s in step s as in dot_pass; B from M_h in LDS.
    // Ends with a workgroup barrier (the owners then read x).
    auto mv_pass = [&](auto sym, int ys, int xs) __attribute__((always_inline)) {
        constexpr bool SYM = decltype(sym)::value;
        if (wave < 4 * MT) {
            const int mt = wave >> 2, nt = wave & 3;
            const double *arow = row_vec(ys, min(16 * mt + col, RW - 1)) + 16 * grp;
            const int n = 16 * nt + col;
            v4d c = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const double2 a = *reinterpret_cast<const double2 *>(arow + 2 * u);
                const int k = 16 * grp + 2 * u;
                double b0 = (double)Ms[n * (kD + 1) + k], b1 = (double)Ms[n * (kD + 1) + k + 1];
                if (SYM) {
                    b0 = 0.5 * (b0 + (double)Ms[k * (kD + 1) + n]);
                    b1 = 0.5 * (b1 + (double)Ms[(k + 1) * (kD + 1) + n]);
                }
                c = mfma_f64(a.x, b0, c);
                c = mfma_f64(a.y, b1, c);
            }
            // c[v] = x[row 16 mt + 4 v + l / 16][channel n]
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int m = 16 * mt + 4 * v + grp;
                if (m < RW) row_vec(xs, m)[n] = c[v];
            }
        }
        __syncthreads();
    };
    using plain_mv = std::integral_constant<bool, false>;
    using sym_mv = std::integral_constant<bool, true>;

    const double eps = p.eps;
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
    int jc[CPL];  // this lane's key block per slot, clamped into range for reads
    bool valid[CPL];
    unsigned long long cand_bits = 0;  // bit c: slot c of this lane is a candidate
#pragma unroll
    for (int c = 0; c < CPL; ++c) {
        const int j = lane + 64 * c;
        valid[c] = j < nkb;
        jc[c] = valid[c] ? j : nkb - 1;
        if (j < n_p) cand_bits |= 1ull << c;
    }
    __syncthreads();  // M_h and every row's Qbar in place

    // Pooled logits Qbar_i . Kbar_j / sqrt(D) (Eq. 1).
    double acc[R][CPL], P[R][CPL], S2[R][CPL];
    dot_pass(0, rsK, acc);
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

    // Dense pooled output vbar_i = sum_j P_ij Vbar_j (over Qbar_i, no longer
    // needed), w_i = S vbar_i with S the symmetric part of M (lane <-> channel),
    // and vbar_i^T S vbar_i.
    double vsv[R];
    {
        wsum_pass(P, 0);
        mv_pass(sym_mv{}, 0, 1);  // every row's w in place
#pragma unroll
        for (int r = 0; r < R; ++r) vsv[r] = wave_sum(vbv[r][lane] * wvv[r][lane]);
    }

    // q_ij = e^T M e with e = vbar_i - Vbar_j (Eq. 9), expanded through the symmetric
    // part S of M (same quadratic form): q = vbar_i^T S vbar_i - 2 Vbar_j . w_i +
    // Vbar_j^T M Vbar_j, the last term per block from the pooling pass.
    // s_ij = P_ij sqrt(q_ij), key_ij = s_ij / max(1 - P_ij, eps) (Eqs. 6-7).
    double cj[CPL];
#pragma unroll
    for (int c = 0; c < CPL; ++c) cj[c] = cT[jc[c]];
    dot_pass(1, rsV, acc);
    // The block with P > 1/2, if a row has one (at most one does): there e = vbar_i -
    // Vbar_j shrinks with 1 - P while the expansion's terms do not, so the expansion
    // would leave mostly rounding error (a single-block row: e = 0 exactly). Its q is
    // taken directly as e^T M e (M_h from LDS; e through the wave's staging rows, idle
    // after the product): lane t forms e_t (M e)_t.
    int dom_c[R], dom_l[R];
    double q_dom[R];
    {
        double *ebuf = stage + (size_t)wave * R * SROW;
#pragma unroll
        for (int r = 0; r < R; ++r) {
            dom_c[r] = -1;
            dom_l[r] = 0;
            q_dom[r] = 0.0;
#pragma unroll
            for (int c = 0; c < CPL; ++c) {
                const unsigned long long b = __ballot(valid[c] && P[r][c] > 0.5);
                if (b != 0ull) {
                    dom_c[r] = c;
                    dom_l[r] = __builtin_ctzll(b);
                }
            }
            if (dom_c[r] < 0) continue;
            const double e = vbv[r][lane] - pooled_row(rsV, dom_l[r] + 64 * dom_c[r], lane);
            ebuf[lane] = e;
            __builtin_amdgcn_wave_barrier();
            double u = 0.0;
            for (int c = 0; c < kD; ++c) u = fma((double)Ms[lane * (kD + 1) + c], ebuf[c], u);
            __builtin_amdgcn_wave_barrier();
            q_dom[r] = wave_sum(e * u);
        }
    }
#pragma unroll
    for (int r = 0; r < R; ++r) {
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
            const double q = (c == dom_c[r] && lane == dom_l[r]) ? q_dom[r] : fma(-2.0, acc[r][c], vsv[r] + cj[c]);
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
    double K[R], G[R], J[R], J0[R], Jb[R], msum[R];
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
            if (crit == RESS_CRITERION_PROBABILITY && p.cdf_tau > 0.0) {
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
                    const unsigned long long sel = topk_slots<CPL>(ko, cand_bits, n, lane_lt);
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
            const unsigned long long keep = topk_slots<CPL>(ko, cand_bits, crow[r], lane_lt);
            inD[r] = cand_bits & ~keep;
        }
        double mass = 0.0;
#pragma unroll
        for (int c = 0; c < CPL; ++c) {
            acc[r][c] = ((inD[r] >> c) & 1ull) ? P[r][c] : 0.0;  // weights of the g pass
            mass += acc[r][c];
        }
        msum[r] = wave_sum(mass);
        K[r] = 1.0 - msum[r];
    }
    // g = sum_{j in D} P_j (vbar - Vbar_j) = (sum_{j in D} P_j) vbar - sum_{j in D} P_j Vbar_j
    wsum_pass(acc, 2);
#pragma unroll
    for (int r = 0; r < R; ++r) gv[r][lane] = fma(msum[r], vbv[r][lane], -gv[r][lane]);
    double *hv[R];  // M g reuses the slot of S vbar
#pragma unroll
    for (int r = 0; r < R; ++r) hv[r] = wvv[r];
    // h = M g, G = g . h, J = G / max(K, eps)^2, and vbar . h for the next round's gains.
    double vmg[R];
    auto objective = [&]() {
        __syncthreads();  // every row's g in place
        mv_pass(plain_mv{}, 2, 1);
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const double hh = hv[r][lane];
            wave_sum2(gv[r][lane] * hh, vbv[r][lane] * hh, G[r], vmg[r]);
            const double Kh = K[r] > eps ? K[r] : eps;
            J[r] = G[r] / (Kh * Kh);
        }
    };
    objective();
#pragma unroll
    for (int r = 0; r < R; ++r) {
        J0[r] = Jb[r] = J[r];
        best[r] = inD[r];
    }

    // Budget-neutral restoration rounds (Eqs. 13-17) with track-best. The swap
    // count follows each row's kept count; the workgroup stops once no row of it
    // swaps anything.
    double *swap_w = lds.swap_w();
    int *swap_j = lds.swap_j();
    // The wave's own staging rows, idle between the products: scratch for packing
    // sparse member sets in the searches.
    unsigned int *scr = reinterpret_cast<unsigned int *>(stage + (size_t)wave * R * SROW);
    for (int rr = 0; rr < p.rounds; ++rr) {
        int mrow[R], mmax = 0;
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int m = swaps_of_round(crow[r], p.rho, rr, p.swap_floor);
            mrow[r] = dense[r] ? 0 : min(m, min(n_p - crow[r], crow[r]));
            mmax = max(mmax, mrow[r]);
        }
        if (!__syncthreads_or(mmax > 0)) break;
        // e_k . (M g) = vbar . (M g) - Vbar_k . (M g) for every candidate k of every row.
        dot_pass(1, rsV, acc);
#pragma unroll
        for (int r = 0; r < R; ++r)
#pragma unroll
            for (int c = 0; c < CPL; ++c) acc[r][c] = vmg[r] - acc[r][c];
        // Gains of every single restore / drop at the round-start state; the m best
        // of each kind are applied together, g and K following Eq. 13.
#pragma unroll
        for (int r = 0; r < R; ++r) {
            const int m = mrow[r];
            if (m <= 0) continue;
            unsigned long long dj[CPL];
#pragma unroll
            for (int c = 0; c < CPL; ++c) {
                const bool in = (inD[r] >> c) & 1ull;
                const double dkMg = P[r][c] * acc[r][c];
                const double dG = in ? -2.0 * dkMg + S2[r][c] : 2.0 * dkMg + S2[r][c];  // Eqs. 14-15
                const double Kn = K[r] + (in ? P[r][c] : -P[r][c]);
                const double Knh = Kn > eps ? Kn : eps;
                const double dJ = J[r] - (G[r] + dG) / (Knh * Knh);  // Eq. 16
                dj[c] = order_key(maximise ? -dJ : dJ);
            }
            const unsigned long long rest = topk_any<CPL>(dj, inD[r], m, lane, lane_lt, scr);
            const unsigned long long drop = topk_any<CPL>(dj, cand_bits & ~inD[r], m, lane, lane_lt, scr);
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
                    for (int u = 0; u < 8; ++u) vj[u] = pooled_row(rsV, js[u], lane);
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
            K[r] += wave_sum(mr - md);
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

template <int CPL, int R, int NW>
hipError_t launch_cfg(const SelectParams &p, hipStream_t s)
{
    SelectParams q = p;
    const int groups = (p.n_qb + NW * R - 1) / (NW * R);
    q.items_per_xcd = (p.H * groups + 7) / 8;
    hipLaunchKernelGGL((select_kernel<CPL, R, NW>), dim3((unsigned)(8 * q.items_per_xcd)), dim3(NW * 64), 0, s, q);
    return hipGetLastError();
}

// Rows per workgroup, among 24 (8 waves of 3 rows), 16 (8 waves of 2), 8 (8
// waves of 1) and 4 (4 waves of 1): the one with the fewest rounds of
// workgroups over the chip's 256 compute units (one workgroup each), weighted
// by the rows each wave carries plus one (its serial row work); 4 rows over 8
// on a tie (more compute units busy), and 16 or 24 only when strictly cheaper.
// Several rows per wave only up to 6 slots per lane (their candidate state must
// fit the registers of two waves per SIMD); 4 waves of 1 row beyond 1088 key
// blocks.
constexpr long long kCUs = 256;
template <int CPL, bool MULTI_ROW>
hipError_t launch_rows(const SelectParams &p, hipStream_t s)
{
    auto cost = [&](int rows, int r) {
        const long long wg = (long long)p.H * ((p.n_qb + rows - 1) / rows);
        return ((wg + kCUs - 1) / kCUs) * (r + 1);
    };
    int best = 8;
    long long bc = cost(8, 1);
    if (cost(4, 1) <= bc) best = 4, bc = cost(4, 1);
    if constexpr (MULTI_ROW) {
        if (cost(16, 2) < bc) best = 16, bc = cost(16, 2);
        if (cost(24, 3) < bc) best = 24, bc = cost(24, 3);
        if (best == 24) return launch_cfg<CPL, 3, 8>(p, s);
        if (best == 16) return launch_cfg<CPL, 2, 8>(p, s);
    }
    if (best == 8) return launch_cfg<CPL, 1, 8>(p, s);
    return launch_cfg<CPL, 1, 4>(p, s);
}

}  // namespace

hipError_t launch_select(const SelectParams &p, hipStream_t s)
{
    if (p.H == 0 || p.n_qb == 0) return hipSuccess;
    const int n = p.n_kb;
    if (n <= 128) return launch_rows<2, true>(p, s);
    if (n <= 256) return launch_rows<4, true>(p, s);
    if (n <= 384) return launch_rows<6, true>(p, s);
    if (n <= 512) return launch_rows<8, false>(p, s);
    if (n <= 768) return launch_rows<12, false>(p, s);
    if (n <= 1088) return launch_rows<17, false>(p, s);
    if (n <= 2048) return launch_cfg<32, 1, 4>(p, s);
    return launch_cfg<64, 1, 4>(p, s);
}

}  // namespace ress
