// Exact attention over kept key blocks (block-sparse, Sec. 3 step (3)) or over
// all key blocks (dense), bf16 inputs, bf16 MFMA products with float32
// accumulation, float32 online softmax.
//
// One workgroup per (head, query block), BQ/32 waves, each wave owning 32 query
// rows. The score tile is computed transposed, S^T = K Q^T, with
// v_mfma_f32_32x32x16_bf16: its accumulator puts one query per lane (lane l and
// l+32 share query l%32, each holding 16 of every 32 keys), so row sums stay in
// the lane except for one exchange with lane l^32, and the probabilities already
// sit in the B-operand layout of O^T = V^T P^T.
//
// Keys are consumed in 128-key tiles (one 128-key block, or two 64-key blocks
// of the list) split into 64-key halves, software-pipelined over halves: the
// step that forms the probabilities of half n also issues the score MFMAs of
// half n+1 and the PV MFMAs of half n-1, so one basic block holds 16 MFMAs next
// to the softmax arithmetic and the matrix and vector pipes run side by side.
// K and V tiles move from global memory straight into LDS (global_load_lds, 16
// bytes per lane, 1 KB per wave instruction) in two-slot rings; one barrier per
// tile, between its two halves, both publishes the tiles loaded one tile earlier
// and frees the slots the next loads overwrite (K of tile t+2, V of tile t+1).
// Tiles stay row-major (64 channels = 128 bytes per key) with their 16-byte
// chunks XOR-swizzled per key; the swizzle is applied by choosing each lane's
// source chunk, since a DMA instruction fills LDS contiguously. The V^T operand
// comes from ds_read_b64_tr_b16: within 16 lanes, lane s points at 4 channels
// of key k0 + s/4 and lane i receives channel d0 + i of keys k0..k0+3, which is
// the transpose the PV product needs.
//
// Softmax: base-2 exponentials; row sums over the bf16-rounded probabilities
// (the values the PV product consumes) with packed bf16 dot products. There is
// no per-half maximum: every row starts with reference 0 and forms its
// probabilities against its reference; only when a half's sum exceeds 2^50, or
// the row's running sum is still below 2^-100, is the half redone against its
// true maximum (a result within +-40 of 0 is rounded to 0) and O rescaled.
// While every row of a wave has reference 0, the wave runs a copy of the tile
// loop whose probabilities are exp2 of the score accumulators with nothing
// else: Q is multiplied by scale*log2(e) when its fragments are loaded (one extra
// bf16 rounding of Q), so the accumulators are base-2 logits. A wave whose first
// 64 scores reach beyond +-24 in some row reloads Q unscaled instead, so large
// logits are formed exactly; either way every score of a row has one form.
// Softmax is invariant to the reference, so this changes rounding only.
//
// Workgroups are numbered so that neighbouring query blocks of a head share an
// XCD and its L2, where their K/V tiles are re-read, and heads of different cost
// (ragged budgets) still split evenly over the XCDs (see row_of).
#include <type_traits>

#include "ress_internal.h"

namespace ress {
namespace {

typedef __bf16 bf16x8 __attribute__((__vector_size__(8 * sizeof(__bf16))));
typedef __bf16 bf16x2 __attribute__((__vector_size__(2 * sizeof(__bf16))));
typedef short s16x4 __attribute__((__vector_size__(4 * sizeof(short))));
typedef float f32x16 __attribute__((__vector_size__(16 * sizeof(float))));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

constexpr float kSumLimit = 0x1p50f;  // largest probability sum a half may reach
constexpr float kTiny = 0x1p-100f;    // a row whose running sum is below this has no usable reference
constexpr float kZeroBand = 40.f;     // references within +-40 (base-2 logits) become 0
constexpr float kStartBand = 24.f;    // first-half maxima a wave may have to start with reference 0

__device__ __forceinline__ unsigned int bf16_bits(float x)
{
    return (unsigned int)__builtin_bit_cast(unsigned short, (__bf16)x);
}

// XOR applied to the 16-byte chunk index of LDS row `row` (K and V tiles, 128-byte
// rows, two rows per 256-byte bank row). With s = swz(row):
//  - 16 consecutive rows read at one logical chunk (score operand, 16 lanes x 16 B)
//    land on 16 distinct (bank half, chunk) pairs, since (row>>1)&7 -> s is a bijection;
//  - the transpose reads (32 lanes x 8 B: keys 8n..8n+3 or 8n+4..8n+7, each at the 4
//    chunks of one 32-channel half) are split by bit 2 of s between rows 8n and 8n+2.
__device__ __forceinline__ int swz(int row) { return (((row >> 1) & 1) << 2) | ((row >> 2) & 3); }

__device__ __forceinline__ void wait_vm_all() { __builtin_amdgcn_s_waitcnt(0x0F70); }  // vmcnt(0)

// Work order, two forms; within a head, last blocks first (the dense special
// blocks early). Returns false for a workgroup with no row.
//  - Segments (the K and V of all heads fit the infinity cache): the (head, query
//    block) rows, head-major, are cut into 8 contiguous segments of about equal
//    work, one per XCD, so that each XCD fills its L2 with few heads' K and V
//    (neighbouring query blocks of a head share it) while ragged per-head budgets
//    stay balanced. A row's work is its head's kept count of query block 0 (the
//    rows of a head keep the same number of blocks, the dense special rows aside;
//    dense attention: equal). Boundaries follow the work split, clamped so that no
//    segment exceeds seg_cap rows (the grid is 8 x seg_cap workgroups; every row
//    lands in exactly one segment).
//  - Rotation (larger layers): XCD x runs, head after head, a chunk of seg_cap
//    consecutive query blocks of every head, chunk (x - h) mod 8 of head h, so
//    that each head's chunks are spread over all XCDs and the XCDs move through the
//    heads together (the grid is 8 x H x seg_cap workgroups).
__device__ __forceinline__ bool row_of(const AttnParams &p, bool sparse, int xcd, int local, int &h, int &i)
{
    const int H = p.H, n = p.n_qb;
    if (p.rotate) {
        const int chunk = p.seg_cap;
        const int slot = local / chunk, r = local - slot * chunk;
        if (slot >= H) return false;
        h = (xcd + slot) % H;
        const int i_fwd = ((xcd - h % 8 + 8) & 7) * chunk + r;
        if (i_fwd >= n) return false;
        i = n - 1 - i_fwd;
        return true;
    }
    const long long T = (long long)H * n, cap = p.seg_cap;
    auto weight = [&](int hh) -> long long {
        return sparse ? (long long)max(p.kept_count[(size_t)hh * n], 1) : 1ll;
    };
    long long W = 0;
    for (int hh = 0; hh < H; ++hh) W += weight(hh) * n;
    // First row whose work prefix reaches x W / 8.
    auto split = [&](int x) -> long long {
        const long long target = (W / 8) * x + ((W % 8) * x + 7) / 8;
        long long acc = 0;
        for (int hh = 0; hh < H; ++hh) {
            const long long w = weight(hh), seg = w * n;
            if (acc + seg >= target)  // 0 < target - acc <= w n < 2^31
                return (long long)hh * n + ((int)(target - acc) + (int)w - 1) / (int)w;
            acc += seg;
        }
        return T;
    };
    long long b = 0, e = 0;
    for (int x = 1; x <= xcd + 1; ++x) {
        const long long lo = max(e, T - (8 - x) * cap), hi = min(e + cap, T);
        b = e;
        e = min(max(split(x), lo), hi);
    }
    const int g = (int)b + local;  // rows < 2^31 (checked on the host)
    if (g >= (int)e) return false;
    h = g / n;
    i = n - 1 - (g - h * n);
    return true;
}

// Two waves per SIMD for 128-query blocks (two 64 KB workgroups per CU); the LDS
// allows 64-query blocks only one.
template <int BQ, int BK, bool SPARSE>
__global__ void __launch_bounds__(BQ * 2, BQ == 128 ? 2 : 1) attn_kernel(const AttnParams p)
{
    constexpr int T = BQ * 2;                 // threads
    constexpr int NW = BQ / 32;               // waves
    constexpr int EPT = BK == 128 ? 1 : 2;    // kept-list entries per 128-key tile
    constexpr int LPH = 64 * 8 / T;           // 16-byte DMA loads per thread, tensor and half
    constexpr int TILE = 128 * 128;           // bytes of one K (or V) tile
    constexpr int HALF = TILE / 2;
    static_assert(64 * 8 % T == 0 && LPH >= 1, "a half tile must split evenly over the threads");
    __shared__ __attribute__((aligned(1024))) unsigned char k_lds0[TILE];
    __shared__ __attribute__((aligned(1024))) unsigned char k_lds1[TILE];
    __shared__ __attribute__((aligned(1024))) unsigned char v_lds0[TILE];
    __shared__ __attribute__((aligned(1024))) unsigned char v_lds1[TILE];

    const int xcd = blockIdx.x & 7, local = blockIdx.x >> 3;
    int h, i;
    if (!row_of(p, SPARSE, xcd, local, h, i)) return;
    const int N = p.N, n_kb = p.n_kb;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int hh = lane >> 5, ql = lane & 31;
    const int g16 = (lane >> 4) & 1, s16 = lane & 15;
    const int q0 = i * BQ + wave * 32 + ql;
    const size_t head = (size_t)h * N;

    // Q fragments, pre-multiplied by scale*log2(e) so that scores are base-2 logits,
    // unless the wave's first scores show logits beyond kStartBand (then unscaled).
    const float c = p.scale_log2;
    bf16x8 qf[4];
    auto load_q = [&](bool scaled) __attribute__((always_inline)) {
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
            if (q0 < N) {
                const bf16x8 x = *reinterpret_cast<const bf16x8 *>(p.q + (head + q0) * kD + kk * 16 + hh * 8);
                if (scaled) {
#pragma unroll
                    for (int e = 0; e < 8; ++e) qf[kk][e] = (__bf16)((float)x[e] * c);
                } else {
                    qf[kk] = x;
                }
            } else {
                qf[kk] = bf16x8{};
            }
        }
    };
    load_q(true);

    int n_ent;  // key blocks to visit
    const int32_t *list = nullptr;
    if constexpr (SPARSE) {
        const size_t row = (size_t)h * p.n_qb + i;
        n_ent = min(max(p.kept_count[row], 0), n_kb);
        list = p.kept_idx + row * n_kb;
    } else {
        n_ent = n_kb;
    }
    const int L = (n_ent + EPT - 1) / EPT;  // 128-key tiles

    // Kept block indices, read 64 at a time: lane l of idx_lo holds entry 64c + l of
    // the list, idx_hi the next 64, loaded one chunk ahead of use.
    int idx_lo = -1, idx_hi = -1;
    auto load_chunk = [&](int c) __attribute__((always_inline)) -> int {
        const int t = 64 * c + lane;
        return t < n_ent ? list[t] : -1;
    };
    if constexpr (SPARSE) {
        idx_lo = load_chunk(0);
        idx_hi = load_chunk(1);
    }
    // Block index of entry e (-1 past the end); called for e = 0, 1, 2, ... in order.
    auto entry = [&](int e) __attribute__((always_inline)) -> int {
        if constexpr (SPARSE) {
            if (e > 0 && (e & 63) == 0) {
                idx_lo = idx_hi;
                idx_hi = load_chunk((e >> 6) + 1);
            }
            return __builtin_amdgcn_readlane(idx_lo, e & 63);
        } else {
            return e < n_ent ? e : -1;
        }
    };
    auto fetch_tile = [&](int t, int (&jt)[EPT]) __attribute__((always_inline)) {
#pragma unroll
        for (int e = 0; e < EPT; ++e) jt[e] = entry(t * EPT + e);
    };
    auto valid = [&](int j) __attribute__((always_inline)) { return j >= 0 && j < n_kb; };
    // First token of half hf of a tile, and how many of its 64 keys are real.
    auto half_row0 = [&](const int (&jt)[EPT], int hf) __attribute__((always_inline)) -> int {
        if constexpr (EPT == 1) return valid(jt[0]) ? jt[0] * 128 + 64 * hf : 0;
        else return valid(jt[hf]) ? jt[hf] * 64 : 0;
    };
    auto half_keys = [&](const int (&jt)[EPT], int hf) __attribute__((always_inline)) -> int {
        if constexpr (EPT == 1) return valid(jt[0]) ? max(0, min(64, N - jt[0] * 128 - 64 * hf)) : 0;
        else return valid(jt[hf]) ? min(64, N - jt[hf] * 64) : 0;
    };

    // DMA: thread-constant byte offsets within a 64-row half (row r of the half,
    // the logical chunk that belongs at physical chunk lane&7).
    const unsigned char *kbytes = reinterpret_cast<const unsigned char *>(p.k + head * kD);
    const unsigned char *vbytes = reinterpret_cast<const unsigned char *>(p.v + head * kD);
    unsigned int doff[LPH];
#pragma unroll
    for (int u = 0; u < LPH; ++u) {
        const int r = (u * NW + wave) * 8 + (lane >> 3);
        doff[u] = (unsigned int)(r * 128 + (((lane & 7) ^ swz(r)) << 4));
    }
    // Rows row0..row0+63 of one tensor into a half slot; rows past N repeat row N-1.
    auto dma_half = [&](const unsigned char *src, int row0, unsigned char *dst) __attribute__((always_inline)) {
        if (row0 + 64 <= N) {
            const unsigned char *s = src + (size_t)row0 * 128;
#pragma unroll
            for (int u = 0; u < LPH; ++u)
                __builtin_amdgcn_global_load_lds((const void *)(s + doff[u]), (lds_void *)(dst + (u * NW + wave) * 1024), 16, 0, 0);
        } else {
#pragma unroll
            for (int u = 0; u < LPH; ++u) {
                const int r = (u * NW + wave) * 8 + (lane >> 3);
                const int row = min(row0 + r, N - 1);
                __builtin_amdgcn_global_load_lds((const void *)(src + (size_t)row * 128 + (doff[u] & 127)),
                                                 (lds_void *)(dst + (u * NW + wave) * 1024), 16, 0, 0);
            }
        }
    };
    auto dma_tile = [&](const unsigned char *src, const int (&jt)[EPT], unsigned char *dst) __attribute__((always_inline)) {
        dma_half(src, half_row0(jt, 0), dst);
        dma_half(src, half_row0(jt, 1), dst + HALF);
    };

    // Per-lane LDS byte offsets of the operand reads (tile-relative; the key
    // offset of a half / sub-tile is added as an immediate).
    int koff[4];  // score operand: key ql, logical chunk 2kk+hh
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) koff[kk] = ql * 128 + (((2 * kk + hh) ^ swz(ql)) << 4);
    int voff[2][2];  // transpose reads: key 8r + 4hh + s16/4, channels 32dh + 16g16 + 4(s16&3)
#pragma unroll
    for (int dh = 0; dh < 2; ++dh)
#pragma unroll
        for (int r = 0; r < 2; ++r) {
            const int key = 8 * r + 4 * hh + (s16 >> 2);
            const int d = 32 * dh + 16 * g16 + 4 * (s16 & 3);
            voff[dh][r] = key * 128 + (((d >> 3) ^ swz(key)) << 4) + (d & 7) * 2;
        }

    float mref = 0.f;   // reference of this lane's query row (shared with lane^32), base-2 logits
    bool zref = true;   // wave-uniform: every row has reference 0 (Q then is pre-scaled)
    float cw = 1.f;     // wave-uniform: base-2 logit per unit score (1 for pre-scaled Q, else c)
    float lrow = 0.f;
    f32x16 acc_o[2];
#pragma unroll
    for (int dh = 0; dh < 2; ++dh)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc_o[dh][v] = 0.f;
    const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};

    // S^T of one half: two 32-key sub-tiles, 4 MFMAs each.
    auto qk = [&](const unsigned char *kt, int hf, f32x16 (&s)[2]) __attribute__((always_inline)) {
#pragma unroll
        for (int t = 0; t < 2; ++t) {
#pragma unroll
            for (int v = 0; v < 16; ++v) s[t][v] = 0.f;
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) {
                const bf16x8 a = *reinterpret_cast<const bf16x8 *>(kt + hf * HALF + t * 32 * 128 + koff[kk]);
                s[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[kk], s[t], 0, 0, 0);
            }
        }
    };
    // O^T += V^T P^T for one half, 16 keys per MFMA.
    auto pv = [&](const unsigned char *vt, int hf, const bf16x8 (&pb)[2][2]) __attribute__((always_inline)) {
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int u = 0; u < 2; ++u)
#pragma unroll
                for (int dh = 0; dh < 2; ++dh) {
                    const unsigned char *base = vt + hf * HALF + (t * 32 + u * 16) * 128;
                    const s16x4 r0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(base + voff[dh][0]));
                    const s16x4 r1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(base + voff[dh][1]));
                    const bf16x8 a = __builtin_bit_cast(
                        bf16x8, (short __attribute__((__vector_size__(8 * sizeof(short))))){
                                    r0[0], r0[1], r0[2], r0[3], r1[0], r1[1], r1[2], r1[3]});
                    acc_o[dh] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[t][u], acc_o[dh], 0, 0, 0);
                }
    };
    // Key of element (t, v) of a half: t 32 + (v / 4) 8 + (v % 4) + 4 hh; compared as
    // 4 hh >= nv - (the lane-independent part), a scalar per element.
    const int hh4 = hh * 4;
    auto mask = [&](f32x16 (&s)[2], int nv) __attribute__((always_inline)) {
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int lim = __builtin_amdgcn_readfirstlane(nv - (t * 32 + (v >> 2) * 8 + (v & 3)));
                if (hh4 >= lim) s[t][v] = -INFINITY;
            }
    };
    // Probabilities of sub-tile t (32 keys) of a half, exp2(s) when every row has
    // reference 0 (Z), else exp2(s * cw - mref); adds the bf16-rounded values to
    // the lane's partial sums.
    auto probs_part = [&](auto z, const f32x16 (&s)[2], bf16x8 (&pb)[2][2], int t, float &l0,
                          float &l1) __attribute__((always_inline)) {
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            float e[8];
#pragma unroll
            for (int jj = 0; jj < 8; ++jj) {
                const float x = s[t][u * 8 + jj];
                e[jj] = __builtin_amdgcn_exp2f(decltype(z)::value ? x : fmaf(x, cw, -mref));
            }
            pb[t][u] = bf16x8{(__bf16)e[0], (__bf16)e[1], (__bf16)e[2], (__bf16)e[3],
                              (__bf16)e[4], (__bf16)e[5], (__bf16)e[6], (__bf16)e[7]};
#pragma unroll
            for (int jj = 0; jj < 8; jj += 4) {
                l0 = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{pb[t][u][jj], pb[t][u][jj + 1]}, ones, l0, false);
                l1 = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{pb[t][u][jj + 2], pb[t][u][jj + 3]}, ones, l1, false);
            }
        }
    };
    // Tile-loop variants: every row's reference is 0 (zero), or per-row references (general).
    using general = std::integral_constant<bool, false>;
    using zero = std::integral_constant<bool, true>;
    // All probabilities of one half against the current references; returns the lane's sum.
    auto probs = [&](const f32x16 (&s)[2], bf16x8 (&pb)[2][2]) __attribute__((always_inline)) -> float {
        float l0 = 0.f, l1 = 0.f;
        probs_part(general{}, s, pb, 0, l0, l1);
        probs_part(general{}, s, pb, 1, l0, l1);
        return l0 + l1;
    };
    // Accept the half's probabilities, or redo them against a new reference
    // (rescaling O and the running sum) when the half's sum exceeds kSumLimit,
    // the row still has no mass above kTiny, or (zero variant) a row of the wave
    // already left reference 0 earlier in this tile.
    auto settle = [&](auto z, const f32x16 (&s)[2], bf16x8 (&pb)[2][2], float lh) __attribute__((always_inline)) {
        constexpr bool Z = decltype(z)::value;
        if (__any(!(lh <= kSumLimit) || lrow + lh < kTiny || (Z && mref != 0.f))) {
            float tmax = -INFINITY;
#pragma unroll
            for (int t = 0; t < 2; ++t)
#pragma unroll
                for (int v = 0; v < 16; ++v) tmax = fmaxf(tmax, s[t][v]);
            tmax = fmaxf(tmax, __shfl_xor(tmax, 32)) * cw;
            // Decisions about the row's mass use the row's running sum: lanes l and
            // l^32 each sum half of the row's keys (one of them may have no mass yet
            // while the row has), and both must take the same reference.
            const float lsum = lrow + __shfl_xor(lrow, 32);
            // The reference only rises, except while the row has no usable mass yet:
            // then it may fall to this half's maximum, but not below
            // mref + log2(lsum), an upper bound of every earlier logit of the row, so
            // that the rescaled running sums stay at most 1 (finite).
            float mnew = fmaxf(mref, tmax);
            // (log2 of a denormal sum may come back as -inf: -149 bounds it.)
            if (lsum < kTiny) mnew = lsum > 0.f ? fmaxf(tmax, mref + fmaxf(__log2f(lsum), -149.f)) : tmax;
            if (tmax == -INFINITY) mnew = mref;  // a fully masked half says nothing
            if (fabsf(mnew) <= kZeroBand) mnew = 0.f;
            // A row without mass has nothing to rescale (and 0 * exp2(large) must not
            // happen); otherwise the factor is applied as two halves, each finite
            // for shifts up to 2^8 (a running sum as small as the smallest denormal).
            const float alpha = lsum > 0.f ? __builtin_amdgcn_exp2f(0.5f * (mref - mnew)) : 0.f;
            lrow = (lrow * alpha) * alpha;
#pragma unroll
            for (int dh = 0; dh < 2; ++dh)
#pragma unroll
                for (int v = 0; v < 16; ++v) acc_o[dh][v] = (acc_o[dh][v] * alpha) * alpha;
            mref = mnew;
            if (Z) zref = __all(mref == 0.f);
            lh = probs(s, pb);
        }
        lrow += lh;
    };
    // One pipeline step: softmax of the current half (scores sc, nv real keys)
    // beside the score MFMAs of the next half (kt, khf -> sn) and the PV MFMAs
    // of the previous half (probabilities pp, vt, vhf).
    auto step = [&](auto z, f32x16 (&sc)[2], bf16x8 (&pc)[2][2], int nv, f32x16 (&sn)[2], const unsigned char *kt,
                    int khf, const bf16x8 (&pp)[2][2], const unsigned char *vt, int vhf) __attribute__((always_inline)) {
        if (nv < 64) {
            // A real branch: only partial halves pay for the mask (the empty asm
            // keeps the compiler from if-converting it into every step).
            asm volatile("" ::: "memory");
            mask(sc, nv);
        }
        // Two scheduling regions. First the score MFMAs of the next half (their
        // results are consumed at the next step) beside the softmax of sub-tile 0,
        // then the PV MFMAs of the previous half beside the softmax of sub-tile 1.
        // In each, the compiler's MFMA/LDS interleaving strategy 0 (measured: the
        // same results, dense 1.5% and the 128/64 grid 1% faster).
        float l0 = 0.f, l1 = 0.f;
        __builtin_amdgcn_iglp_opt(0);
        qk(kt, khf, sn);
        probs_part(z, sc, pc, 0, l0, l1);
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_iglp_opt(0);
        pv(vt, vhf, pp);
        probs_part(z, sc, pc, 1, l0, l1);
        const float lh = l0 + l1;
        settle(z, sc, pc, lh);
    };

    f32x16 sA[2], sB[2];
    bf16x8 pA[2][2], pB[2][2];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int u = 0; u < 2; ++u) pB[t][u] = bf16x8{};
    int jt0[EPT], jt1[EPT], jt2[EPT];

    // Tile it (it = 0 .. L-1): K in kc, V in vc; K of tile it+1 in kn; V of tile
    // it-1 in vp. sA holds the scores of (it, half 0), pB the probabilities of
    // (it-1, half 1).
    auto iter = [&](auto z, int it, unsigned char *kc, const unsigned char *kn, const unsigned char *vc,
                    unsigned char *vp) __attribute__((always_inline)) {
        fetch_tile(it + 2, jt2);
        step(z, sA, pA, half_keys(jt0, 0), sB, kc, 1, pB, vp, 1);
        wait_vm_all();    // this wave's loads of K(it+1) and V(it) have landed
        __syncthreads();  // ... and every wave's; K(it) and V(it-1) are no longer read
        if (it + 2 < L) dma_tile(kbytes, jt2, kc);
        if (it + 1 < L) dma_tile(vbytes, jt1, vp);
        step(z, sB, pB, half_keys(jt0, 1), sA, kn, 0, pA, vc, 0);
#pragma unroll
        for (int e = 0; e < EPT; ++e) {
            jt0[e] = jt1[e];
            jt1[e] = jt2[e];
        }
    };

    if (L > 0) {
        fetch_tile(0, jt0);
        fetch_tile(1, jt1);
        // The first step multiplies zero probabilities with V slot 1, half 1.
        for (int u = tid; u < HALF / 16; u += T) reinterpret_cast<uint4 *>(v_lds1 + HALF)[u] = make_uint4(0, 0, 0, 0);
        dma_tile(kbytes, jt0, k_lds0);
        if (L > 1) dma_tile(kbytes, jt1, k_lds1);
        dma_tile(vbytes, jt0, v_lds0);
        wait_vm_all();
        __syncthreads();
        qk(k_lds0, 0, sA);
        {
            // Start with reference 0 only if every row's first logits lie within
            // kStartBand; otherwise use unscaled Q (exact scores) from the start.
            float m0 = -INFINITY;
#pragma unroll
            for (int t = 0; t < 2; ++t)
#pragma unroll
                for (int v = 0; v < 16; ++v) m0 = fmaxf(m0, sA[t][v]);
            m0 = fmaxf(m0, __shfl_xor(m0, 32));
            zref = __all(fabsf(m0) <= kStartBand);
            if (!zref) {
                load_q(false);
                cw = c;
                qk(k_lds0, 0, sA);
            }
        }
        int it = 0;
        // A wave leaves the zero variant (for good) when a row's reference leaves 0;
        // its Q stays pre-scaled (cw = 1), so every score of a row has one form.
        for (;;) {
            if (zref) iter(zero{}, it, k_lds0, k_lds1, v_lds0, v_lds1);
            else iter(general{}, it, k_lds0, k_lds1, v_lds0, v_lds1);
            if (++it >= L) break;
            if (zref) iter(zero{}, it, k_lds1, k_lds0, v_lds1, v_lds0);
            else iter(general{}, it, k_lds1, k_lds0, v_lds1, v_lds0);
            if (++it >= L) break;
        }
        // PV of the last half; its tile sits in V slot (L-1) % 2.
        pv((L & 1) ? v_lds0 : v_lds1, 1, pB);
    }

    // Each lane summed half of its row's keys; lanes l and l^32 share the row.
    const float ltot = lrow + __shfl_xor(lrow, 32);
    const float inv = ltot > 0.f ? 1.f / ltot : 0.f;
    if (q0 < N && p.o32) {
        float *orow = p.o32 + (head + q0) * kD;
#pragma unroll
        for (int dh = 0; dh < 2; ++dh)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int d0 = dh * 32 + g * 8 + hh * 4;
                *reinterpret_cast<float4 *>(orow + d0) =
                    make_float4(acc_o[dh][g * 4 + 0] * inv, acc_o[dh][g * 4 + 1] * inv,
                                acc_o[dh][g * 4 + 2] * inv, acc_o[dh][g * 4 + 3] * inv);
            }
    } else if (q0 < N) {
        uint16_t *orow = p.o + (head + q0) * kD;
#pragma unroll
        for (int dh = 0; dh < 2; ++dh)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int d0 = dh * 32 + g * 8 + hh * 4;
                const unsigned int lo = bf16_bits(acc_o[dh][g * 4 + 0] * inv) |
                                        (bf16_bits(acc_o[dh][g * 4 + 1] * inv) << 16);
                const unsigned int hi = bf16_bits(acc_o[dh][g * 4 + 2] * inv) |
                                        (bf16_bits(acc_o[dh][g * 4 + 3] * inv) << 16);
                *reinterpret_cast<uint2 *>(orow + d0) = make_uint2(lo, hi);
            }
    }
}

template <int BQ, int BK>
hipError_t launch_bk(const AttnParams &p, bool sparse, hipStream_t s)
{
    const dim3 grid((unsigned)(p.rotate ? 8 * p.H * p.seg_cap : 8 * p.seg_cap)), block(BQ * 2);
    if (sparse)
        hipLaunchKernelGGL((attn_kernel<BQ, BK, true>), grid, block, 0, s, p);
    else
        hipLaunchKernelGGL((attn_kernel<BQ, BK, false>), grid, block, 0, s, p);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_attn(const AttnParams &p, int bq, int bk, bool sparse, hipStream_t s)
{
    if (p.H == 0 || p.n_qb == 0) return hipSuccess;
    if (bq == 128 && bk == 128) return launch_bk<128, 128>(p, sparse, s);
    if (bq == 128 && bk == 64) return launch_bk<128, 64>(p, sparse, s);
    if (bq == 64 && bk == 128) return launch_bk<64, 128>(p, sparse, s);
    return launch_bk<64, 64>(p, sparse, s);
}

}  // namespace ress
