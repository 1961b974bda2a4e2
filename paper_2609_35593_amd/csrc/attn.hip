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
// Keys are consumed in 64-key chunks (one 64-key block of the kept list, or half
// of a 128-key block). A chunk is two 32-key sub-tiles; for each, a wave issues
// its 4 score MFMAs, forms the probabilities and issues its 4 PV MFMAs (the score
// MFMAs of the second sub-tile go ahead of the PV MFMAs of the first). Latency is
// hidden by occupancy rather than by a software pipeline across chunks:
// K and V chunks sit in two-slot rings of 8 KB per tensor and slot (32 KB per
// workgroup), and the kernel fits 128 registers, so four 128-query workgroups
// share a CU (four waves per SIMD), and the matrix and vector pipes of a SIMD
// serve whichever of its waves is ready. (Measured: at D = 64 the softmax needs
// about as many issue slots as the MFMAs; two waves per SIMD with a software
// pipeline reached the same rate as three without one, four waves run 4-8%
// faster.)
//
// Chunks move from global memory straight into LDS (buffer_load ... lds, 16
// bytes per lane, 1 KB per wave instruction, 32-bit offsets against a per-head
// buffer resource): chunk c+1 is loaded while chunk c is computed, and one
// barrier per chunk both publishes chunk c+1 and frees chunk c's slots. Rows stay
// row-major (64 channels = 128 bytes per key) with their 16-byte chunks
// XOR-swizzled per key; the swizzle is applied by choosing each lane's source
// chunk, since a DMA instruction fills LDS contiguously. The V^T operand comes
// from ds_read_b64_tr_b16: within 16 lanes, lane s points at 4 channels of key
// k0 + s/4 and lane i receives channel d0 + i of keys k0..k0+3, which is the
// transpose the PV product needs. The kept list is read through the scalar
// cache (wave-uniform addresses).
//
// Softmax: base-2 exponentials; row sums over the bf16-rounded probabilities
// (the values the PV product consumes) with packed bf16 dot products. There is
// no per-tile maximum: every row starts with reference 0 and forms its
// probabilities against its reference; only when a sub-tile's sum exceeds 2^50,
// or the row's running sum is still below 2^-100, is the sub-tile redone against
// its true maximum (a result within +-40 of 0 is rounded to 0) and O rescaled.
// While every row of a wave has reference 0, the wave runs a copy of the chunk
// loop whose probabilities are exp2 of the score accumulators with nothing
// else: Q is multiplied by scale*log2(e) when its fragments are loaded (one extra
// bf16 rounding of Q), so the accumulators are base-2 logits. A wave whose first
// 64 scores reach beyond +-24 in some row reloads Q unscaled instead, so large
// logits are formed exactly; either way every score of a row has one form.
// Softmax is invariant to the reference, so this changes rounding only.
//
// Workgroups are numbered so that neighbouring query blocks of a head share an
// XCD and its L2, where their K/V chunks are re-read, and heads of different cost
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

constexpr float kSumLimit = 0x1p50f;  // largest probability sum a sub-tile may reach
constexpr float kTiny = 0x1p-100f;    // a row whose running sum is below this has no usable reference
constexpr float kZeroBand = 40.f;     // references within +-40 (base-2 logits) become 0
constexpr float kStartBand = 24.f;    // first-chunk maxima a wave may have to start with reference 0

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

// Four waves per SIMD for 128-query blocks (four 32 KB workgroups per CU); 64-query
// blocks are held to two by the LDS (five 2-wave workgroups per CU).
template <int BQ, int BK, bool SPARSE>
__global__ void __launch_bounds__(BQ * 2, BQ == 128 ? 4 : 2) attn_kernel(const AttnParams p)
{
    constexpr int T = BQ * 2;                 // threads
    constexpr int NW = BQ / 32;               // waves
    constexpr int CPE = BK / 64;              // 64-key chunks per kept-list entry
    constexpr int LPC = 64 * 8 / T;           // 16-byte DMA loads per thread, tensor and chunk
    constexpr int SLOT = 64 * 128;            // bytes of one chunk of K (or V)
    static_assert(64 * 8 % T == 0 && LPC >= 1, "a chunk must split evenly over the threads");
    __shared__ __attribute__((aligned(1024))) unsigned char k_s0[SLOT];
    __shared__ __attribute__((aligned(1024))) unsigned char k_s1[SLOT];
    __shared__ __attribute__((aligned(1024))) unsigned char v_s0[SLOT];
    __shared__ __attribute__((aligned(1024))) unsigned char v_s1[SLOT];

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
    int C = n_ent * CPE;  // 64-key chunks
    if (CPE == 2 && n_ent > 0 && N - (n_kb - 1) * BK <= 64) {
        // The last block holds at most 64 tokens: its second chunk is empty.
        int jl;
        if constexpr (SPARSE) jl = list[n_ent - 1];
        else jl = n_ent - 1;
        if (__builtin_amdgcn_readfirstlane(jl) == n_kb - 1) C -= 1;
    }

    // Kept block indices through the scalar cache (wave-uniform addresses; the list
    // is read-only here).
    typedef const __attribute__((address_space(4))) int32_t cint32;
    const cint32 *klist = (const cint32 *)list;
    auto block_of = [&](int ch) __attribute__((always_inline)) -> int {
        const int e = ch / CPE;
        if constexpr (SPARSE) return e < n_ent ? klist[e] : -1;
        else return e < n_ent ? e : -1;
    };
    auto valid = [&](int j) __attribute__((always_inline)) { return j >= 0 && j < n_kb; };
    // First token of chunk ch of block j, and how many of its 64 keys are real.
    auto chunk_row0 = [&](int j, int ch) __attribute__((always_inline)) -> int {
        return valid(j) ? j * BK + 64 * (ch & (CPE - 1)) : 0;
    };
    auto chunk_keys = [&](int j, int ch) __attribute__((always_inline)) -> int {
        return valid(j) ? max(0, min(64, N - j * BK - 64 * (ch & (CPE - 1)))) : 0;
    };

    // This head's K and V as buffer resources: N * 128 bytes (at most 2^31 for
    // N <= 2^24, as a 32-bit unsigned record count; row offsets stay below 2^31).
    const int head_bytes = (int)((unsigned int)N * 128u);
    const __amdgpu_buffer_rsrc_t krs =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t *>(p.k + head * kD), 0, head_bytes, 0x00020000);
    const __amdgpu_buffer_rsrc_t vrs =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t *>(p.v + head * kD), 0, head_bytes, 0x00020000);
    // DMA lane constants: load u of a thread fills row r0 + 8 NW u of the slot, at
    // physical chunk lane & 7, from source chunk (lane & 7) ^ swz(row) (the same for
    // every u: the swizzle depends on row bits 1-3 only).
    const int r0 = wave * 8 + (lane >> 3);
    const unsigned int coff = (unsigned int)(((lane & 7) ^ swz(r0)) << 4);
    // Rows row0..row0+63 of one tensor into a slot; rows past N repeat row N-1.
    auto dma_chunk = [&](__amdgpu_buffer_rsrc_t rs, int row0, unsigned char *dst) __attribute__((always_inline)) {
#pragma unroll
        for (int u = 0; u < LPC; ++u) {
            const int row = min(row0 + r0 + 8 * NW * u, N - 1);
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void *)(dst + (u * NW + wave) * 1024), 16,
                                                     (unsigned int)(row * 128) + coff, 0, 0, 0);
        }
    };

    // Per-lane LDS byte offsets of the operand reads (chunk-relative; the key offset
    // of a sub-tile is added as an immediate).
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

    // S^T of sub-tile t (32 keys) of a chunk: 4 MFMAs.
    auto qk = [&](const unsigned char *kt, int t, f32x16 &s) __attribute__((always_inline)) {
#pragma unroll
        for (int v = 0; v < 16; ++v) s[v] = 0.f;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
            const bf16x8 a = *reinterpret_cast<const bf16x8 *>(kt + t * 32 * 128 + koff[kk]);
            s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[kk], s, 0, 0, 0);
        }
    };
    // O^T += V^T P^T for sub-tile t, 16 keys per MFMA.
    auto pv = [&](const unsigned char *vt, int t, const bf16x8 (&pb)[2]) __attribute__((always_inline)) {
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
            for (int dh = 0; dh < 2; ++dh) {
                const unsigned char *base = vt + (t * 32 + u * 16) * 128;
                const s16x4 r0v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(base + voff[dh][0]));
                const s16x4 r1v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(base + voff[dh][1]));
                const bf16x8 a = __builtin_bit_cast(
                    bf16x8, (short __attribute__((__vector_size__(8 * sizeof(short))))){
                                r0v[0], r0v[1], r0v[2], r0v[3], r1v[0], r1v[1], r1v[2], r1v[3]});
                acc_o[dh] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[u], acc_o[dh], 0, 0, 0);
            }
    };
    // Key of element v of sub-tile t: t 32 + (v / 4) 8 + (v % 4) + 4 hh; compared as
    // 4 hh >= nv - (the lane-independent part), a scalar per element.
    const int hh4 = hh * 4;
    auto mask = [&](f32x16 &s, int nv, int t) __attribute__((always_inline)) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int lim = __builtin_amdgcn_readfirstlane(nv - (t * 32 + (v >> 2) * 8 + (v & 3)));
            if (hh4 >= lim) s[v] = -INFINITY;
        }
    };
    // Probabilities of a sub-tile, exp2(s) when every row has reference 0 (z), else
    // exp2(s * cw - mref); returns the lane's sum of the bf16-rounded values.
    auto probs = [&](auto z, const f32x16 &s, bf16x8 (&pb)[2]) __attribute__((always_inline)) -> float {
        float l0 = 0.f, l1 = 0.f;
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            float e[8];
#pragma unroll
            for (int jj = 0; jj < 8; ++jj) {
                const float x = s[u * 8 + jj];
                e[jj] = __builtin_amdgcn_exp2f(decltype(z)::value ? x : fmaf(x, cw, -mref));
            }
            pb[u] = bf16x8{(__bf16)e[0], (__bf16)e[1], (__bf16)e[2], (__bf16)e[3],
                           (__bf16)e[4], (__bf16)e[5], (__bf16)e[6], (__bf16)e[7]};
#pragma unroll
            for (int jj = 0; jj < 8; jj += 4) {
                l0 = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{pb[u][jj], pb[u][jj + 1]}, ones, l0, false);
                l1 = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{pb[u][jj + 2], pb[u][jj + 3]}, ones, l1, false);
            }
        }
        return l0 + l1;
    };
    // Chunk-loop variants: every row's reference is 0 (zero), or per-row references (general).
    using general = std::integral_constant<bool, false>;
    using zero = std::integral_constant<bool, true>;
    // Accept the sub-tile's probabilities, or redo them against a new reference
    // (rescaling O and the running sum) when the sub-tile's sum exceeds kSumLimit,
    // the row still has no mass above kTiny, or (zero variant) a row of the wave
    // already left reference 0 in this chunk.
    auto settle = [&](auto z, const f32x16 &s, bf16x8 (&pb)[2], float lh) __attribute__((always_inline)) {
        constexpr bool Z = decltype(z)::value;
        if (__any(!(lh <= kSumLimit) || lrow + lh < kTiny || (Z && mref != 0.f))) {
            float tmax = -INFINITY;
#pragma unroll
            for (int v = 0; v < 16; ++v) tmax = fmaxf(tmax, s[v]);
            tmax = fmaxf(tmax, __shfl_xor(tmax, 32)) * cw;
            // Decisions about the row's mass use the row's running sum: lanes l and
            // l^32 each sum half of the row's keys (one of them may have no mass yet
            // while the row has), and both must take the same reference.
            const float lsum = lrow + __shfl_xor(lrow, 32);
            // The reference only rises, except while the row has no usable mass yet:
            // then it may fall to this sub-tile's maximum, but not below
            // mref + log2(lsum), an upper bound of every earlier logit of the row, so
            // that the rescaled running sums stay at most 1 (finite).
            float mnew = fmaxf(mref, tmax);
            // (log2 of a denormal sum may come back as -inf: -149 bounds it.)
            if (lsum < kTiny) mnew = lsum > 0.f ? fmaxf(tmax, mref + fmaxf(__log2f(lsum), -149.f)) : tmax;
            if (tmax == -INFINITY) mnew = mref;  // a fully masked sub-tile says nothing
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
            lh = probs(general{}, s, pb);
        }
        lrow += lh;
    };

    int nv0 = 0, nv1 = 0;  // real keys of chunks ch and ch+1
    int jnext = -1;        // block of chunk ch+1, read one chunk ahead
    // Chunk ch from slots (ks, vs); first the DMA of chunk ch+1 into (kd, vd), the
    // slots of chunk ch-1 (free since the barrier that ended it).
    auto iter = [&](auto z, int ch, const unsigned char *ks, const unsigned char *vs, unsigned char *kd,
                    unsigned char *vd) __attribute__((always_inline)) {
        if (ch + 1 < C) {
            const int j1 = jnext;
            jnext = ch + 2 < C ? block_of(ch + 2) : -1;
            nv1 = __builtin_amdgcn_readfirstlane(chunk_keys(j1, ch + 1));
            const int row1 = chunk_row0(j1, ch + 1);
            dma_chunk(krs, row1, kd);
            dma_chunk(vrs, row1, vd);
        }
        // Sub-tile 0, then the score MFMAs of sub-tile 1 ahead of the PV MFMAs of
        // sub-tile 0, so that the softmax of sub-tile 1 can start while those run.
        // Partial chunks pay for the mask on a real branch (the empty asm keeps the
        // compiler from if-converting it into every sub-tile).
        f32x16 s0, s1;
        bf16x8 p0[2], p1[2];
        qk(ks, 0, s0);
        if (nv0 < 64) {
            asm volatile("" ::: "memory");
            mask(s0, nv0, 0);
        }
        settle(z, s0, p0, probs(z, s0, p0));
        qk(ks, 1, s1);
        pv(vs, 0, p0);
        if (nv0 < 64) {
            asm volatile("" ::: "memory");
            mask(s1, nv0, 1);
        }
        settle(z, s1, p1, probs(z, s1, p1));
        pv(vs, 1, p1);
        wait_vm_all();    // this wave's loads of chunk ch+1 have landed
        __syncthreads();  // ... and every wave's; chunk ch's slots are no longer read
        nv0 = nv1;
    };

    if (C > 0) {
        {
            const int j0 = block_of(0);
            nv0 = __builtin_amdgcn_readfirstlane(chunk_keys(j0, 0));
            const int row0 = chunk_row0(j0, 0);
            dma_chunk(krs, row0, k_s0);
            dma_chunk(vrs, row0, v_s0);
            jnext = C > 1 ? block_of(1) : -1;
        }
        wait_vm_all();
        __syncthreads();
        {
            // Start with reference 0 only if every row's first 64 logits lie within
            // kStartBand; otherwise use unscaled Q (exact scores) from the start.
            float m0 = -INFINITY;
#pragma unroll
            for (int t = 0; t < 2; ++t) {
                f32x16 s0;
                qk(k_s0, t, s0);
#pragma unroll
                for (int v = 0; v < 16; ++v) m0 = fmaxf(m0, s0[v]);
            }
            m0 = fmaxf(m0, __shfl_xor(m0, 32));
            zref = __all(fabsf(m0) <= kStartBand);
            if (!zref) {
                load_q(false);
                cw = c;
                wait_vm_all();  // Q lands here, not at the first MFMA of every chunk
            }
        }
        int ch = 0;
        // A wave leaves the zero variant (for good) when a row's reference leaves 0;
        // its Q stays pre-scaled (cw = 1), so every score of a row has one form.
        for (;;) {
            if (zref) iter(zero{}, ch, k_s0, v_s0, k_s1, v_s1);
            else iter(general{}, ch, k_s0, v_s0, k_s1, v_s1);
            if (++ch >= C) break;
            if (zref) iter(zero{}, ch, k_s1, v_s1, k_s0, v_s0);
            else iter(general{}, ch, k_s1, v_s1, k_s0, v_s0);
            if (++ch >= C) break;
        }
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
