// Exact attention over kept key blocks (block-sparse, Sec. 3 step (3)) or over
// all key blocks (dense), bf16 inputs, bf16 MFMA products with float32
// accumulation, float32 online softmax.
//
// One workgroup per (head, query block), BQ/32 waves, each wave owning 32 query
// rows. The score tile is computed transposed, S^T = K Q^T, with
// v_mfma_f32_32x32x16_bf16: its accumulator puts one query per lane (lane l and
// l+32 share query l%32, each holding 16 of every 32 keys), so the row max and
// row sum stay in the lane except for one exchange with lane l^32, and the
// probabilities already sit in the B-operand layout of O^T = V^T P^T. V is
// stored transposed in LDS with its keys permuted inside each group of 16 to
// match that layout. K rows and V^T rows are XOR-swizzled in 16-byte chunks so
// that the MFMA operand reads and the tile writes are free of bank conflicts.
//
// Softmax details: exponentials in base 2 with the scale folded in; row sums are
// taken on the bf16-rounded probabilities (the values the PV product uses) with
// packed bf16 dot products; the running maximum is only raised, and O rescaled,
// when some row's maximum grows by more than 2^8, so probabilities stay below
// 256 and most tiles skip the rescale.
//
// Workgroups are numbered so that the 8 XCDs each receive a contiguous range of
// (head, query block) items: neighbouring query blocks of a head share an XCD
// and its L2, where their K/V tiles are re-read.
#include "ress_internal.h"

namespace ress {
namespace {

typedef __bf16 bf16x8 __attribute__((__vector_size__(8 * sizeof(__bf16))));
typedef __bf16 bf16x2 __attribute__((__vector_size__(2 * sizeof(__bf16))));
typedef float f32x16 __attribute__((__vector_size__(16 * sizeof(float))));

constexpr float kRescaleLog2 = 8.0f;  // lazy-rescale threshold, in powers of two

__device__ __forceinline__ unsigned int bf16_bits(float x)
{
    return (unsigned int)__builtin_bit_cast(unsigned short, (__bf16)x);
}

// Position of key kk (0..15) inside its 16-key group of the V^T tile: bits 2 and
// 3 swapped, so that lane half hh reads the 8 keys it holds probabilities for.
__device__ __forceinline__ int vt_pos(int kk) { return (kk & 3) | ((kk & 4) << 1) | ((kk & 8) >> 1); }

// LDS swizzles (16-byte chunk index within a row). A 16-lane phase of a 16-byte
// read and a 32-lane phase of an 8-byte write must hit distinct bank groups of a
// 256-byte bank row.
// K rows are 128 bytes: 16 consecutive rows read one logical chunk.
__device__ __forceinline__ int k_chunk(int row, int ch) { return ch ^ ((row >> 1) & 7); }
// V^T rows (one channel d, BK keys). With 128 keys (16 chunks): reads cover 16
// consecutive channels, writes cover channels 8dc + e for dc = 0..7 and two
// logical chunks; h(d) is a bijection on each 16 consecutive channels and its
// bits 1..3 take 8 distinct values over dc. With 64 keys (8 chunks, two rows
// per bank row) the reads are conflict-free.
template <int BK>
__device__ __forceinline__ int v_chunk(int d, int ch)
{
    if constexpr (BK == 128)
        return ch ^ ((d & 15) ^ (((d >> 3) & 7) << 1));
    else
        return ch ^ ((d >> 1) & 7);
}

template <int BQ, int BK, bool SPARSE>
__global__ void __launch_bounds__(BQ * 2, 2) attn_kernel(const AttnParams p)
{
    constexpr int T = BQ * 2;         // threads
    constexpr int NT = BK / 32;       // 32-key sub-tiles per key block
    constexpr int KU = BK * 8 / T;    // 16-byte K pieces per thread
    constexpr int VUNITS = BK * 2;    // 4-key x 8-channel V pieces per tile
    constexpr int VU = (VUNITS + T - 1) / T;
    constexpr int VROW = BK * 2;      // bytes per V^T row
    __shared__ __attribute__((aligned(16))) unsigned char k_lds[BK * 128];
    __shared__ __attribute__((aligned(16))) unsigned char v_lds[kD * VROW];

    const int xcd = blockIdx.x & 7, local = blockIdx.x >> 3;
    const int item = xcd * p.items_per_xcd + local;
    if (item >= p.H * p.n_qb) return;
    const int h = item / p.n_qb;
    const int i = p.n_qb - 1 - item % p.n_qb;  // last query blocks first (they may be dense)
    const int N = p.N, n_kb = p.n_kb;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int hh = lane >> 5, ql = lane & 31;
    const int q0 = i * BQ + wave * 32 + ql;
    const size_t head = (size_t)h * N;

    bf16x8 qf[4];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
        if (q0 < N)
            qf[kk] = *reinterpret_cast<const bf16x8 *>(p.q + (head + q0) * kD + kk * 16 + hh * 8);
        else
            qf[kk] = bf16x8{};
    }

    int ntiles;
    const int32_t *list = nullptr;
    if constexpr (SPARSE) {
        const size_t row = (size_t)h * p.n_qb + i;
        ntiles = min(max(p.kept_count[row], 0), n_kb);
        list = p.kept_idx + row * n_kb;
    } else {
        ntiles = n_kb;
    }

    uint4 kreg[KU];
    uint4 vreg[VU][4];
    auto tile_index = [&](int it) -> int {
        if constexpr (SPARSE) return list[it];
        else return it;
    };
    auto load_tile = [&](int j) {
        const bool valid = j >= 0 && j < n_kb;
        const size_t base = (size_t)(valid ? j : 0) * BK;
#pragma unroll
        for (int u = 0; u < KU; ++u) {
            const int unit = tid + u * T, kr = unit >> 3, ch = unit & 7;
            const size_t tok = base + kr;
            kreg[u] = (valid && tok < (size_t)N)
                          ? *reinterpret_cast<const uint4 *>(p.k + (head + tok) * kD + ch * 8)
                          : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int u = 0; u < VU; ++u) {
            const int unit = tid + u * T, kg = unit >> 3, dc = unit & 7;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const size_t tok = base + kg * 4 + r;
                vreg[u][r] = (unit < VUNITS && valid && tok < (size_t)N)
                                 ? *reinterpret_cast<const uint4 *>(p.v + (head + tok) * kD + dc * 8)
                                 : make_uint4(0, 0, 0, 0);
            }
        }
    };
    auto store_tile = [&]() {
#pragma unroll
        for (int u = 0; u < KU; ++u) {
            const int unit = tid + u * T, kr = unit >> 3, ch = unit & 7;
            *reinterpret_cast<uint4 *>(k_lds + kr * 128 + (k_chunk(kr, ch) << 4)) = kreg[u];
        }
#pragma unroll
        for (int u = 0; u < VU; ++u) {
            const int unit = tid + u * T;
            if (unit >= VUNITS) continue;
            const int kg = unit >> 3, dc = unit & 7;
            const int pos = (kg >> 2) * 16 + vt_pos((kg & 3) * 4);  // V^T position of key 4*kg
            const unsigned int w[4][4] = {{vreg[u][0].x, vreg[u][0].y, vreg[u][0].z, vreg[u][0].w},
                                          {vreg[u][1].x, vreg[u][1].y, vreg[u][1].z, vreg[u][1].w},
                                          {vreg[u][2].x, vreg[u][2].y, vreg[u][2].z, vreg[u][2].w},
                                          {vreg[u][3].x, vreg[u][3].y, vreg[u][3].z, vreg[u][3].w}};
#pragma unroll
            for (int e = 0; e < 4; ++e) {  // channels 2e, 2e+1 of this unit
                // v_perm_b32 picks the low (even channel) or high (odd channel) halves of
                // two keys' words: {key b low half, key a low half} etc.
                const unsigned int lo01 = __builtin_amdgcn_perm(w[1][e], w[0][e], 0x05040100u);
                const unsigned int lo23 = __builtin_amdgcn_perm(w[3][e], w[2][e], 0x05040100u);
                const unsigned int hi01 = __builtin_amdgcn_perm(w[1][e], w[0][e], 0x07060302u);
                const unsigned int hi23 = __builtin_amdgcn_perm(w[3][e], w[2][e], 0x07060302u);
                const int d0 = dc * 8 + 2 * e, d1 = d0 + 1;
                *reinterpret_cast<uint2 *>(v_lds + d0 * VROW + (v_chunk<BK>(d0, pos >> 3) << 4) + (pos & 7) * 2) =
                    make_uint2(lo01, lo23);
                *reinterpret_cast<uint2 *>(v_lds + d1 * VROW + (v_chunk<BK>(d1, pos >> 3) << 4) + (pos & 7) * 2) =
                    make_uint2(hi01, hi23);
            }
        }
    };

    const float c = p.scale_log2;
    float mref = -INFINITY;  // running reference maximum of this lane's query row
    float lrow = 0.f;
    f32x16 acc_o[2];
#pragma unroll
    for (int dh = 0; dh < 2; ++dh)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc_o[dh][v] = 0.f;
    const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};

    // One key block: scores, online softmax, PV; nvalid < BK masks a partial block.
    auto process = [&](int nvalid) {
        f32x16 s[NT];
#pragma unroll
        for (int t = 0; t < NT; ++t) {
#pragma unroll
            for (int v = 0; v < 16; ++v) s[t][v] = 0.f;
            const int kr = t * 32 + ql;
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) {
                const int ch = kk * 2 + hh;
                const bf16x8 a = *reinterpret_cast<const bf16x8 *>(k_lds + kr * 128 + (k_chunk(kr, ch) << 4));
                s[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[kk], s[t], 0, 0, 0);
            }
        }
        if (nvalid < BK) {
            // A real branch: only partial blocks pay for the mask (the empty asm
            // keeps the compiler from if-converting it into every tile).
            asm volatile("" ::: "memory");
#pragma unroll
            for (int t = 0; t < NT; ++t)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int key = t * 32 + (v >> 2) * 8 + hh * 4 + (v & 3);
                    if (key >= nvalid) s[t][v] = -INFINITY;
                }
        }
        float tmax = -INFINITY;
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
            for (int v = 0; v < 16; ++v) tmax = fmaxf(tmax, s[t][v]);
        tmax = fmaxf(tmax, __shfl_xor(tmax, 32));
        // Raise the reference maximum only when this tile exceeds it by more than
        // 2^kRescaleLog2 in probability (or on the first keys of the row).
        const bool raise = tmax > mref && (mref == -INFINITY || (tmax - mref) * c > kRescaleLog2);
        if (__any(raise)) {
            const float mnew = raise ? tmax : mref;
            const float alpha = mref == -INFINITY ? 0.f : __builtin_amdgcn_exp2f((mref - mnew) * c);
            lrow *= alpha;
#pragma unroll
            for (int dh = 0; dh < 2; ++dh)
#pragma unroll
                for (int v = 0; v < 16; ++v) acc_o[dh][v] *= alpha;
            mref = mnew;
        }
        const float mc = mref == -INFINITY ? 0.f : mref * c;
        bf16x8 pb[NT][2];
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                float e[8];
#pragma unroll
                for (int jj = 0; jj < 8; ++jj) e[jj] = __builtin_amdgcn_exp2f(fmaf(s[t][u * 8 + jj], c, -mc));
                pb[t][u] = bf16x8{(__bf16)e[0], (__bf16)e[1], (__bf16)e[2], (__bf16)e[3],
                                  (__bf16)e[4], (__bf16)e[5], (__bf16)e[6], (__bf16)e[7]};
#pragma unroll
                for (int jj = 0; jj < 8; jj += 2)
                    lrow = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{pb[t][u][jj], pb[t][u][jj + 1]}, ones, lrow,
                                                           false);
            }
        // O^T += V^T P^T, 16 keys per MFMA.
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                const int chunk = (2 * t + u) * 2 + hh;
#pragma unroll
                for (int dh = 0; dh < 2; ++dh) {
                    const int dim = dh * 32 + ql;
                    const bf16x8 a =
                        *reinterpret_cast<const bf16x8 *>(v_lds + dim * VROW + (v_chunk<BK>(dim, chunk) << 4));
                    acc_o[dh] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[t][u], acc_o[dh], 0, 0, 0);
                }
            }
    };
    if (ntiles > 0) load_tile(tile_index(0));
    for (int it = 0; it < ntiles; ++it) {
        const int j = tile_index(it);
        const int nvalid = (j >= 0 && j < n_kb) ? min(BK, N - j * BK) : 0;
        __syncthreads();
        store_tile();
        __syncthreads();
        if (it + 1 < ntiles) load_tile(tile_index(it + 1));
        process(nvalid);
    }

    // Each lane summed half of its row's keys; lanes l and l^32 share the row.
    const float ltot = lrow + __shfl_xor(lrow, 32);
    const float inv = ltot > 0.f ? 1.f / ltot : 0.f;
    if (q0 < N) {
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
    const dim3 grid((unsigned)(8 * p.items_per_xcd)), block(BQ * 2);
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
