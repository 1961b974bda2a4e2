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
// that the MFMA operand reads are free of bank conflicts.
//
// Workgroups are numbered so that the 8 XCDs each receive a contiguous range of
// (head, query block) items: neighbouring query blocks of a head share an XCD
// and its L2, where their K/V tiles are re-read.
#include "ress_internal.h"

namespace ress {
namespace {

typedef __bf16 bf16x8 __attribute__((__vector_size__(8 * sizeof(__bf16))));
typedef float f32x16 __attribute__((__vector_size__(16 * sizeof(float))));

__device__ __forceinline__ unsigned int bf16_bits(float x)
{
    return (unsigned int)__builtin_bit_cast(unsigned short, (__bf16)x);
}

// Position of key kk (0..15) inside its 16-key group of the V^T tile: bits 2 and
// 3 swapped, so that lane half hh reads the 8 keys it holds probabilities for.
__device__ __forceinline__ int vt_pos(int kk) { return (kk & 3) | ((kk & 4) << 1) | ((kk & 8) >> 1); }

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
            *reinterpret_cast<uint4 *>(k_lds + kr * 128 + ((ch ^ (kr & 7)) << 4)) = kreg[u];
        }
#pragma unroll
        for (int u = 0; u < VU; ++u) {
            const int unit = tid + u * T;
            if (unit >= VUNITS) continue;
            const int kg = unit >> 3, dc = unit & 7;
            const int pos = (kg >> 2) * 16 + vt_pos((kg & 3) * 4);  // position of key 4*kg
            const unsigned int w[4][4] = {{vreg[u][0].x, vreg[u][0].y, vreg[u][0].z, vreg[u][0].w},
                                          {vreg[u][1].x, vreg[u][1].y, vreg[u][1].z, vreg[u][1].w},
                                          {vreg[u][2].x, vreg[u][2].y, vreg[u][2].z, vreg[u][2].w},
                                          {vreg[u][3].x, vreg[u][3].y, vreg[u][3].z, vreg[u][3].w}};
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int dim = dc * 8 + e, sh = (e & 1) * 16;
                const unsigned int a0 = (w[0][e >> 1] >> sh) & 0xffffu, a1 = (w[1][e >> 1] >> sh) & 0xffffu;
                const unsigned int a2 = (w[2][e >> 1] >> sh) & 0xffffu, a3 = (w[3][e >> 1] >> sh) & 0xffffu;
                const int chunk = (pos >> 3) ^ (dim & 7);
                *reinterpret_cast<uint2 *>(v_lds + dim * VROW + (chunk << 4) + (pos & 7) * 2) =
                    make_uint2(a0 | (a1 << 16), a2 | (a3 << 16));
            }
        }
    };

    const float c = p.scale_log2;
    float mrow = -INFINITY, lrow = 0.f;
    f32x16 acc_o[2];
#pragma unroll
    for (int dh = 0; dh < 2; ++dh)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc_o[dh][v] = 0.f;

    if (ntiles > 0) load_tile(tile_index(0));
    for (int it = 0; it < ntiles; ++it) {
        const int j = tile_index(it);
        const int nvalid = (j >= 0 && j < n_kb) ? min(BK, N - j * BK) : 0;
        __syncthreads();
        store_tile();
        __syncthreads();
        if (it + 1 < ntiles) load_tile(tile_index(it + 1));

        // S^T = K Q^T, one 32x32 accumulator per 32-key sub-tile.
        f32x16 s[NT];
#pragma unroll
        for (int t = 0; t < NT; ++t) {
#pragma unroll
            for (int v = 0; v < 16; ++v) s[t][v] = 0.f;
            const int kr = t * 32 + ql;
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) {
                const int ch = kk * 2 + hh;
                const bf16x8 a = *reinterpret_cast<const bf16x8 *>(k_lds + kr * 128 + ((ch ^ (kr & 7)) << 4));
                s[t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qf[kk], s[t], 0, 0, 0);
            }
        }
        if (nvalid < BK) {
#pragma unroll
            for (int t = 0; t < NT; ++t)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int key = t * 32 + (v >> 2) * 8 + hh * 4 + (v & 3);
                    if (key >= nvalid) s[t][v] = -INFINITY;
                }
        }
        // Online softmax (base 2, scale folded into the exponent).
        float tmax = -INFINITY;
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
            for (int v = 0; v < 16; ++v) tmax = fmaxf(tmax, s[t][v]);
        tmax = fmaxf(tmax, __shfl_xor(tmax, 32));
        const float mnew = fmaxf(mrow, tmax);
        const float mc = mnew == -INFINITY ? 0.f : mnew * c;
        const float alpha = mrow == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mrow * c - mc);
        float psum = 0.f;
        bf16x8 pb[NT][2];
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                float e[8];
#pragma unroll
                for (int jj = 0; jj < 8; ++jj) {
                    e[jj] = __builtin_amdgcn_exp2f(fmaf(s[t][u * 8 + jj], c, -mc));
                    psum += e[jj];
                }
                pb[t][u] = bf16x8{(__bf16)e[0], (__bf16)e[1], (__bf16)e[2], (__bf16)e[3],
                                  (__bf16)e[4], (__bf16)e[5], (__bf16)e[6], (__bf16)e[7]};
            }
        lrow = lrow * alpha + psum;
        mrow = mnew;
#pragma unroll
        for (int dh = 0; dh < 2; ++dh)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc_o[dh][v] *= alpha;
        // O^T += V^T P^T, 16 keys per MFMA.
#pragma unroll
        for (int t = 0; t < NT; ++t)
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                const int chunk = (2 * t + u) * 2 + hh;
#pragma unroll
                for (int dh = 0; dh < 2; ++dh) {
                    const int dim = dh * 32 + ql;
                    const bf16x8 a = *reinterpret_cast<const bf16x8 *>(
                        v_lds + dim * VROW + ((chunk ^ (dim & 7)) << 4));
                    acc_o[dh] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[t][u], acc_o[dh], 0, 0, 0);
                }
            }
    }

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
