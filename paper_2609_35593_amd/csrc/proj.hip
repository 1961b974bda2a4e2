// The two steps on either side of the path, as bf16 MFMA GEMMs with fused
// epilogues (token-major activations, nn.Linear-style [out][in] weights):
//  - QKV projection, [Q K V] = X W_qkv^T, written head-major [H][N][64], with the
//    block mean pooling of Sec. 3 step (1) taken from the bf16-rounded outputs in
//    the epilogue (plus c_j = Vbar_j^T M_h Vbar_j for Eq. 9), so the selection never reads
//    Q, K, V again;
//  - output projection and residual add, R' = R + concat_h(O_h) W_O^T, reading
//    the head-major attention output directly (the k-slice of one 64-wide k-tile
//    is one head), into a bf16 or a float32 residual stream.
//
// Tiling: 256 x 256 output tile per workgroup, k-tiles of 64, 8 waves, each wave
// a 64 x 128 sub-tile of 2 x 4 v_mfma_f32_32x32x16_bf16 accumulators (lane l
// holds output column l%32 of each 32 x 32 block, 16 of its rows). A and B
// k-tiles (256 rows x 128 bytes each) move global -> LDS with global_load_lds in
// two slots; rows keep their 16-byte chunks XOR-swizzled per row, applied by
// choosing each lane's source chunk. Rows of A past the last token repeat the
// last token and are excluded from every output.
#include "ress_internal.h"

namespace ress {
namespace {

typedef __bf16 bf16x8 __attribute__((__vector_size__(8 * sizeof(__bf16))));
typedef float f32x16 __attribute__((__vector_size__(16 * sizeof(float))));
typedef __attribute__((address_space(3))) void lds_void;

constexpr int kThreads = 512;
constexpr int BM = 256, BN = 256;   // output tile
constexpr int kTileBytes = 256 * 128;  // one operand k-tile: 256 rows x 64 bf16
constexpr int kStageRow = BN * 2 + 16;  // bf16 staging row of the output tile (padded)
constexpr int kOperandBytes = 2 * 2 * kTileBytes;                        // two slots of A and B
constexpr int kEpilogue0 = BM * kStageRow + 2 * 4 * BN * (int)sizeof(double);  // tile + sums + means
constexpr int kEpilogue1 = 128 * (BN + 4) * (int)sizeof(float);         // half a float32 tile
constexpr int kSmem = kEpilogue0 > kOperandBytes ? (kEpilogue0 > kEpilogue1 ? kEpilogue0 : kEpilogue1)
                                                 : (kOperandBytes > kEpilogue1 ? kOperandBytes : kEpilogue1);
static_assert(kSmem <= 160 * 1024, "LDS per workgroup");

__device__ __forceinline__ int swz(int row) { return (((row >> 1) & 1) << 2) | ((row >> 2) & 3); }
__device__ __forceinline__ void wait_vm_all() { __builtin_amdgcn_s_waitcnt(0x0F70); }  // vmcnt(0)

__device__ __forceinline__ float bf16_round(float x) { return (float)(__bf16)x; }
__device__ __forceinline__ unsigned int bf16_bits(float x)
{
    return (unsigned int)__builtin_bit_cast(unsigned short, (__bf16)x);
}

// 0: QKV projection + pooling, 1: output projection + bf16 residual, 2: output
// projection + float32 residual.
template <int MODE>
__global__ void __launch_bounds__(kThreads, 1) proj_kernel(const ProjParams p)
{
    __shared__ __attribute__((aligned(1024))) unsigned char smem[kSmem];  // operand slots, then epilogue staging
    auto slot_ptr = [&](int slot, int b_operand) __attribute__((always_inline)) {
        return smem + (2 * slot + b_operand) * kTileBytes;
    };
    const int xcd = blockIdx.x & 7, local = blockIdx.x >> 3;
    const int item = xcd * p.items_per_xcd + local;
    if (item >= p.m_tiles * p.n_tiles) return;
    // Tile order within an XCD's range: groups of 8 M tiles, N-major inside a group,
    // so the ~32 tiles an XCD runs at once share 8 A and ~4 B k-slices in its L2
    // (measured: 4-6% faster than sweeping all N tiles of one M tile at a time).
    constexpr int GM = 8;
    const int grp = item / (GM * p.n_tiles), rem = item % (GM * p.n_tiles);
    const int gmc = min(GM, p.m_tiles - grp * GM);  // M tiles in this group (fewer in the last)
    const int mt = grp * GM + rem % gmc, nt = rem / gmc;
    const int T = p.T, dm = 64 * p.H, KT = p.H;              // k-tiles of 64: one head each
    const int m0 = mt * BM, n0 = nt * BN;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave & 3, wn = wave >> 2;  // rows 64 wm, columns 128 wn of the tile
    const int hh = lane >> 5, ql = lane & 31;

    // DMA: each thread moves 4 chunks of A and 4 of B per k-tile; instruction u of
    // wave w fills rows 8 (8u + w) .. +7 (lane / 8), physical chunk lane & 7.
    int arow[4], brow[4];
    unsigned int chunk_off[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
        const int r = (u * 8 + wave) * 8 + (lane >> 3);
        arow[u] = min(m0 + r, T - 1);
        brow[u] = n0 + r;
        chunk_off[u] = (unsigned int)(((lane & 7) ^ swz(r)) << 4);
    }
    auto dma = [&](int kt, int slot) __attribute__((always_inline)) {
        unsigned char *a_dst = slot_ptr(slot, 0), *b_dst = slot_ptr(slot, 1);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const uint16_t *asrc = MODE == 0 ? p.a + (size_t)arow[u] * dm + kt * 64
                                             : p.a + ((size_t)kt * T + arow[u]) * 64;
            const uint16_t *bsrc = p.w + (size_t)brow[u] * dm + kt * 64;
            __builtin_amdgcn_global_load_lds((const void *)((const unsigned char *)asrc + chunk_off[u]),
                                             (lds_void *)(a_dst + (u * 8 + wave) * 1024), 16, 0, 0);
            __builtin_amdgcn_global_load_lds((const void *)((const unsigned char *)bsrc + chunk_off[u]),
                                             (lds_void *)(b_dst + (u * 8 + wave) * 1024), 16, 0, 0);
        }
    };
    // Operand read offsets: row, logical chunk 2 kk + hh.
    int aoff[2][4], boff[4][4];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
#pragma unroll
        for (int mi = 0; mi < 2; ++mi) {
            const int r = 64 * wm + 32 * mi + ql;
            aoff[mi][kk] = r * 128 + (((2 * kk + hh) ^ swz(r)) << 4);
        }
#pragma unroll
        for (int ni = 0; ni < 4; ++ni) {
            const int r = 128 * wn + 32 * ni + ql;
            boff[ni][kk] = r * 128 + (((2 * kk + hh) ^ swz(r)) << 4);
        }
    }

    f32x16 acc[2][4];
#pragma unroll
    for (int mi = 0; mi < 2; ++mi)
#pragma unroll
        for (int ni = 0; ni < 4; ++ni)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[mi][ni][v] = 0.f;

    // Operand fragments are read one k-step (16) ahead into two register sets, so
    // the LDS latency of step kk+1 hides behind the 8 MFMAs of step kk; the first
    // step of the next k-tile is read right after the barrier, beside the MFMAs of
    // the last step of this one.
    bf16x8 fa[2][2], fb[2][4];
    auto read_frags = [&](int slot, int kk, int buf) __attribute__((always_inline)) {
        const unsigned char *A = slot_ptr(slot, 0), *B = slot_ptr(slot, 1);
#pragma unroll
        for (int mi = 0; mi < 2; ++mi) fa[buf][mi] = *reinterpret_cast<const bf16x8 *>(A + aoff[mi][kk]);
#pragma unroll
        for (int ni = 0; ni < 4; ++ni) fb[buf][ni] = *reinterpret_cast<const bf16x8 *>(B + boff[ni][kk]);
    };
    auto mfmas = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
        for (int mi = 0; mi < 2; ++mi)
#pragma unroll
            for (int ni = 0; ni < 4; ++ni)
                acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[buf][mi], fb[buf][ni], acc[mi][ni], 0, 0, 0);
    };

    dma(0, 0);
    wait_vm_all();
    __syncthreads();
    read_frags(0, 0, 0);
    for (int kt = 0; kt < KT; ++kt) {
        const int slot = kt & 1;
        if (kt + 1 < KT) dma(kt + 1, slot ^ 1);
#pragma unroll
        for (int kk = 0; kk < 3; ++kk) {
            read_frags(slot, kk + 1, (kk + 1) & 1);
            mfmas(kk & 1);
        }
        wait_vm_all();    // k-tile kt + 1 has landed (this wave's part) ...
        __syncthreads();  // ... every wave's, and slot kt & 1 is no longer read
        if (kt + 1 < KT) read_frags(slot ^ 1, 0, 0);
        mfmas(1);         // step 3 of this k-tile
    }

    // Accumulator element (mi, ni, v) of this lane: tile row and column.
    auto row_of = [&](int mi, int v) __attribute__((always_inline)) {
        return 64 * wm + 32 * mi + (v >> 2) * 8 + hh * 4 + (v & 3);
    };
    auto col_of = [&](int ni) __attribute__((always_inline)) { return 128 * wn + 32 * ni + ql; };

    if constexpr (MODE == 0) {
        // Round to the bf16 outputs; everything below uses the rounded values.
#pragma unroll
        for (int mi = 0; mi < 2; ++mi)
#pragma unroll
            for (int ni = 0; ni < 4; ++ni)
#pragma unroll
                for (int v = 0; v < 16; ++v) acc[mi][ni][v] = bf16_round(acc[mi][ni][v]);

        // Pooling: column sums over this wave's 64 rows (valid tokens only), in
        // float64 (exact for bf16 values of moderate span).
        double csum[4];
#pragma unroll
        for (int ni = 0; ni < 4; ++ni) {
            double s = 0.0;
#pragma unroll
            for (int mi = 0; mi < 2; ++mi)
#pragma unroll
                for (int v = 0; v < 16; ++v)
                    s += (m0 + row_of(mi, v) < T) ? (double)acc[mi][ni][v] : 0.0;
            csum[ni] = s + __shfl_xor(s, 32);
        }
        // Output tile as bf16, staged row-major in LDS (the operand slots are free).
        unsigned char *stage = smem;
#pragma unroll
        for (int mi = 0; mi < 2; ++mi)
#pragma unroll
            for (int ni = 0; ni < 4; ++ni)
#pragma unroll
                for (int v = 0; v < 16; ++v)
                    *reinterpret_cast<unsigned short *>(stage + row_of(mi, v) * kStageRow + col_of(ni) * 2) =
                        (unsigned short)bf16_bits(acc[mi][ni][v]);
        // Per-wave column sums next to it: psum[wm][column].
        double *psum = reinterpret_cast<double *>(stage + BM * kStageRow);
        if (hh == 0) {
#pragma unroll
            for (int ni = 0; ni < 4; ++ni) psum[wm * BN + col_of(ni)] = csum[ni];
        }
        __syncthreads();

        // Head-major bf16 stores: 16 bytes (8 channels of one token) per thread and step.
        const int which = n0 / dm;  // 0: Q, 1: K, 2: V (a tile never straddles two)
        uint16_t *dst = which == 0 ? p.q : which == 1 ? p.k : p.v;
        for (int e = tid; e < BM * (BN / 8); e += kThreads) {
            const int r = e >> 5, c8 = (e & 31) * 8;
            const int t = m0 + r;
            if (t >= T) continue;
            const int f = n0 - which * dm + c8, h = f >> 6, d = f & 63;
            *reinterpret_cast<uint4 *>(dst + ((size_t)h * T + t) * 64 + d) =
                *reinterpret_cast<const uint4 *>(stage + r * kStageRow + c8 * 2);
        }

        // Block means: a block of b rows is 1 (b = 64) or 2 (b = 128) wave row groups.
        const int b = which == 0 ? p.bq : p.bk;
        const int groups = b / 64;
        double *vmean = psum + 4 * BN;  // Vbar of each (block, column) of the tile, for U
        for (int e = tid; e < (BM / b) * BN; e += kThreads) {
            const int blk = e / BN, c = e % BN;
            const int t0 = m0 + blk * b;
            if (t0 >= T) continue;
            double s = 0.0;
            for (int g = 0; g < groups; ++g) s += psum[(blk * groups + g) * BN + c];
            const double mean = s / (double)min(b, T - t0);
            const int blk_g = t0 / b;
            const int f = n0 - which * dm + c, h = f >> 6, d = f & 63;
            if (which == 0) {
                p.pooled.qbar[((size_t)h * p.n_qb + blk_g) * 64 + d] = mean;
            } else if (which == 1) {
                p.pooled.kbar[((size_t)h * p.n_kb + blk_g) * 64 + d] = mean;
            } else {
                p.pooled.vbar[((size_t)h * p.n_kb + blk_g) * 64 + d] = mean;
                vmean[blk * BN + c] = mean;
            }
        }
        if (which == 2) {
            // c_j = Vbar_j . (M_h Vbar_j): one wave per (block, head) of the tile, lane <->
            // channel, in the same order as the pooling pass of the selection.
            __syncthreads();
            const int nblk = BM / b, pairs = nblk * (BN / 64);
            for (int pr = wave; pr < pairs; pr += kThreads / 64) {
                const int blk = pr / (BN / 64), hl = pr % (BN / 64);
                const int t0 = m0 + blk * b;
                if (t0 >= T) continue;
                const int h = (n0 - 2 * dm) / 64 + hl;
                const float *Mrow = p.gram + ((size_t)h * 64 + lane) * 64;
                const double *vb = vmean + blk * BN + hl * 64;
                double u = 0.0;
#pragma unroll 8
                for (int c = 0; c < 64; ++c) u = fma((double)Mrow[c], vb[c], u);
                double cj = u * vb[lane];
#pragma unroll
                for (int o = 32; o >= 1; o >>= 1) cj += __shfl_xor(cj, o);
                if (lane == 0) p.pooled.cT[(size_t)h * p.n_kb + t0 / b] = cj;
            }
        }
    } else {
        // R' = R + acc (bf16 stream: rounded once); the float32 tile is staged in two
        // halves of 128 rows (128 KB each) and combined with R in 16-byte pieces.
        float *stage = reinterpret_cast<float *>(smem);
        constexpr int SR = BN + 4;  // padded float row
        for (int half = 0; half < 2; ++half) {
            if ((wm >> 1) == half) {
#pragma unroll
                for (int mi = 0; mi < 2; ++mi)
#pragma unroll
                    for (int ni = 0; ni < 4; ++ni)
#pragma unroll
                        for (int v = 0; v < 16; ++v)
                            stage[(row_of(mi, v) - 128 * half) * SR + col_of(ni)] = acc[mi][ni][v];
            }
            __syncthreads();
            if constexpr (MODE == 1) {
                for (int e = tid; e < 128 * (BN / 8); e += kThreads) {
                    const int r = e >> 5, c8 = (e & 31) * 8;
                    const int t = m0 + 128 * half + r;
                    if (t >= T) continue;
                    const size_t off = (size_t)t * dm + n0 + c8;
                    const uint4 rin = *reinterpret_cast<const uint4 *>(p.resid_in + off);
                    const unsigned int w[4] = {rin.x, rin.y, rin.z, rin.w};
                    unsigned int o[4];
#pragma unroll
                    for (int q2 = 0; q2 < 4; ++q2) {
                        const float lo = __uint_as_float(w[q2] << 16) + stage[r * SR + c8 + 2 * q2];
                        const float hi = __uint_as_float(w[q2] & 0xffff0000u) + stage[r * SR + c8 + 2 * q2 + 1];
                        o[q2] = bf16_bits(lo) | (bf16_bits(hi) << 16);
                    }
                    *reinterpret_cast<uint4 *>(p.resid_out + off) = make_uint4(o[0], o[1], o[2], o[3]);
                }
            } else {
                // float32 stream: R' = R + acc, one float32 add per element, 16 bytes at a time.
                for (int e = tid; e < 128 * (BN / 4); e += kThreads) {
                    const int r = e >> 6, c4 = (e & 63) * 4;
                    const int t = m0 + 128 * half + r;
                    if (t >= T) continue;
                    const size_t off = (size_t)t * dm + n0 + c4;
                    const float4 rin = *reinterpret_cast<const float4 *>(p.resid_in_f32 + off);
                    const float *st = stage + r * SR + c4;
                    *reinterpret_cast<float4 *>(p.resid_out_f32 + off) =
                        make_float4(rin.x + st[0], rin.y + st[1], rin.z + st[2], rin.w + st[3]);
                }
            }
            __syncthreads();
        }
    }
}

}  // namespace

hipError_t launch_proj(const ProjParams &p, hipStream_t s)
{
    if (p.m_tiles == 0 || p.n_tiles == 0) return hipSuccess;
    const dim3 grid((unsigned)(8 * p.items_per_xcd)), block(kThreads);
    if (p.mode == 0)
        hipLaunchKernelGGL(proj_kernel<0>, grid, block, 0, s, p);
    else if (p.mode == 1)
        hipLaunchKernelGGL(proj_kernel<1>, grid, block, 0, s, p);
    else
        hipLaunchKernelGGL(proj_kernel<2>, grid, block, 0, s, p);
    return hipGetLastError();
}

}  // namespace ress
