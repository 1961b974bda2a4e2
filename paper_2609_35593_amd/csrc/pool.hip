// Block mean pooling of Q, K and V (the coarse block grid of Sec. 3, step (1)),
// plus c_j = Vbar_j^T M_h Vbar_j for the drift scores (Eq. 9).
//
// One wave per pooled block; a workgroup holds 4 waves that pool 4 consecutive
// blocks of the same head and tensor, so that for V the head's M_h is staged in
// LDS once for 4 blocks. Outputs are row-major (lane t writes channel t). Lane l
// streams the 16-byte chunk l/8 (channels 8(l/8)..+7) of
// tokens l%8, l%8 + 8, ...: every load instruction of a wave covers 8 whole
// 128-byte token rows, and a block is one batch of independent loads. Partial
// sums are float64; the 8 lanes of a chunk are combined with a fixed butterfly,
// after which lane t holds channel t. A float64 sum of bf16 values is exact
// unless the block's values span more than about 2^40 in magnitude, so the
// means equal the float64 means computed in any order. This pass is the only
// part of the selection that reads Q, K, V from HBM.
#include "ress_internal.h"

namespace ress {
namespace {

typedef unsigned int v4u32 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;  // blocks per workgroup

// Sum over the wave by a fixed butterfly (commutative adds: identical in every lane).
__device__ __forceinline__ double wave_sum(double x)
{
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o);
    return x;
}

__device__ __forceinline__ void accum_bf16x8(double (&acc)[8], uint4 w)
{
    const unsigned int u[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        acc[2 * e] += (double)__uint_as_float(u[e] << 16);
        acc[2 * e + 1] += (double)__uint_as_float(u[e] & 0xffff0000u);
    }
}

// Mean over rows [row0, row0 + cnt) (cnt <= 128) of x[.][64]; lane t of the wave
// returns channel t.
__device__ __forceinline__ double wave_block_mean(const uint16_t *__restrict__ x, size_t row0, int cnt)
{
    const int lane = threadIdx.x & 63, chunk = lane >> 3, sub = lane & 7;
    double acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    // All 16 loads are issued unconditionally (tokens past the block's end read its
    // last token, cnt >= 1) and zeroed afterwards, so that a wave has its whole
    // block in flight at once. Q, K and V are read once here: non-temporal loads,
    // which leave the caches' resident lines in place (measured: with the caches
    // full of dirty lines, the pass takes ~45 us less at 32 views).
    const uint16_t *base = x + row0 * kD + chunk * 8;
    uint4 w[16];
#pragma unroll
    for (int r = 0; r < 16; ++r)
        w[r] = __builtin_bit_cast(uint4, __builtin_nontemporal_load(reinterpret_cast<const v4u32 *>(
                                             base + (size_t)min(sub + 8 * r, cnt - 1) * kD)));
#pragma unroll
    for (int r = 0; r < 16; ++r)
        if (sub + 8 * r >= cnt) w[r] = make_uint4(0, 0, 0, 0);
#pragma unroll
    for (int r = 0; r < 16; ++r) accum_bf16x8(acc, w[r]);
#pragma unroll
    for (int o = 1; o <= 4; o <<= 1)
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[e] += __shfl_xor(acc[e], o);
    // Every lane of a chunk now holds the chunk's 8 channel sums; lane t keeps
    // channel t = 8 * chunk + (t & 7).
    double s = acc[0];
#pragma unroll
    for (int e = 1; e < 8; ++e) s = (sub == e) ? acc[e] : s;
    return s / (double)cnt;
}

__global__ void __launch_bounds__(kThreads) pool_kernel(const PoolParams p)
{
    __shared__ float Ms[kD * (kD + 1)];       // M_h, padded rows (V workgroups)
    __shared__ double vb[kWaves][kD];         // each wave's Vbar_j
    const int t = threadIdx.x, lane = t & 63;
    const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
    const int gq = (p.n_qb + kWaves - 1) / kWaves, gk = (p.n_kb + kWaves - 1) / kWaves;
    const int per_head = gq + 2 * gk;
    const int h = blockIdx.x / per_head, g = blockIdx.x % per_head;

    if (g < gq) {  // query blocks: row-major output only
        const int i = g * kWaves + wave;
        if (i >= p.n_qb) return;
        const int lo = i * p.bq, cnt = min(p.bq, p.N - lo);
        p.out.qbar[((size_t)h * p.n_qb + i) * kD + lane] = wave_block_mean(p.q, (size_t)h * p.N + lo, cnt);
        return;
    }
    const bool is_v = g >= gq + gk;
    const int j0 = (is_v ? g - gq - gk : g - gq) * kWaves;
    const int j = j0 + wave;
    constexpr int MPT = kD * kD / 4 / kThreads;  // float4 pieces of M_h per thread
    float4 mreg[MPT];
    if (is_v) {  // issued before the block loads, stored to LDS after them
        const float4 *Mh = reinterpret_cast<const float4 *>(p.gram + (size_t)h * kD * kD);
#pragma unroll
        for (int u = 0; u < MPT; ++u) mreg[u] = Mh[u * kThreads + t];
    }
    if (j < p.n_kb) {
        const int lo = j * p.bk, cnt = min(p.bk, p.N - lo);
        const double mean = wave_block_mean(is_v ? p.v : p.k, (size_t)h * p.N + lo, cnt);
        (is_v ? p.out.vbar : p.out.kbar)[((size_t)h * p.n_kb + j) * kD + lane] = mean;
        if (is_v) vb[wave][lane] = mean;
    }
    if (is_v) {  // M_h row r, column c at r * 65 + c
#pragma unroll
        for (int u = 0; u < MPT; ++u) {
            const int e = 4 * (u * kThreads + t), r = e >> 6, c = e & 63;
            float *dst = Ms + r * (kD + 1) + c;
            dst[0] = mreg[u].x;
            dst[1] = mreg[u].y;
            dst[2] = mreg[u].z;
            dst[3] = mreg[u].w;
        }
    }
    __syncthreads();
    if (is_v && j < p.n_kb) {  // c_j = sum_t Vbar_jt (M_h Vbar_j)_t
        double u = 0.0;
        for (int c = 0; c < kD; ++c) u = fma((double)Ms[lane * (kD + 1) + c], vb[wave][c], u);
        const double cj = wave_sum(u * vb[wave][lane]);
        if (lane == 0) p.out.cT[(size_t)h * p.n_kb + j] = cj;
    }
}

}  // namespace

hipError_t launch_pool(const PoolParams &p, hipStream_t s)
{
    const int gq = (p.n_qb + kWaves - 1) / kWaves, gk = (p.n_kb + kWaves - 1) / kWaves;
    const long long blocks = (long long)p.H * (gq + 2 * gk);
    if (blocks == 0) return hipSuccess;
    hipLaunchKernelGGL(pool_kernel, dim3((unsigned)blocks), dim3(kThreads), 0, s, p);
    return hipGetLastError();
}

}  // namespace ress
