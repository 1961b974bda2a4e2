// Block mean pooling of Q, K and V (the coarse block grid of Sec. 3, step (1)),
// plus U_j = M_h Vbar_j for the drift scores (Eq. 9).
//
// One workgroup per (head, block). Each thread streams 16-byte rows segments of
// the block (8 channels of one token); partial sums are float64, which holds the
// sum of bf16 values of a block exactly, so the mean (one division) equals the
// float64 mean computed in any order. This pass is the only part of the
// selection that reads Q, K, V from HBM.
#include "ress_internal.h"

namespace ress {
namespace {

constexpr int kThreads = 256;
constexpr int kTokLanes = kThreads / 8;  // threads that share one 8-channel chunk

__device__ __forceinline__ void accum_bf16x8(double (&acc)[8], uint4 w)
{
    const unsigned int u[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        acc[2 * e] += (double)__uint_as_float(u[e] << 16);
        acc[2 * e + 1] += (double)__uint_as_float(u[e] & 0xffff0000u);
    }
}

// Sums rows [lo, lo+cnt) of x[h] into red[kTokLanes][64], then returns (to the
// first 64 threads) the block mean of channel threadIdx.x.
__device__ __forceinline__ double block_mean(const uint16_t *__restrict__ x, size_t row0, int cnt,
                                             int maxb, double *red)
{
    const int t = threadIdx.x, ch = t & 7, sub = t >> 3;
    double acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    uint4 w[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const int tok = sub + r * kTokLanes;
        w[r] = (r * kTokLanes < maxb && tok < cnt)
                   ? *reinterpret_cast<const uint4 *>(x + (row0 + tok) * kD + ch * 8)
                   : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) accum_bf16x8(acc, w[r]);
#pragma unroll
    for (int e = 0; e < 8; ++e) red[sub * kD + ch * 8 + e] = acc[e];
    __syncthreads();
    double mean = 0.0;
    if (t < kD) {
        double s = 0.0;
        for (int r = 0; r < kTokLanes; ++r) s += red[r * kD + t];
        mean = s / (double)cnt;
    }
    __syncthreads();
    return mean;
}

__global__ void __launch_bounds__(kThreads) pool_kernel(const PoolParams p)
{
    __shared__ double red[kTokLanes * kD];
    __shared__ double vmean[kD];
    __shared__ float Ms[kD * (kD + 1)];
    const int t = threadIdx.x;
    const int nq = p.H * p.n_qb;
    if ((int)blockIdx.x < nq) {
        const int h = blockIdx.x / p.n_qb, i = blockIdx.x % p.n_qb;
        const int lo = i * p.bq, cnt = min(p.bq, p.N - lo);
        const double m = block_mean(p.q, (size_t)h * p.N + lo, cnt, p.bq, red);
        if (t < kD) p.out.qbar[((size_t)h * p.n_qb + i) * kD + t] = m;
        return;
    }
    const int b = blockIdx.x - nq;
    const int h = b / p.n_kb, j = b % p.n_kb;
    const int lo = j * p.bk, cnt = min(p.bk, p.N - lo);
    const float *Mh = p.gram + (size_t)h * kD * kD;
    for (int e = t; e < kD * kD; e += kThreads) Ms[(e >> 6) * (kD + 1) + (e & 63)] = Mh[e];
    const double km = block_mean(p.k, (size_t)h * p.N + lo, cnt, p.bk, red);
    const double vm = block_mean(p.v, (size_t)h * p.N + lo, cnt, p.bk, red);
    if (t < kD) {
        p.out.kbarT[((size_t)h * kD + t) * p.n_kb + j] = km;
        p.out.vbar[((size_t)h * p.n_kb + j) * kD + t] = vm;
        p.out.vbarT[((size_t)h * kD + t) * p.n_kb + j] = vm;
        vmean[t] = vm;
    }
    __syncthreads();
    if (t < kD) {
        double u = 0.0;
        for (int c = 0; c < kD; ++c) u = fma((double)Ms[t * (kD + 1) + c], vmean[c], u);
        p.out.uT[((size_t)h * kD + t) * p.n_kb + j] = u;
    }
}

}  // namespace

hipError_t launch_pool(const PoolParams &p, hipStream_t s)
{
    const long long blocks = (long long)p.H * (p.n_qb + p.n_kb);
    if (blocks == 0) return hipSuccess;
    hipLaunchKernelGGL(pool_kernel, dim3((unsigned)blocks), dim3(kThreads), 0, s, p);
    return hipGetLastError();
}

}  // namespace ress
