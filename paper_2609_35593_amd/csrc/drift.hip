// The change that masking makes in what attention writes into the residual
// stream, per query block (the reference measurement of Sec. 3, "Testing the
// Probability Assumption"): out[h][i] = sum over the block's tokens t of
// x_t^T M_h x_t = ||W_O^h x_t||^2, with x_t = a_t - b_t the difference of two
// float32 attention outputs of the same queries.
//
// One workgroup per (head, query block), 4 waves; a wave takes every fourth
// token of the block, lane <-> channel: x in float64 (the difference of two
// float32 values is exact there), M_h x by broadcasts of x from the wave's LDS
// area against M_h's rows in LDS, x . (M_h x) by a wave butterfly, summed over
// the wave's tokens in order and then over the 4 waves in order.
#include "ress_internal.h"

namespace ress {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;

__device__ __forceinline__ double wave_sum(double x)
{
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o);
    return x;
}

__global__ void __launch_bounds__(kThreads) drift_sq_kernel(const DriftSqParams p)
{
    __shared__ float Ms[kD * (kD + 1)];
    __shared__ __align__(16) double xs[kWaves][kD];
    __shared__ double part[kWaves];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int h = blockIdx.x / p.n_qb, i = blockIdx.x % p.n_qb;
    const float *Mh = p.gram + (size_t)h * kD * kD;
    for (int e = tid; e < kD * kD; e += kThreads) Ms[(e >> 6) * (kD + 1) + (e & 63)] = Mh[e];
    __syncthreads();
    const int t0 = i * p.bq, t1 = min(t0 + p.bq, p.N);
    double acc = 0.0;
    for (int t = t0 + wave; t < t1; t += kWaves) {
        const size_t off = ((size_t)h * p.N + t) * kD + lane;
        const double x = (double)p.a[off] - (double)p.b[off];
        xs[wave][lane] = x;
        __builtin_amdgcn_wave_barrier();
        double u = 0.0;
#pragma unroll 8
        for (int c = 0; c < kD; c += 2) {
            const double2 xc = *reinterpret_cast<const double2 *>(&xs[wave][c]);
            u = fma((double)Ms[lane * (kD + 1) + c + 1], xc.y, fma((double)Ms[lane * (kD + 1) + c], xc.x, u));
        }
        acc += wave_sum(x * u);
        __builtin_amdgcn_wave_barrier();
    }
    if (lane == 0) part[wave] = acc;
    __syncthreads();
    if (tid == 0) {
        double s = 0.0;
        for (int w = 0; w < kWaves; ++w) s += part[w];
        p.out[(size_t)h * p.n_qb + i] = s;
    }
}

}  // namespace

hipError_t launch_drift_sq(const DriftSqParams &p, hipStream_t s)
{
    const long long blocks = (long long)p.H * p.n_qb;
    if (blocks == 0) return hipSuccess;
    hipLaunchKernelGGL(drift_sq_kernel, dim3((unsigned)blocks), dim3(kThreads), 0, s, p);
    return hipGetLastError();
}

}  // namespace ress
