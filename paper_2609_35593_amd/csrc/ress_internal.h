// Internal declarations shared by the HIP kernels and the C ABI layer of libress.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "ress.h"

namespace ress {

constexpr int kD = 64;      // head dimension handled by every kernel
constexpr int kWave = 64;   // CDNA wavefront width

// Pooled tensors of one layer, float64, row-major, carved out of the selection
// workspace.
struct Pooled {
    double *qbar;   // [H][n_qb][64]  query block means
    double *kbar;   // [H][n_kb][64]  key block means
    double *vbar;   // [H][n_kb][64]  value block means
    double *cT;     // [H][n_kb]      Vbar_j^T M_h Vbar_j
};

struct PoolParams {
    int H, N, bq, bk, n_qb, n_kb;
    const uint16_t *q, *k, *v;  // bf16 bits [H][N][64]
    const float *gram;          // [H][64][64]
    Pooled out;
};

struct SelectParams {
    int H, n_qb, n_kb;
    int first_forced;    // key blocks j >= first_forced are always kept (n_kb if none)
    int first_dense_qb;  // query blocks i >= first_dense_qb keep every block (n_qb if none)
    int rounds, swap_floor;
    int items_per_xcd;   // (head, row group) items per XCD, set by the launcher
    int criterion;       // RESS_CRITERION_*
    double rho, eps;
    double cdf_tau;      // 0 = no CDF cap
    Pooled pooled;
    const float *gram;
    int32_t *kept_count, *kept_idx;
    double *drift, *key_out, *prob_out;
    int32_t budgets[RESS_MAX_HEADS];
};

struct AttnParams {
    int H, N, n_qb, n_kb;
    int rotate;         // work order: 0 work-balanced segments, 1 rotating chunks (see attn.hip)
    int seg_cap;        // segments: most rows one XCD runs; rotation: query blocks per chunk
    float scale_log2;   // softmax scale * log2(e)
    const uint16_t *q, *k, *v;
    uint16_t *o;                           // bf16 output, unless o32 is set
    float *o32;                            // float32 output (null: write o)
    const int32_t *kept_count, *kept_idx;  // null for dense attention
};

// The projections on either side of the path (mode 0: QKV + pooling, mode 1:
// output projection + bf16 residual, mode 2: output projection + float32
// residual), one bf16 GEMM with per-mode epilogues.
struct ProjParams {
    int mode;
    int T, H;                 // tokens, heads (model width 64 H)
    int bq, bk, n_qb, n_kb;   // pooling grid (mode 0)
    int m_tiles, n_tiles, items_per_xcd;
    const uint16_t *a;        // mode 0: x [T][64H]; modes 1, 2: o [H][T][64]
    const uint16_t *w;        // [n_out][64H] (out features x in features)
    uint16_t *q, *k, *v;      // mode 0: bf16 [H][T][64]
    const uint16_t *resid_in; // mode 1: bf16 [T][64H]
    uint16_t *resid_out;
    const float *resid_in_f32;  // mode 2: float32 [T][64H]
    float *resid_out_f32;
    const float *gram;        // mode 0: [H][64][64]
    Pooled pooled;            // mode 0
};

// Per-query-block squared projected norm of the difference of two float32
// attention outputs (the masking reference of Sec. 3).
struct DriftSqParams {
    int H, N, bq, n_qb;
    const float *a, *b;   // [H][N][64]
    const float *gram;    // [H][64][64]
    double *out;          // [H][n_qb]
};

hipError_t launch_pool(const PoolParams &p, hipStream_t s);
hipError_t launch_drift_sq(const DriftSqParams &p, hipStream_t s);
hipError_t launch_proj(const ProjParams &p, hipStream_t s);
hipError_t launch_select(const SelectParams &p, hipStream_t s);
hipError_t launch_attn(const AttnParams &p, int bq, int bk, bool sparse, hipStream_t s);

}  // namespace ress
