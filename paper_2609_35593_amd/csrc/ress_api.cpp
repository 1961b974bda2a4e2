// C ABI of libress: argument validation, workspace layout and kernel launches.
// Every check runs on the host before anything is enqueued, so an error status
// means no device work and no output writes.
#include <math.h>
#include <string.h>

#include <mutex>

#include "ress_internal.h"

// Device memory of ress_select_noalloc: the selection's workspace for callers that
// cannot allocate. One copy per GPU (at its own address), held until the process
// ends; host code never passes this name to a kernel, only the per-device address
// hipGetSymbolAddress returns for it.
static __device__ __align__(256) unsigned char scratch[RESS_NOALLOC_SCRATCH_BYTES];

namespace {

using ress::kD;

struct Grid {
    long long n_qb, n_kb;
};

int check_shape(const ress_shape *s, Grid *g)
{
    if (!s) return RESS_E_INVALID_ARG;
    if (s->H < 0 || s->N < 0 || s->n_special_tail < 0 || s->n_special_tail > s->N) return RESS_E_INVALID_ARG;
    if (s->D != kD) return RESS_E_UNSUPPORTED;
    if ((s->bq != 64 && s->bq != 128) || (s->bk != 64 && s->bk != 128)) return RESS_E_UNSUPPORTED;
    if (s->H > RESS_MAX_HEADS || s->N > RESS_MAX_TOKENS) return RESS_E_UNSUPPORTED;
    g->n_qb = ((long long)s->N + s->bq - 1) / s->bq;
    g->n_kb = ((long long)s->N + s->bk - 1) / s->bk;
    return RESS_OK;
}

bool has_work(const ress_shape *s) { return s->H > 0 && s->N > 0; }

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }
bool aligned16(const void *ptr) { return ((uintptr_t)ptr & 15u) == 0; }

// Workspace: qbar [H][n_qb][64], kbar [H][n_kb][64], vbar [H][n_kb][64], cT
// [H][n_kb] (float64), every region 256-byte aligned.
struct Regions {
    size_t qb, kb, cb;  // qbar; kbar and vbar (each); cT
};

Regions regions(const ress_shape *s, const Grid &g)
{
    return {align256((size_t)s->H * g.n_qb * kD * sizeof(double)), align256((size_t)s->H * g.n_kb * kD * sizeof(double)),
            align256((size_t)s->H * g.n_kb * sizeof(double))};
}

size_t workspace_bytes(const ress_shape *s, const Grid &g)
{
    const Regions r = regions(s, g);
    return r.qb + 2 * r.kb + r.cb;
}

// Pooled state inside the workspace (the regions workspace_bytes sizes).
ress::Pooled pooled_layout(const ress_shape *s, const Grid &g, void *workspace)
{
    char *w = static_cast<char *>(workspace);
    const Regions r = regions(s, g);
    ress::Pooled pooled;
    pooled.qbar = reinterpret_cast<double *>(w);
    pooled.kbar = reinterpret_cast<double *>(w + r.qb);
    pooled.vbar = reinterpret_cast<double *>(w + r.qb + r.kb);
    pooled.cT = reinterpret_cast<double *>(w + r.qb + 2 * r.kb);
    return pooled;
}

// Address of the current device's copy of `scratch`, looked up once per device
// (with that device current) and kept.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void *g_scratch_ptr[kMaxDevices];

int scratch_of_current_device(void **out)
{
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return RESS_E_HIP;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (!g_scratch_ptr[dev]) {
        void *ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return RESS_E_HIP;
        g_scratch_ptr[dev] = ptr;
    }
    *out = g_scratch_ptr[dev];
    return RESS_OK;
}

int first_forced_block(const ress_shape *s, const Grid &g)
{
    return s->n_special_tail > 0 ? (s->N - s->n_special_tail) / s->bk : (int)g.n_kb;
}

}  // namespace

extern "C" {

const char *ress_status_string(int status)
{
    switch (status) {
    case RESS_OK: return "RESS_OK";
    case RESS_E_INVALID_ARG: return "RESS_E_INVALID_ARG: invalid argument";
    case RESS_E_UNSUPPORTED: return "RESS_E_UNSUPPORTED: unsupported shape (D must be 64, blocks 64/128, n_kb <= 4096, H <= 256)";
    case RESS_E_WORKSPACE: return "RESS_E_WORKSPACE: workspace missing, too small or not 256-byte aligned";
    case RESS_E_HIP: return "RESS_E_HIP: HIP launch failed";
    default: return "unknown ress status";
    }
}

int ress_select_workspace_size(const ress_shape *shape, size_t *bytes)
{
    Grid g;
    int st = check_shape(shape, &g);
    if (st != RESS_OK) return st;
    if (!bytes) return RESS_E_INVALID_ARG;
    if (g.n_kb > RESS_MAX_KEY_BLOCKS) return RESS_E_UNSUPPORTED;
    *bytes = has_work(shape) ? workspace_bytes(shape, g) : 0;
    return RESS_OK;
}

int ress_select(const ress_shape *shape, const ress_select_params *params, const void *q,
                const void *k, const void *v, const float *gram, const int32_t *keep_budget,
                int32_t *kept_count, int32_t *kept_idx, double *drift, double *key_out,
                double *prob_out, void *workspace, size_t ws_bytes, hipStream_t stream)
{
    Grid g;
    int st = check_shape(shape, &g);
    if (st != RESS_OK) return st;
    if (g.n_kb > RESS_MAX_KEY_BLOCKS) return RESS_E_UNSUPPORTED;
    if (!params) return RESS_E_INVALID_ARG;
    if (params->rounds < 0 || params->rounds > RESS_MAX_ROUNDS || params->swap_floor < 0 ||
        !(params->rho >= 0.0) || !isfinite(params->rho) || !(params->eps > 0.0) || !isfinite(params->eps))
        return RESS_E_INVALID_ARG;
    if (params->criterion < RESS_CRITERION_DRIFT || params->criterion > RESS_CRITERION_DRIFT_MAX_FULL ||
        !(params->cdf_tau >= 0.0 && params->cdf_tau <= 1.0) ||
        (params->cdf_tau > 0.0 && params->criterion != RESS_CRITERION_PROBABILITY))
        return RESS_E_INVALID_ARG;
    if (!has_work(shape)) return RESS_OK;
    const bool pooled_ready = params->pooled_in_workspace != 0;
    if (!gram || !keep_budget || !kept_count || !kept_idx || !aligned16(gram)) return RESS_E_INVALID_ARG;
    if (!pooled_ready && (!q || !k || !v || !aligned16(q) || !aligned16(k) || !aligned16(v)))
        return RESS_E_INVALID_ARG;

    const int n_kb = (int)g.n_kb, n_qb = (int)g.n_qb;
    const int first_forced = first_forced_block(shape, g);
    const int n_forced = n_kb - first_forced, n_p = first_forced;
    const int floor2 = 2 - n_forced > 0 ? 2 - n_forced : 0;  // at least two kept blocks per row
    const int lo = n_p < floor2 ? n_p : floor2;
    for (int h = 0; h < shape->H; ++h)
        if (keep_budget[h] < lo || keep_budget[h] > n_p) return RESS_E_INVALID_ARG;

    const size_t need = workspace_bytes(shape, g);
    if (!workspace || ws_bytes < need || ((uintptr_t)workspace & 255u)) return RESS_E_WORKSPACE;

    const ress::Pooled pooled = pooled_layout(shape, g, workspace);

    ress::PoolParams pp;
    pp.H = shape->H;
    pp.N = shape->N;
    pp.bq = shape->bq;
    pp.bk = shape->bk;
    pp.n_qb = n_qb;
    pp.n_kb = n_kb;
    pp.q = static_cast<const uint16_t *>(q);
    pp.k = static_cast<const uint16_t *>(k);
    pp.v = static_cast<const uint16_t *>(v);
    pp.gram = gram;
    pp.out = pooled;

    ress::SelectParams sp;
    memset(&sp, 0, sizeof sp);
    sp.H = shape->H;
    sp.n_qb = n_qb;
    sp.n_kb = n_kb;
    sp.first_forced = first_forced;
    sp.first_dense_qb = (params->dense_special_queries && shape->n_special_tail > 0)
                            ? (shape->N - shape->n_special_tail) / shape->bq
                            : n_qb;
    sp.rounds = params->rounds;
    sp.swap_floor = params->swap_floor;
    sp.rho = params->rho;
    sp.eps = params->eps;
    sp.criterion = params->criterion;
    sp.cdf_tau = params->cdf_tau;
    sp.pooled = pooled;
    sp.gram = gram;
    sp.kept_count = kept_count;
    sp.kept_idx = kept_idx;
    sp.drift = drift;
    sp.key_out = key_out;
    sp.prob_out = prob_out;
    for (int h = 0; h < shape->H; ++h) sp.budgets[h] = keep_budget[h];

    if (!pooled_ready && ress::launch_pool(pp, stream) != hipSuccess) return RESS_E_HIP;
    if (ress::launch_select(sp, stream) != hipSuccess) return RESS_E_HIP;
    return RESS_OK;
}

int ress_select_noalloc(const ress_shape *shape, const ress_select_params *params, const void *q, const void *k,
                        const void *v, const float *gram, const int32_t *keep_budget, int32_t *kept_count,
                        int32_t *kept_idx, double *drift, double *key_out, double *prob_out, hipStream_t stream)
{
    Grid g;
    int st = check_shape(shape, &g);
    if (st != RESS_OK) return st;
    if (g.n_kb > RESS_MAX_KEY_BLOCKS) return RESS_E_UNSUPPORTED;
    if (!params) return RESS_E_INVALID_ARG;
    if (params->pooled_in_workspace) return RESS_E_INVALID_ARG;  // the caller cannot reach this workspace
    if (!has_work(shape)) return RESS_OK;
    if (workspace_bytes(shape, g) > (size_t)RESS_NOALLOC_SCRATCH_BYTES) return RESS_E_UNSUPPORTED;
    void *ws = nullptr;
    st = scratch_of_current_device(&ws);
    if (st != RESS_OK) return st;
    return ress_select(shape, params, q, k, v, gram, keep_budget, kept_count, kept_idx, drift, key_out, prob_out,
                       ws, (size_t)RESS_NOALLOC_SCRATCH_BYTES, stream);
}

// Shared checks of the two projections: shape, H a multiple of 4, grid size.
static int proj_common(const ress_shape *shape, Grid *g, ress::ProjParams *pp, int n_out_per_head)
{
    int st = check_shape(shape, g);
    if (st != RESS_OK) return st;
    if (shape->H % 4 != 0) return RESS_E_UNSUPPORTED;
    memset(pp, 0, sizeof *pp);
    pp->T = shape->N;
    pp->H = shape->H;
    pp->m_tiles = (shape->N + 255) / 256;
    pp->n_tiles = n_out_per_head * shape->H / 256;
    const long long items = (long long)pp->m_tiles * pp->n_tiles;
    const long long per_xcd = (items + 7) / 8;
    if (8 * per_xcd > 0x7fffffffLL) return RESS_E_UNSUPPORTED;
    pp->items_per_xcd = (int)per_xcd;
    return RESS_OK;
}

int ress_qkv_proj_pool(const ress_shape *shape, const void *x, const void *w_qkv, void *q, void *k, void *v,
                       const float *gram, void *workspace, size_t ws_bytes, hipStream_t stream)
{
    Grid g;
    ress::ProjParams pp;
    int st = proj_common(shape, &g, &pp, 3 * kD);
    if (st != RESS_OK) return st;
    if (g.n_kb > RESS_MAX_KEY_BLOCKS) return RESS_E_UNSUPPORTED;
    if (!has_work(shape)) return RESS_OK;
    if (!x || !w_qkv || !q || !k || !v || !gram) return RESS_E_INVALID_ARG;
    if (!aligned16(x) || !aligned16(w_qkv) || !aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(gram))
        return RESS_E_INVALID_ARG;
    const void *ins[2] = {x, w_qkv};
    void *outs[3] = {q, k, v};
    for (void *o : outs)
        for (const void *in : ins)
            if (o == in) return RESS_E_INVALID_ARG;
    if (q == k || q == v || k == v) return RESS_E_INVALID_ARG;
    const size_t need = workspace_bytes(shape, g);
    if (!workspace || ws_bytes < need || ((uintptr_t)workspace & 255u)) return RESS_E_WORKSPACE;
    pp.mode = 0;
    pp.bq = shape->bq;
    pp.bk = shape->bk;
    pp.n_qb = (int)g.n_qb;
    pp.n_kb = (int)g.n_kb;
    pp.a = static_cast<const uint16_t *>(x);
    pp.w = static_cast<const uint16_t *>(w_qkv);
    pp.q = static_cast<uint16_t *>(q);
    pp.k = static_cast<uint16_t *>(k);
    pp.v = static_cast<uint16_t *>(v);
    pp.gram = gram;
    pp.pooled = pooled_layout(shape, g, workspace);
    if (ress::launch_proj(pp, stream) != hipSuccess) return RESS_E_HIP;
    return RESS_OK;
}

int ress_out_proj_residual(const ress_shape *shape, const void *o, const void *w_o, const void *resid_in,
                           void *resid_out, hipStream_t stream)
{
    Grid g;
    ress::ProjParams pp;
    int st = proj_common(shape, &g, &pp, kD);
    if (st != RESS_OK) return st;
    if (!has_work(shape)) return RESS_OK;
    if (!o || !w_o || !resid_in || !resid_out) return RESS_E_INVALID_ARG;
    if (!aligned16(o) || !aligned16(w_o) || !aligned16(resid_in) || !aligned16(resid_out))
        return RESS_E_INVALID_ARG;
    if (resid_out == o || resid_out == w_o) return RESS_E_INVALID_ARG;
    pp.mode = 1;
    pp.a = static_cast<const uint16_t *>(o);
    pp.w = static_cast<const uint16_t *>(w_o);
    pp.resid_in = static_cast<const uint16_t *>(resid_in);
    pp.resid_out = static_cast<uint16_t *>(resid_out);
    if (ress::launch_proj(pp, stream) != hipSuccess) return RESS_E_HIP;
    return RESS_OK;
}

int ress_out_proj_residual_f32(const ress_shape *shape, const void *o, const void *w_o, const float *resid_in,
                               float *resid_out, hipStream_t stream)
{
    Grid g;
    ress::ProjParams pp;
    int st = proj_common(shape, &g, &pp, kD);
    if (st != RESS_OK) return st;
    if (!has_work(shape)) return RESS_OK;
    if (!o || !w_o || !resid_in || !resid_out) return RESS_E_INVALID_ARG;
    if (!aligned16(o) || !aligned16(w_o) || !aligned16(resid_in) || !aligned16(resid_out))
        return RESS_E_INVALID_ARG;
    if ((const void *)resid_out == o || (const void *)resid_out == w_o) return RESS_E_INVALID_ARG;
    pp.mode = 2;
    pp.a = static_cast<const uint16_t *>(o);
    pp.w = static_cast<const uint16_t *>(w_o);
    pp.resid_in_f32 = resid_in;
    pp.resid_out_f32 = resid_out;
    if (ress::launch_proj(pp, stream) != hipSuccess) return RESS_E_HIP;
    return RESS_OK;
}

int ress_block_drift_sq(const ress_shape *shape, const float *a, const float *b, const float *gram, double *out,
                        hipStream_t stream)
{
    Grid g;
    int st = check_shape(shape, &g);
    if (st != RESS_OK) return st;
    if (!has_work(shape)) return RESS_OK;
    if (!a || !b || !gram || !out) return RESS_E_INVALID_ARG;
    if (!aligned16(a) || !aligned16(b) || !aligned16(gram)) return RESS_E_INVALID_ARG;
    if ((const void *)out == a || (const void *)out == b || (const void *)out == gram) return RESS_E_INVALID_ARG;
    if ((long long)shape->H * g.n_qb > 0x7fffffffLL) return RESS_E_UNSUPPORTED;
    ress::DriftSqParams dp;
    dp.H = shape->H;
    dp.N = shape->N;
    dp.bq = shape->bq;
    dp.n_qb = (int)g.n_qb;
    dp.a = a;
    dp.b = b;
    dp.gram = gram;
    dp.out = out;
    if (ress::launch_drift_sq(dp, stream) != hipSuccess) return RESS_E_HIP;
    return RESS_OK;
}

static int attn_common(const ress_shape *shape, const void *q, const void *k, const void *v,
                       const int32_t *kept_count, const int32_t *kept_idx, float scale, void *o,
                       bool sparse, bool out_f32, hipStream_t stream)
{
    Grid g;
    int st = check_shape(shape, &g);
    if (st != RESS_OK) return st;
    if (!(scale > 0.f) || !isfinite(scale)) return RESS_E_INVALID_ARG;
    if (!has_work(shape)) return RESS_OK;
    if (!q || !k || !v || !o) return RESS_E_INVALID_ARG;
    if (o == q || o == k || o == v) return RESS_E_INVALID_ARG;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o)) return RESS_E_INVALID_ARG;
    if (sparse && (!kept_count || !kept_idx)) return RESS_E_INVALID_ARG;
    // Work order (attn.hip): contiguous work-balanced segments per XCD while the
    // K and V of all heads fit the 256 MB infinity cache, rotating per-head chunks
    // beyond. Segments: up to 1.5 times an even share of rows per XCD, so that
    // per-head work differing by up to that factor still splits evenly.
    const long long rows = (long long)shape->H * g.n_qb;
    const bool rotate = 2ll * shape->H * shape->N * kD * 2 > (256ll << 20);
    const long long cap = rotate ? (g.n_qb + 7) / 8 : (3 * rows + 15) / 16;
    const long long grid = rotate ? 8 * cap * shape->H : 8 * cap;
    if (grid > 0x7fffffffLL) return RESS_E_UNSUPPORTED;
    ress::AttnParams ap;
    ap.H = shape->H;
    ap.N = shape->N;
    ap.n_qb = (int)g.n_qb;
    ap.n_kb = (int)g.n_kb;
    ap.rotate = rotate ? 1 : 0;
    ap.seg_cap = (int)cap;
    ap.scale_log2 = scale * 1.4426950408889634f;
    ap.q = static_cast<const uint16_t *>(q);
    ap.k = static_cast<const uint16_t *>(k);
    ap.v = static_cast<const uint16_t *>(v);
    ap.o = out_f32 ? nullptr : static_cast<uint16_t *>(o);
    ap.o32 = out_f32 ? static_cast<float *>(o) : nullptr;
    ap.kept_count = kept_count;
    ap.kept_idx = kept_idx;
    if (ress::launch_attn(ap, shape->bq, shape->bk, sparse, stream) != hipSuccess) return RESS_E_HIP;
    return RESS_OK;
}

int ress_sparse_attn(const ress_shape *shape, const void *q, const void *k, const void *v,
                     const int32_t *kept_count, const int32_t *kept_idx, float scale, void *o,
                     hipStream_t stream)
{
    return attn_common(shape, q, k, v, kept_count, kept_idx, scale, o, true, false, stream);
}

int ress_sparse_attn_out_f32(const ress_shape *shape, const void *q, const void *k, const void *v,
                             const int32_t *kept_count, const int32_t *kept_idx, float scale, float *o,
                             hipStream_t stream)
{
    return attn_common(shape, q, k, v, kept_count, kept_idx, scale, o, true, true, stream);
}

int ress_dense_attn(const ress_shape *shape, const void *q, const void *k, const void *v, float scale,
                    void *o, hipStream_t stream)
{
    return attn_common(shape, q, k, v, nullptr, nullptr, scale, o, false, false, stream);
}

}  // extern "C"
