/*
 * ress.h - C ABI of the MI355X (gfx950) hot path of ReSS, "Residual-Restoring
 * Sparse Attention for 3D Vision Transformers": drift-based block selection
 * followed by block-sparse attention over the kept blocks, plus the dense
 * attention it is measured against, and the projections on either side of the
 * path (QKV projection with the pooling fused in, output projection with the
 * residual add).
 *
 * Conventions shared by every entry point
 *  - Tensors Q, K, V, O are bf16, laid out [H][N][D] contiguous (head-major, then
 *    token, then channel), one layer of batch 1, with D == 64. The projections'
 *    activations and weights are token-major / [out][in], as documented there.
 *  - Tokens are grouped into fixed-size blocks: query block i covers tokens
 *    [i*bq, min((i+1)*bq, N)), key block j covers [j*bk, min((j+1)*bk, N))
 *    (the paper's block grid, Sec. 3 step (1)); the last block of each kind may be
 *    partial. n_qb = ceil(N / bq), n_kb = ceil(N / bk).
 *  - The last n_special_tail tokens are special (camera / register) tokens. Key
 *    blocks that hold any of them are always kept and are not candidates
 *    (Sec. 4.1; the trailing "sink" block of Supp. F).
 *  - Device pointers are owned by the caller; the library never allocates,
 *    frees or copies device memory and never synchronises. All work is enqueued
 *    on `stream` in order; a status of RESS_OK means the work was enqueued.
 *    Device-side failures surface at the caller's next synchronisation.
 *  - On any error status nothing is enqueued and no output is written.
 *  - Calls are stateless; concurrent calls on different streams are safe as
 *    long as their output buffers (and workspaces) do not overlap.
 */
#ifndef RESS_H
#define RESS_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes. */
#define RESS_OK 0
#define RESS_E_INVALID_ARG (-1) /* null pointer, negative size, bad parameter or budget */
#define RESS_E_UNSUPPORTED (-2) /* D != 64, block size not 64/128, n_kb > 4096, H > 256, N > 2^24 */
#define RESS_E_WORKSPACE (-3)   /* workspace missing, too small or misaligned */
#define RESS_E_HIP (-4)         /* a HIP launch call failed */

/* Largest number of key blocks per row: one row of the selection is held in
 * registers, the same cap as the paper's fused round kernel (Supp. E). */
#define RESS_MAX_KEY_BLOCKS 4096
#define RESS_MAX_HEADS 256
#define RESS_MAX_ROUNDS 32
/* Largest N accepted by every entry point (token offsets within a head stay in 32 bits). */
#define RESS_MAX_TOKENS (1 << 24)

typedef struct {
    int H;              /* heads, 0..RESS_MAX_HEADS */
    int N;              /* tokens per head (all views concatenated), 0..RESS_MAX_TOKENS */
    int D;              /* head dimension; must be 64 */
    int bq;             /* query block size: 64 or 128 */
    int bk;             /* key block size: 64 or 128 */
    int n_special_tail; /* trailing special tokens, 0..N */
} ress_shape;

/* Selection criteria. RESS_CRITERION_DRIFT is the method (Secs. 4.2-4.3); the
 * others are the comparisons the paper makes with the same budget:
 *   PROBABILITY     keep the c_h largest pooled probabilities P_ij (the
 *                   probability rule of the ablation, Table 2); with cdf_tau > 0
 *                   keep only the shortest prefix in descending P whose mass,
 *                   the always-kept forced blocks included, reaches cdf_tau (the
 *                   CDF threshold row of Table 2), never below the two-block
 *                   floor; the realised count replaces c_h in that row's rounds;
 *   DRIFT_MAX_SWAP  sign-flipped objective in the rounds only (Fig. 8, Sec. 6.1): the
 *                   initial set as for DRIFT, every round makes the swaps that
 *                   raise J most, and the largest J seen is kept;
 *   DRIFT_MAX_FULL  sign flipped from the start: keep the c_h smallest keys, then
 *                   rounds as for DRIFT_MAX_SWAP.
 * Restoration (rounds > 0) applies to every criterion. */
#define RESS_CRITERION_DRIFT 0
#define RESS_CRITERION_PROBABILITY 1
#define RESS_CRITERION_DRIFT_MAX_SWAP 2
#define RESS_CRITERION_DRIFT_MAX_FULL 3

/* Selection parameters (Secs. 4.2-4.3). The paper's values: rounds = 5,
 * rho = 0.5, eps = 1e-4 (Eqs. 7 and 17), criterion = RESS_CRITERION_DRIFT,
 * cdf_tau = 0. */
typedef struct {
    int rounds;                /* restoration rounds R, 0..RESS_MAX_ROUNDS */
    double rho;                /* total swap budget as a fraction of c_h (Eq. 17), >= 0 */
    double eps;                /* guard of Eq. 7, also applied to K in J and dJ, > 0 */
    int swap_floor;            /* round r swaps max(swap_floor, floor(rho c_h 2^-(r+1))), >= 0 */
    int dense_special_queries; /* nonzero: query blocks holding special tokens keep every key block */
    int criterion;             /* RESS_CRITERION_*, 0..3 */
    double cdf_tau;            /* CDF threshold in [0, 1]; 0 = off; nonzero only with PROBABILITY */
    int pooled_in_workspace;   /* nonzero: step 1 was done by ress_qkv_proj_pool into this
                                  workspace; q, k, v are then not read (may be NULL) */
} ress_select_params;

/* Bytes of device workspace ress_select needs for `shape` (pooled tensors,
 * float64). Returns RESS_OK, or RESS_E_INVALID_ARG / RESS_E_UNSUPPORTED. */
int ress_select_workspace_size(const ress_shape *shape, size_t *bytes);

/* Drift-based block selection (Secs. 4.2-4.3): for every head h and query
 * block i,
 *   1. pool Q, K, V into block means (Sec. 3 step (1));
 *   2. P_i = softmax_j(Qbar_i . Kbar_j / sqrt(D)) over all key blocks and the
 *      dense pooled output vbar_i = sum_j P_ij Vbar_j (Eq. 1);
 *   3. score every candidate key block by s_ij = P_ij ||W_O^h (vbar_i - Vbar_j)||
 *      through the Gram matrix M_h = W_O^h^T W_O^h (Eqs. 5-9) and keep the c_h
 *      largest keys s_ij / max(1 - P_ij, eps) (Eq. 7);
 *   4. run `rounds` budget-neutral rounds that restore the m_r dropped blocks and
 *      drop the m_r kept candidates with the largest exact decrease of the drift
 *      objective J = g^T M g / K^2 (Eqs. 10-17), keeping the drop set with the
 *      smallest J seen, the initial one included (track-best).
 * Every top-k breaks ties by the lower block index. Scoring and restoration run
 * in float64.
 *
 *   q, k, v       device bf16 [H][N][D], 16-byte aligned
 *   gram          device float32 [H][D][D], M_h row-major (computed once at load,
 *                 Eq. 8), 16-byte aligned; used as given, M_h x means
 *                 sum_b M[a][b] x[b]
 *   keep_budget   HOST int32 [H]: c_h, kept candidate blocks per row. Must lie in
 *                 [min(n_p, max(0, 2 - n_forced)), n_p], n_p = candidates (the
 *                 paper's floor of two kept key blocks per query row, Supp. F)
 *   kept_count    device int32 [H][n_qb] out: kept key blocks per row
 *                 (c_h + n_forced, or n_kb for dense rows; fewer under a CDF cap)
 *   kept_idx      device int32 [H][n_qb][n_kb] out: kept key block indices in
 *                 ascending order, padded with -1
 *   drift         device float64 [H][n_qb][2] out (or NULL): (J of the initial
 *                 selection, J of the returned selection); 0 for rows that drop
 *                 nothing. The criterion changes which selections these are.
 *   key_out       device float64 [H][n_qb][n_kb] out (or NULL): ranking keys of
 *                 Eq. 7; -1 for forced blocks
 *   prob_out      device float64 [H][n_qb][n_kb] out (or NULL): pooled map P
 *   workspace     device, >= ress_select_workspace_size bytes, 256-byte aligned
 * Inputs must be finite; non-finite inputs give unspecified (but in-bounds)
 * selections. */
int ress_select(const ress_shape *shape, const ress_select_params *params, const void *q,
                const void *k, const void *v, const float *gram, const int32_t *keep_budget,
                int32_t *kept_count, int32_t *kept_idx, double *drift, double *key_out,
                double *prob_out, void *workspace, size_t workspace_bytes, hipStream_t stream);

/* For callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid allocation): ress_select without a
 * caller workspace. The pooled state lives in a fixed device array inside the
 * library, RESS_NOALLOC_SCRATCH_BYTES per GPU, created with the library's code
 * object on each GPU it runs on and held until the process ends; this call
 * allocates and frees nothing. The current device's array is used (the stream
 * must belong to the current device). Every call on one GPU shares that GPU's
 * array, which keeps the last call's contents: calls that overlap on one GPU
 * (other streams, other threads) race, and the caller must serialise them.
 * Arguments and results as ress_select; params->pooled_in_workspace must be 0
 * (RESS_E_INVALID_ARG otherwise); shapes whose workspace
 * (ress_select_workspace_size) exceeds RESS_NOALLOC_SCRATCH_BYTES return
 * RESS_E_UNSUPPORTED (the 100-view layer, 16 heads x 1074 blocks, needs 26.5 MB). */
#define RESS_NOALLOC_SCRATCH_BYTES (48u << 20)
int ress_select_noalloc(const ress_shape *shape, const ress_select_params *params, const void *q, const void *k,
                        const void *v, const float *gram, const int32_t *keep_budget, int32_t *kept_count,
                        int32_t *kept_idx, double *drift, double *key_out, double *prob_out, hipStream_t stream);

/* Block-sparse attention (Sec. 3 step (3)): every query token t of query block
 * i attends exactly to the tokens of the key blocks kept_idx[h][i][0 ..
 * kept_count[h][i]-1], with the softmax renormalised among them:
 *   O_t = sum_s softmax_s(scale * Q_t . K_s) V_s.
 * bf16 MFMA products, float32 softmax and accumulation, probabilities rounded to
 * bf16 for the PV product. For a 32-row group of queries whose first 64 logits
 * lie within +-24 (base 2), Q is multiplied by scale * log2(e) and rounded to
 * bf16 before the products (one extra relative rounding of 2^-9 per element of
 * Q); other groups use Q as given.
 *   kept_count  device int32 [H][n_qb]; values are clamped to [0, n_kb]
 *   kept_idx    device int32 [H][n_qb][n_kb]; entries outside [0, n_kb) are
 *               ignored (contribute no keys); duplicates count twice
 *   scale       softmax scale, normally 1/sqrt(D); must be finite
 *   o           device bf16 [H][N][D] out (must not alias q, k, v)
 * A row with no keys gets a zero output. */
int ress_sparse_attn(const ress_shape *shape, const void *q, const void *k, const void *v,
                     const int32_t *kept_count, const int32_t *kept_idx, float scale, void *o,
                     hipStream_t stream);

/* ress_sparse_attn with a float32 output (device float32 [H][N][D], 16-byte
 * aligned, must not alias q, k, v): the same kernels, only the final
 * normalised O is stored unrounded. Differences between two such outputs
 * resolve changes far below the bf16 output's resolution, e.g. the output
 * change caused by masking one key block, the reference measurement of Sec. 3
 * (Fig. 2). */
int ress_sparse_attn_out_f32(const ress_shape *shape, const void *q, const void *k, const void *v,
                             const int32_t *kept_count, const int32_t *kept_idx, float scale, float *o,
                             hipStream_t stream);

/* The change masking makes in what attention writes into the residual
 * stream, per query block: the reference measurement of Sec. 3 ("Testing the
 * Probability Assumption", Fig. 2), which masks one key block and compares the
 * attention outputs after the output projection. For every head h and query
 * block i,
 *   out[h][i] = sum over the block's tokens t of (a_t - b_t)^T M_h (a_t - b_t)
 *             = sum_t ||W_O^h (a_t - b_t)||^2,
 * in float64, with a and b two attention outputs of the same queries (for
 * instance ress_sparse_attn_out_f32 with every key block but j, and with all).
 *   a, b   device float32 [H][N][64], 16-byte aligned
 *   gram   device float32 [H][64][64] (M_h), 16-byte aligned
 *   out    device float64 [H][n_qb] out (must not alias the inputs) */
int ress_block_drift_sq(const ress_shape *shape, const float *a, const float *b, const float *gram, double *out,
                        hipStream_t stream);

/* Dense attention, the same computation over every key block of every row
 * (the baseline the paper compares against, Table S6). */
int ress_dense_attn(const ress_shape *shape, const void *q, const void *k, const void *v,
                    float scale, void *o, hipStream_t stream);

/* The step before the path, fused: the QKV projection of one layer,
 *   [Q K V]_t = W_qkv x_t   (x_t the layer-normed residual-stream token),
 * written head-major, with the block mean pooling of Sec. 3 step (1) (and
 * Vbar_j^T M_h Vbar_j, Eq. 9) taken from the bf16 outputs in the projection's
 * epilogue, so that ress_select with params->pooled_in_workspace set does not
 * read Q, K, V from memory again. bf16 MFMA products, float32 accumulation,
 * outputs rounded to bf16 once; pooled means in float64 over those outputs
 * (identical to what ress_select would pool from them).
 *   x          device bf16 [N][H*64], token-major
 *   w_qkv      device bf16 [3*H*64][H*64], out features x in features: rows
 *              64h .. 64h+63 give head h of Q, then H*64 rows of K, then V
 *   q, k, v    device bf16 [H][N][64] out
 *   gram       device float32 [H][64][64] (M_h, as for ress_select)
 *   workspace  as for ress_select (>= ress_select_workspace_size bytes, 256-byte
 *              aligned); receives the pooled state
 * H must be a multiple of 4 (tiles of 256 features); N <= 2^24. Pointers 16-byte
 * aligned; outputs must not alias inputs. */
int ress_qkv_proj_pool(const ress_shape *shape, const void *x, const void *w_qkv, void *q, void *k, void *v,
                       const float *gram, void *workspace, size_t workspace_bytes, hipStream_t stream);

/* The step after the path, fused: output projection and residual add,
 *   resid_out_t = resid_in_t + W_O concat_h(O[h][t])
 * reading the head-major attention output directly. bf16 MFMA products, float32
 * accumulation, the residual added in float32 and the sum rounded to bf16 once.
 *   o          device bf16 [H][N][64] (ress_sparse_attn's output)
 *   w_o        device bf16 [H*64][H*64], out features x in features (in = 64h + d)
 *   resid_in   device bf16 [N][H*64]
 *   resid_out  device bf16 [N][H*64] out; may be resid_in (in place), must not
 *              alias o or w_o
 * H must be a multiple of 4. Pointers 16-byte aligned. */
int ress_out_proj_residual(const ress_shape *shape, const void *o, const void *w_o, const void *resid_in,
                           void *resid_out, hipStream_t stream);

/* ress_out_proj_residual with a float32 residual stream,
 *   resid_out_t = resid_in_t + W_O concat_h(O[h][t])
 * with the projection accumulated in float32 and added to the stream with one
 * float32 addition per element (no rounding to bf16). The stream then resolves
 * what the attention sublayer adds to it, the quantity whose change under
 * sparsification is the residual drift (Sec. 3, "The Right Objective"): across a
 * stack of layers, calls with O_sparse and W_O and with O_dense and -W_O (exact
 * in bf16) accumulate sum_l W_O(O_sparse - O_dense).
 *   o          device bf16 [H][N][64]
 *   w_o        device bf16 [H*64][H*64], out features x in features (in = 64h + d)
 *   resid_in   device float32 [N][H*64]
 *   resid_out  device float32 [N][H*64] out; may be resid_in (in place), must not
 *              alias o or w_o
 * H must be a multiple of 4. Pointers 16-byte aligned. */
int ress_out_proj_residual_f32(const ress_shape *shape, const void *o, const void *w_o, const float *resid_in,
                               float *resid_out, hipStream_t stream);

/* Human-readable name of a status code (static string). */
const char *ress_status_string(int status);

#ifdef __cplusplus
}
#endif

#endif /* RESS_H */
