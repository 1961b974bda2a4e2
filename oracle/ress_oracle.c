/*
 * ReSS oracle: a plain, slow, float64 CPU implementation of the drift-based block
 * selection and of exact (dense / block-sparse) attention.
 *
 * TEST INFRASTRUCTURE ONLY. It exists to check the GPU path. Only the tests, the
 * smoke check and the benchmark's CPU-baseline leg may load it; the product path
 * never does. It shares no code, header or constant with the GPU library.
 *
 * Paper: "ReSS: Residual-Restoring Sparse Attention for 3D Vision Transformers".
 * Every function names the section / equation it follows. Inputs are bf16 bit
 * patterns (uint16) upcast exactly to float64; the per-head Gram matrix M_h is
 * taken as given (float32, upcast), as the paper computes it once at load time
 * (Eq. 8). All arithmetic is float64, in the paper's order and notation:
 *   P      pooled block attention probabilities (Eq. 1)
 *   e_ij   deviation  vbar_i - V_j  (Eq. 4)
 *   d_ij   P_ij e_ij  (Eq. 5)
 *   s_ij   P_ij ||W_O e_ij|| = P_ij sqrt(e^T M e)  (Eqs. 6, 9)
 *   key    s_ij / max(1 - P_ij, eps)  (Eq. 7)
 *   g, K   net drift and remaining mass of a drop set (Eq. 10)
 *   G, J   g^T M g  and  G / K^2  (Eq. 12)
 *   dJ     exact objective decrease of one restore / drop (Eqs. 14-16)
 *   m_r    swap schedule rho 2^-(r+1) c_h (Eq. 17)
 *
 * Readings where the paper is silent (each is listed in the design notes):
 *   - pooled logits use the attention scale 1/sqrt(D);
 *   - a partial last block is pooled over its valid tokens only;
 *   - the guard max(K, eps) of Eq. 7 is also applied to K in J and dJ;
 *   - ties in every top-k / top-m are broken by lower block index;
 *   - m_r = max(swap_floor, floor(rho c_h 2^-(r+1))), capped by |D| and |S|;
 *   - restore and drop gains of a round are both evaluated at the round-start
 *     state, then applied together; g, K are recomputed from the new drop set and
 *     G = g^T M g exactly (not G + sum of single-swap deltas);
 *   - swaps are always applied; track-best keeps the first drop set with the
 *     strictly smallest J, counting the initial one;
 *   - query blocks that hold special tokens attend densely when asked to.
 *
 * Selection criteria (the paper's comparisons, Table 2 and Fig. 8 / Sec. 6.1):
 *   0  drift (ReSS): keep the c largest keys, rounds minimise J;
 *   1  probability (the SparseVGGT rule): keep the c largest P; optionally capped
 *      by a CDF threshold tau: the shortest prefix in descending P whose mass,
 *      counting the always-kept forced blocks, reaches tau (never below the
 *      two-block floor); rounds, if any, minimise J for the realised count;
 *   2  drift maximisation in the rounds only: initial set as in 0, rounds pick the
 *      swaps that raise J most, track-best keeps the largest J;
 *   3  drift maximisation throughout: keep the c smallest keys, rounds as in 2.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

static double bf16_to_f64(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

static int n_blocks(int N, int b) { return (N + b - 1) / b; }

int ro_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

void ro_set_threads(int n)
{
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/* Block grid and mean pooling (Sec. 3, block-sparse attention step (1)):
 * block i covers tokens [i b, min((i+1) b, N)); its pooled vector is the mean of
 * its tokens. out is [H][n_blocks][D]. */
void ro_pool(int H, int N, int D, int b, const uint16_t *x, double *out)
{
    int nb = n_blocks(N, b);
    for (int h = 0; h < H; ++h)
        for (int i = 0; i < nb; ++i) {
            int lo = i * b, hi = (i + 1) * b < N ? (i + 1) * b : N;
            for (int d = 0; d < D; ++d) {
                double sum = 0.0;
                for (int t = lo; t < hi; ++t)
                    sum += bf16_to_f64(x[((size_t)h * N + t) * D + d]);
                out[((size_t)h * nb + i) * D + d] = sum / (double)(hi - lo);
            }
        }
}

/* Key blocks that hold special tokens are always kept (Sec. 4.1); with the
 * special tokens trailing the patch tokens these are the last key blocks
 * (Supp. F, sink rule). forced is [n_kb], 1 = forced. */
void ro_forced_blocks(int N, int bk, int n_special, unsigned char *forced)
{
    int nkb = n_blocks(N, bk);
    for (int j = 0; j < nkb; ++j) {
        int hi = (j + 1) * bk < N ? (j + 1) * bk : N;
        forced[j] = (n_special > 0 && hi > N - n_special) ? 1 : 0;
    }
}

/* Pooled attention map and dense pooled output of one query block (Eq. 1):
 * P_j = softmax_j(Qbar_i . Kbar_j / sqrt(D)) over all key blocks,
 * vbar_i = sum_j P_j Vbar_j. */
void ro_pooled_row(int D, int nkb, const double *qbar_i, const double *kbar,
                   const double *vbar, double *P, double *vbar_i)
{
    double mx = -INFINITY, z = 0.0;
    double scale = 1.0 / sqrt((double)D);
    for (int j = 0; j < nkb; ++j) {
        double dot = 0.0;
        for (int d = 0; d < D; ++d) dot += qbar_i[d] * kbar[(size_t)j * D + d];
        P[j] = dot * scale;
        if (P[j] > mx) mx = P[j];
    }
    for (int j = 0; j < nkb; ++j) {
        P[j] = exp(P[j] - mx);
        z += P[j];
    }
    for (int j = 0; j < nkb; ++j) P[j] /= z;
    for (int d = 0; d < D; ++d) {
        double acc = 0.0;
        for (int j = 0; j < nkb; ++j) acc += P[j] * vbar[(size_t)j * D + d];
        vbar_i[d] = acc;
    }
}

/* q = e^T M e, the squared residual-space norm ||W_O e||^2 (Eq. 9, first line). */
static double quad_form(int D, const double *M, const double *e)
{
    double q = 0.0;
    for (int a = 0; a < D; ++a) {
        double row = 0.0;
        for (int b = 0; b < D; ++b) row += M[(size_t)a * D + b] * e[b];
        q += e[a] * row;
    }
    return q;
}

/* Block drift score and ranking key of every key block (Eqs. 4-7):
 * e_j = vbar_i - Vbar_j, s_j = P_j sqrt(max(e_j^T M e_j, 0)),
 * key_j = s_j / max(1 - P_j, eps). */
void ro_scores_row(int D, int nkb, const double *P, const double *vbar_i,
                   const double *vbar, const double *M, double eps, double *s, double *key)
{
    double *e = (double *)malloc(sizeof(double) * D);
    for (int j = 0; j < nkb; ++j) {
        for (int d = 0; d < D; ++d) e[d] = vbar_i[d] - vbar[(size_t)j * D + d];
        double q = quad_form(D, M, e);
        s[j] = P[j] * sqrt(q > 0.0 ? q : 0.0);
        double den = 1.0 - P[j];
        key[j] = s[j] / (den > eps ? den : eps);
    }
    free(e);
}

/* Net drift, remaining mass and objective of a drop set (Eqs. 10-12):
 * g = sum_{j in D} P_j e_j, K = 1 - sum_{j in D} P_j, G = g^T M g,
 * J = G / max(K, eps)^2. g_out (length D), K_out, G_out may be NULL. */
double ro_objective(int D, int nkb, const double *P, const double *vbar_i,
                    const double *vbar, const double *M, const unsigned char *inD,
                    double eps, double *g_out, double *K_out, double *G_out)
{
    double *g = (double *)calloc((size_t)D, sizeof(double));
    double mass = 0.0;
    for (int j = 0; j < nkb; ++j) {
        if (!inD[j]) continue;
        for (int d = 0; d < D; ++d) g[d] += P[j] * (vbar_i[d] - vbar[(size_t)j * D + d]);
        mass += P[j];
    }
    double K = 1.0 - mass;
    double G = quad_form(D, M, g);
    double Kh = K > eps ? K : eps;
    if (g_out) memcpy(g_out, g, sizeof(double) * D);
    if (K_out) *K_out = K;
    if (G_out) *G_out = G;
    free(g);
    return G / (Kh * Kh);
}

/* Exact decrease of J for restoring k in D or dropping k in S, at the state of
 * the drop set inD (Eqs. 13-16):
 *   dG+ = -2 d_k^T M g + s_k^2  (restore, u = +P_k)
 *   dG- = +2 d_k^T M g + s_k^2  (drop,    u = -P_k)
 *   dJ  = G / K^2 - (G + dG) / (K + u)^2  with both K guarded by eps.
 * dJ is written for every k with cand[k] set. */
void ro_deltas(int D, int nkb, const double *P, const double *s, const double *vbar_i,
               const double *vbar, const double *M, const unsigned char *inD,
               const unsigned char *cand, double eps, double *dJ)
{
    double *g = (double *)malloc(sizeof(double) * D);
    double *Mg = (double *)malloc(sizeof(double) * D);
    double K, G;
    ro_objective(D, nkb, P, vbar_i, vbar, M, inD, eps, g, &K, &G);
    for (int a = 0; a < D; ++a) {
        double acc = 0.0;
        for (int b = 0; b < D; ++b) acc += M[(size_t)a * D + b] * g[b];
        Mg[a] = acc;
    }
    double Kh = K > eps ? K : eps;
    double J = G / (Kh * Kh);
    for (int k = 0; k < nkb; ++k) {
        if (!cand[k]) continue;
        double ek_Mg = 0.0;
        for (int d = 0; d < D; ++d) ek_Mg += (vbar_i[d] - vbar[(size_t)k * D + d]) * Mg[d];
        double dkMg = P[k] * ek_Mg;
        double dG, u;
        if (inD[k]) {
            dG = -2.0 * dkMg + s[k] * s[k];
            u = P[k];
        } else {
            dG = 2.0 * dkMg + s[k] * s[k];
            u = -P[k];
        }
        double Kn = K + u;
        double Knh = Kn > eps ? Kn : eps;
        dJ[k] = J - (G + dG) / (Knh * Knh);
    }
    free(g);
    free(Mg);
}

/* Total order used by every top-k: larger value first, then lower index. */
typedef struct {
    double v;
    int j;
} ro_item;

static int item_cmp(const void *pa, const void *pb)
{
    const ro_item *a = (const ro_item *)pa, *b = (const ro_item *)pb;
    if (a->v > b->v) return -1;
    if (a->v < b->v) return 1;
    return (a->j < b->j) ? -1 : (a->j > b->j);
}

/* Marks in chosen[] the k members with the largest value under the total order.
 * Returns the gap value_(k) - value_(k+1) between the last chosen and the first
 * unchosen member (+inf when there is no unchosen member or k == 0). */
static double top_k(int n, const double *val, const unsigned char *member, int k,
                    unsigned char *chosen)
{
    ro_item *it = (ro_item *)malloc(sizeof(ro_item) * (n > 0 ? n : 1));
    int cnt = 0;
    for (int j = 0; j < n; ++j) {
        chosen[j] = 0;
        if (member[j]) {
            it[cnt].v = val[j];
            it[cnt].j = j;
            ++cnt;
        }
    }
    qsort(it, (size_t)cnt, sizeof(ro_item), item_cmp);
    if (k > cnt) k = cnt;
    for (int t = 0; t < k; ++t) chosen[it[t].j] = 1;
    double gap = (k > 0 && k < cnt) ? it[k - 1].v - it[k].v : INFINITY;
    free(it);
    return gap;
}

/* Swap count of round r (Eq. 17), with the integer reading documented above. */
int ro_swaps(int c, double rho, int r, int swap_floor)
{
    double m = floor(rho * (double)c * ldexp(1.0, -(r + 1)));
    int mi = (int)m;
    return mi > swap_floor ? mi : swap_floor;
}

static double min2(double a, double b) { return a < b ? a : b; }

/* Full selection for one (query block, head) row (Secs. 4.2-4.3).
 *   forced[j]  key block j is always kept (not a candidate)
 *   c          keep budget c_h (number of kept candidates)
 *   dense_row  the row keeps every block (special-token query block)
 *   criterion, cdf_tau  see the list of criteria at the top of this file
 * Outputs: kept[j] (1 = kept), P, key (forced blocks get key -1), J_init, J_best,
 * margin (smallest relative decision gap along the trajectory), and optionally
 * the trajectory: trace_J[s] and trace_D[s][j] for stages s = 0 (initial set) ..
 * n_stages-1 (one per executed round). */
void ro_select_row(int D, int nkb, const double *qbar_i, const double *kbar,
                   const double *vbar, const double *M, const unsigned char *forced, int c,
                   int rounds, double rho, double eps, int swap_floor, int dense_row,
                   int criterion, double cdf_tau,
                   unsigned char *kept, double *P, double *key, double *J_init,
                   double *J_best, double *margin, double *trace_J,
                   unsigned char *trace_D, int *n_stages)
{
    double *vbar_i = (double *)malloc(sizeof(double) * D);
    double *s = (double *)malloc(sizeof(double) * nkb);
    double *dJ = (double *)malloc(sizeof(double) * nkb);
    unsigned char *cand = (unsigned char *)malloc(nkb);
    unsigned char *inD = (unsigned char *)malloc(nkb);
    unsigned char *best = (unsigned char *)malloc(nkb);
    unsigned char *sel = (unsigned char *)malloc(nkb);
    unsigned char *pick = (unsigned char *)malloc(nkb);

    ro_pooled_row(D, nkb, qbar_i, kbar, vbar, P, vbar_i);
    ro_scores_row(D, nkb, P, vbar_i, vbar, M, eps, s, key);
    int n_p = 0;
    for (int j = 0; j < nkb; ++j) {
        cand[j] = forced[j] ? 0 : 1;
        n_p += cand[j];
        if (forced[j]) key[j] = -1.0;
    }
    double mrg = INFINITY;
    int stages = 0;

    if (dense_row || c >= n_p) {
        for (int j = 0; j < nkb; ++j) kept[j] = 1;
        *J_init = *J_best = 0.0;
        if (trace_J) {
            trace_J[0] = 0.0;
            memset(trace_D, 0, nkb);
        }
        stages = 1;
        goto done;
    }

    /* Initial selection (Eq. 7): keep the c largest keys among the candidates
     * (criterion 1: the c largest P; criterion 3: the c smallest keys). */
    const int maximise = criterion == 2 || criterion == 3;
    {
        double *rank = dJ; /* scratch: the ranking value of each block */
        for (int j = 0; j < nkb; ++j) rank[j] = criterion == 1 ? P[j] : criterion == 3 ? -key[j] : key[j];
        if (criterion == 1 && cdf_tau > 0.0) {
            /* CDF cap: shortest prefix (P descending, lower index first) whose mass
             * together with the forced blocks reaches tau. */
            int n_forced = 0;
            double mass = 0.0;
            for (int j = 0; j < nkb; ++j)
                if (forced[j]) {
                    ++n_forced;
                    mass += P[j];
                }
            int lo = 2 - n_forced > 0 ? 2 - n_forced : 0;
            if (lo > n_p) lo = n_p;
            ro_item *it = (ro_item *)malloc(sizeof(ro_item) * (n_p > 0 ? n_p : 1));
            int cnt = 0;
            for (int j = 0; j < nkb; ++j)
                if (cand[j]) {
                    it[cnt].v = P[j];
                    it[cnt].j = j;
                    ++cnt;
                }
            qsort(it, (size_t)cnt, sizeof(ro_item), item_cmp);
            int n = 0;
            while (n < cnt && mass < cdf_tau) mass += it[n++].v;
            /* decision margin of the cut: distance of the two partial sums around it */
            if (n > 0 && n <= cnt && n < c) {
                double before = mass - it[n - 1].v;
                mrg = min2(mrg, min2(mass - cdf_tau, cdf_tau - before) / cdf_tau);
            }
            free(it);
            if (n < lo) n = lo;
            if (n < c) c = n;
        }
        double gap = top_k(nkb, rank, cand, c, sel);
        double vmax = 0.0;
        for (int j = 0; j < nkb; ++j)
            if (cand[j] && fabs(rank[j]) > vmax) vmax = fabs(rank[j]);
        if (c > 0) mrg = min2(mrg, gap / (vmax > 0.0 ? vmax : 1e-300));
    }
    for (int j = 0; j < nkb; ++j) inD[j] = cand[j] && !sel[j];
    double J = ro_objective(D, nkb, P, vbar_i, vbar, M, inD, eps, NULL, NULL, NULL);
    double Jb = J;
    *J_init = J;
    memcpy(best, inD, nkb);
    if (trace_J) {
        trace_J[0] = J;
        memcpy(trace_D, inD, nkb);
    }
    stages = 1;

    /* Budget-neutral swap rounds (Eqs. 13-17) with track-best. */
    int nD = n_p - c, nS = c;
    for (int r = 0; r < rounds; ++r) {
        int m = ro_swaps(c, rho, r, swap_floor);
        if (m > nD) m = nD;
        if (m > nS) m = nS;
        if (m <= 0) break;
        ro_deltas(D, nkb, P, s, vbar_i, vbar, M, inD, cand, eps, dJ);
        if (maximise) /* the best swaps now raise J the most */
            for (int j = 0; j < nkb; ++j) dJ[j] = -dJ[j];
        unsigned char *memD = sel, *memS = pick; /* reuse buffers */
        unsigned char *restore = (unsigned char *)malloc(nkb);
        unsigned char *drop = (unsigned char *)malloc(nkb);
        for (int j = 0; j < nkb; ++j) {
            memD[j] = inD[j];
            memS[j] = cand[j] && !inD[j];
        }
        double jden = J > 0.0 ? J : 1e-300;
        double gap_r = top_k(nkb, dJ, memD, m, restore);
        double gap_d = top_k(nkb, dJ, memS, m, drop);
        mrg = min2(mrg, gap_r / jden);
        mrg = min2(mrg, gap_d / jden);
        for (int j = 0; j < nkb; ++j) {
            if (restore[j]) inD[j] = 0;
            if (drop[j]) inD[j] = 1;
        }
        free(restore);
        free(drop);
        J = ro_objective(D, nkb, P, vbar_i, vbar, M, inD, eps, NULL, NULL, NULL);
        /* The track-best comparison decides the output only when this stage's
         * drop set differs from the best one (a set revisited has the same J). */
        if (memcmp(inD, best, nkb) != 0) mrg = min2(mrg, fabs(J - Jb) / (Jb > 0.0 ? Jb : 1e-300));
        if (maximise ? J > Jb : J < Jb) {
            Jb = J;
            memcpy(best, inD, nkb);
        }
        if (trace_J) {
            trace_J[stages] = J;
            memcpy(trace_D + (size_t)stages * nkb, inD, nkb);
        }
        ++stages;
    }
    *J_best = Jb;
    for (int j = 0; j < nkb; ++j) kept[j] = forced[j] || (cand[j] && !best[j]);

done:
    *margin = mrg;
    if (n_stages) *n_stages = stages;
    free(vbar_i);
    free(s);
    free(dJ);
    free(cand);
    free(inD);
    free(best);
    free(sel);
    free(pick);
}

/* Query blocks that overlap the special-token tail. */
static int special_query_block(int N, int bq, int n_special, int i)
{
    int hi = (i + 1) * bq < N ? (i + 1) * bq : N;
    return n_special > 0 && hi > N - n_special;
}

/* Selection for a set of (head, query block) rows of one layer.
 * q, k, v: bf16 bits [H][N][D]; gram: float32 [H][D][D]; budgets: [H].
 * rows: flat indices h * n_qb + i (n_rows of them), or NULL for all rows in order.
 * Per selected row r: kept_count[r], kept_idx[r][n_kb] (ascending, -1 padded),
 * drift[r] = (J_init, J_best), key[r][n_kb], prob[r][n_kb], margin[r]
 * (each output may be NULL except kept_count and kept_idx). */
int ro_select(int H, int N, int D, int bq, int bk, int n_special, const uint16_t *q,
              const uint16_t *k, const uint16_t *v, const float *gram, const int *budgets,
              int rounds, double rho, double eps, int swap_floor, int dense_special_queries,
              int criterion, double cdf_tau,
              int n_rows, const int *rows, int *kept_count, int *kept_idx, double *drift,
              double *key, double *prob, double *margin)
{
    int nqb = n_blocks(N, bq), nkb = n_blocks(N, bk);
    if (rows == NULL) n_rows = H * nqb;
    double *qbar = (double *)malloc(sizeof(double) * (size_t)H * nqb * D + 8);
    double *kbar = (double *)malloc(sizeof(double) * (size_t)H * nkb * D + 8);
    double *vbar = (double *)malloc(sizeof(double) * (size_t)H * nkb * D + 8);
    double *M = (double *)malloc(sizeof(double) * (size_t)H * D * D + 8);
    unsigned char *forced = (unsigned char *)malloc((size_t)nkb + 1);
    ro_pool(H, N, D, bq, q, qbar);
    ro_pool(H, N, D, bk, k, kbar);
    ro_pool(H, N, D, bk, v, vbar);
    for (size_t t = 0; t < (size_t)H * D * D; ++t) M[t] = (double)gram[t];
    ro_forced_blocks(N, bk, n_special, forced);

#pragma omp parallel for schedule(dynamic, 1)
    for (int r = 0; r < n_rows; ++r) {
        int flat = rows ? rows[r] : r;
        int h = flat / nqb, i = flat % nqb;
        unsigned char *kept = (unsigned char *)malloc((size_t)nkb + 1);
        double *P = (double *)malloc(sizeof(double) * (nkb + 1));
        double *ky = (double *)malloc(sizeof(double) * (nkb + 1));
        double J0, Jb, mg;
        int dense = dense_special_queries && special_query_block(N, bq, n_special, i);
        ro_select_row(D, nkb, qbar + ((size_t)h * nqb + i) * D, kbar + (size_t)h * nkb * D,
                      vbar + (size_t)h * nkb * D, M + (size_t)h * D * D, forced, budgets[h],
                      rounds, rho, eps, swap_floor, dense, criterion, cdf_tau, kept, P, ky, &J0,
                      &Jb, &mg, NULL, NULL, NULL);
        int cnt = 0;
        for (int j = 0; j < nkb; ++j)
            if (kept[j]) kept_idx[(size_t)r * nkb + cnt++] = j;
        for (int t = cnt; t < nkb; ++t) kept_idx[(size_t)r * nkb + t] = -1;
        kept_count[r] = cnt;
        if (drift) {
            drift[2 * (size_t)r] = J0;
            drift[2 * (size_t)r + 1] = Jb;
        }
        if (key) memcpy(key + (size_t)r * nkb, ky, sizeof(double) * nkb);
        if (prob) memcpy(prob + (size_t)r * nkb, P, sizeof(double) * nkb);
        if (margin) margin[r] = mg;
        free(kept);
        free(P);
        free(ky);
    }
    free(qbar);
    free(kbar);
    free(vbar);
    free(M);
    free(forced);
    return 0;
}

/* Exact attention for selected query tokens (Sec. 3, step (3)): softmax of
 * scale * Q_t . K_s over the key tokens s of the kept key blocks of the token's
 * query block (every key block when kept_idx is NULL), renormalised among them,
 * applied to V. An empty key set gives a zero output.
 * kept_count: [H][n_qb]; kept_idx: [H][n_qb][n_kb], entries past the count ignored.
 * out: [n_sel][D] float64. */
void ro_attn_tokens(int H, int N, int D, int bq, int bk, const uint16_t *q, const uint16_t *k,
                    const uint16_t *v, double scale, const int *kept_count, const int *kept_idx,
                    int n_sel, const int *sel_h, const int *sel_t, double *out)
{
    int nqb = n_blocks(N, bq), nkb = n_blocks(N, bk);
    (void)H;
#pragma omp parallel for schedule(dynamic, 4)
    for (int u = 0; u < n_sel; ++u) {
        int h = sel_h[u], t = sel_t[u], i = t / bq;
        double *qt = (double *)malloc(sizeof(double) * D);
        double *acc = (double *)calloc((size_t)D, sizeof(double));
        double *lg = (double *)malloc(sizeof(double) * (size_t)(N > 0 ? N : 1));
        int *blk = (int *)malloc(sizeof(int) * (nkb > 0 ? nkb : 1));
        int nblk = 0;
        if (kept_idx) {
            int cnt = kept_count[(size_t)h * nqb + i];
            for (int m = 0; m < cnt; ++m) blk[nblk++] = kept_idx[((size_t)h * nqb + i) * nkb + m];
        } else {
            for (int j = 0; j < nkb; ++j) blk[nblk++] = j;
        }
        for (int d = 0; d < D; ++d) qt[d] = bf16_to_f64(q[((size_t)h * N + t) * D + d]);
        double mx = -INFINITY;
        int ns = 0;
        for (int b = 0; b < nblk; ++b) {
            int lo = blk[b] * bk, hi = (blk[b] + 1) * bk < N ? (blk[b] + 1) * bk : N;
            for (int s = lo; s < hi; ++s) {
                double dot = 0.0;
                for (int d = 0; d < D; ++d) dot += qt[d] * bf16_to_f64(k[((size_t)h * N + s) * D + d]);
                lg[ns] = dot * scale;
                if (lg[ns] > mx) mx = lg[ns];
                ++ns;
            }
        }
        double z = 0.0;
        ns = 0;
        for (int b = 0; b < nblk; ++b) {
            int lo = blk[b] * bk, hi = (blk[b] + 1) * bk < N ? (blk[b] + 1) * bk : N;
            for (int s = lo; s < hi; ++s) {
                double p = exp(lg[ns++] - mx);
                z += p;
                for (int d = 0; d < D; ++d) acc[d] += p * bf16_to_f64(v[((size_t)h * N + s) * D + d]);
            }
        }
        for (int d = 0; d < D; ++d) out[(size_t)u * D + d] = z > 0.0 ? acc[d] / z : 0.0;
        free(qt);
        free(acc);
        free(lg);
        free(blk);
    }
}
