/*
 * apml_oracle.c - CPU oracle for the sparse APML loss, forward and backward.
 *
 * TEST INFRASTRUCTURE. Only the tests, the smoke check and the benchmark's CPU
 * baseline load this library. It shares no code, header or table with the GPU
 * library, and nothing on the GPU path may call it.
 *
 * It computes, plainly and slowly, what the paper defines, in the paper's
 * order (Algorithm 1) and in double precision:
 *   1. cost C_ij = ||x_i - y_j||_2                          (Sec. III-A)
 *   2. per row: min and second min of the cost, gap, clamp,
 *      temperature (Eq. 1 with the clamp of Sec. III-D); count of kept
 *      entries s_ij >= tau (Sec. III-B); exclusive scan; rewrite of the
 *      kept entries normalised by the kept sum (Sec. III-C)  (Alg. 1, step 1)
 *   3. the same per column with roles swapped                (Alg. 1, step 2)
 *   4. symmetrization: concatenate both COO streams, sort by the 64-bit key
 *      i*M + j, merge duplicates into P0 = (P_row + P_col)/2 (Sec. III-A
 *      initial plan, Sec. III-C, Alg. 1 step 3)
 *   5. Sinkhorn: column scaling (Eq. 3) then row scaling (Eq. 4), L times,
 *      with dense length-M / length-N accumulation buffers   (Alg. 1, steps 4-7)
 *   6. loss = sum_t v_t ||x_{i_t} - y_{j_t}||_2               (Sec. III-D)
 *   7. reverse mode through 6..1 written out by hand, with the distance
 *      gradient of Eq. 5.
 *
 * Readings where the paper is silent or ambiguous:
 *   R1  The cost is the Euclidean (not squared) distance.
 *   R2  The minimum and second minimum are decided on the squared distance in
 *       single precision (the paper's precision), from the coordinates rounded
 *       to float, as dx*dx, then fma(dy,dy,.), then fma(dz,dz,.) with
 *       d = x - y in float.  Ties go to the smallest index; the second minimum
 *       is the second order statistic of the multiset (a tie with the minimum
 *       gives a zero gap).  The cost values of the two selected entries are
 *       then taken in double precision.
 *   R3  The gap is clamped, g = max(C2 - C1 + delta, eps_g) (Sec. III-D states
 *       that the clamp replaces the uniform fallback); a clamped row carries no
 *       gradient through its temperature.
 *   R4  K in Eq. 1 is the full row (M) or column (N) length.
 *   R5  The threshold is inclusive, s >= tau, on the min-shifted unnormalised
 *       similarity, and a row is normalised by the sum of its kept entries.
 *   R6  Duplicates are merged as P0 = (P_row + P_col)/2 with an absent side
 *       counted as zero, which is the dense initial plan restricted to the
 *       union support.
 *   R7  The loss is the plain per-sample sum (no 1/N, no batch mean).
 *   R8  eps_dist appears only in the gradient (Eq. 5), not in the forward cost.
 *   R9  No gradient flows through the choice of the support or of the argmins.
 *
 * Variants (selected by orc_params, for ablation):
 *   gap_mode = 1     uniform fallback instead of the clamp: an owner whose gap
 *                    C2 - C1 is below eps_g gets P = 1/K on all K entries
 *                    (Sec. III-A; the kernel of Sec. III-C writes it), which is
 *                    the softmax at T = 0; no gradient flows through it.
 *   sym_mode = 1     duplicates averaged literally (Sec. III-C, Alg. 1 step 3):
 *                    P0 = (P_row + P_col)/2 where both directions keep the
 *                    pair, the one present value elsewhere.
 *   tgrad_mode = 1   the temperature is a constant in the backward pass.
 *   select_mode = 1  the minimum and second minimum are decided on the cost
 *                    in double precision instead of reading R2 (the paper
 *                    defines them on C, Sec. III-A, Eq. 1; this variant
 *                    measures how much the single-precision decision moves
 *                    the result).
 *
 * Build: gcc -O2 -fopenmp -ffp-contract=off -fPIC -shared (fmaf is the
 * correctly rounded C library fused multiply-add).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

typedef struct {
    double p_min;    /* minimum probability of the nearest entry (Eq. 1) */
    double tau;      /* pruning threshold on s (Sec. III-B) */
    double eps_stab; /* Sinkhorn stability constant (Eq. 3, Eq. 4) */
    double delta;    /* gap offset g = c2 + delta (Sec. III-A) */
    double eps_gap;  /* gap clamp (Sec. III-D) */
    double eps_dist; /* distance-gradient guard (Eq. 5) */
    int32_t n_iter;  /* L_iter */
    int32_t gap_mode;   /* 0: clamp (Sec. III-D); 1: uniform fallback (Sec. III-A, III-C) */
    int32_t sym_mode;   /* 0: P0 = (P_row + P_col)/2, absent side 0; 1: mean of the present sides */
    int32_t tgrad_mode; /* 0: full gradient; 1: temperature treated as a constant */
    int32_t select_mode; /* 0: minima decided in single precision (R2); 1: in double precision */
} orc_params;

enum { ORC_GAP_CLAMP = 0, ORC_GAP_FALLBACK = 1 };
enum { ORC_SYM_HALF_SUM = 0, ORC_SYM_MEAN_DUP = 1 };
enum { ORC_TGRAD_FULL = 0, ORC_TGRAD_DETACHED = 1 };

enum { ORC_ROW = 1, ORC_COL = 2 };
enum { ORC_OK = 0, ORC_BAD_ARG = 1, ORC_NO_MEMORY = 2 };

/* ------------------------------------------------------------------------ */
/* distances                                                                */
/* ------------------------------------------------------------------------ */

/* Squared distance in single precision (reading R2): the precision in which
 * the minimum and second minimum are decided. */
static float sqdist_single(const double *a, const double *b)
{
    const float dx = (float)a[0] - (float)b[0];
    const float dy = (float)a[1] - (float)b[1];
    const float dz = (float)a[2] - (float)b[2];
    float s = dx * dx;
    s = fmaf(dy, dy, s);
    s = fmaf(dz, dz, s);
    return s;
}

/* Squared distance in double precision (the select_mode = 1 variant). The
 * order of a square root is that of its argument, so deciding on it decides
 * on the cost itself. */
static double sqdist_double(const double *a, const double *b)
{
    const double dx = a[0] - b[0], dy = a[1] - b[1], dz = a[2] - b[2];
    return dx * dx + dy * dy + dz * dz;
}

/* Cost C = ||a - b||_2 (Sec. III-A), double precision. */
static double cost(const double *a, const double *b)
{
    const double dx = a[0] - b[0], dy = a[1] - b[1], dz = a[2] - b[2];
    return sqrt(dx * dx + dy * dy + dz * dz);
}

/* ------------------------------------------------------------------------ */
/* one direction of the adaptive softmax (Alg. 1 steps 1 and 2)            */
/* ------------------------------------------------------------------------ */

/* Per-owner statistics of one direction. "Owner" is a row (a point of X) in
 * the row direction and a column (a point of Y) in the column direction. */
typedef struct {
    double T;      /* temperature, Eq. 1 (0 for a uniform fallback) */
    double c1;     /* minimum cost of the owner */
    double g;      /* clamped gap */
    int32_t k1;    /* index of the minimum */
    int32_t k2;    /* index of the second minimum */
    uint8_t clamped; /* the gap was clamped, or the fallback taken: no temperature gradient */
} owner_stats;

/* Minimum, second minimum, gap and temperature of the cost vector between
 * point p and the K points of Q (Sec. III-A, Eq. 1, clamp of Sec. III-D). */
static void owner_statistics(const double *p, const double *Q, int K, const orc_params *prm,
                             owner_stats *st)
{
    double m1 = INFINITY, m2 = INFINITY;
    int k1 = -1, k2 = -1;
    for (int k = 0; k < K; ++k) {
        const double d = prm->select_mode ? sqdist_double(p, Q + 3 * (size_t)k)
                                          : (double)sqdist_single(p, Q + 3 * (size_t)k);
        if (d < m1) {
            m2 = m1;
            k2 = k1;
            m1 = d;
            k1 = k;
        } else if (d < m2) {
            m2 = d;
            k2 = k;
        }
    }
    st->k1 = k1;
    st->k2 = k2;
    st->c1 = cost(p, Q + 3 * (size_t)k1);
    const double c2 = cost(p, Q + 3 * (size_t)k2);
    const double gap = (c2 - st->c1) + prm->delta; /* g = c~(2) + delta */
    st->clamped = gap < prm->eps_gap;             /* max(gap, eps_g) */
    st->g = st->clamped ? prm->eps_gap : gap;
    /* Eq. 1: T = -log((1 - p_min) / ((K - 1) p_min)) / g */
    st->T = -log((1.0 - prm->p_min) / ((double)(K - 1) * prm->p_min)) / st->g;
    if (prm->gap_mode == ORC_GAP_FALLBACK && c2 - st->c1 < prm->eps_gap) {
        /* uniform fallback: s = 1 for every entry, all kept, P = 1/K */
        st->T = 0.0;
        st->g = gap;
        st->clamped = 1;
    }
}

/* Unnormalised similarity s = exp(-T (C - C_min)) (Sec. III-B). */
static double similarity(const owner_stats *st, double c)
{
    return exp(-st->T * (c - st->c1));
}

typedef struct {
    int64_t nnz;
    int32_t *own; /* owner index (row i, or column j) */
    int32_t *oth; /* other index */
    double *val;  /* normalised probability on the kept support */
} coo_stream;

/* Pass 1 (count), exclusive scan, pass 2 (write and normalise by the kept
 * sum) for every owner in P against all points of Q (Sec. III-C). */
static int softmax_direction(const double *P, int nP, const double *Q, int nQ,
                             const orc_params *prm, int nthreads, owner_stats *st,
                             coo_stream *out)
{
    int64_t *offset = (int64_t *)calloc((size_t)nP + 1, sizeof(int64_t));
    if (!offset)
        return ORC_NO_MEMORY;

    /* pass 1: statistics, then the count of entries with s >= tau */
#pragma omp parallel for num_threads(nthreads) schedule(dynamic, 8)
    for (int a = 0; a < nP; ++a) {
        const double *p = P + 3 * (size_t)a;
        owner_statistics(p, Q, nQ, prm, &st[a]);
        int64_t count = 0;
        for (int b = 0; b < nQ; ++b)
            if (similarity(&st[a], cost(p, Q + 3 * (size_t)b)) >= prm->tau)
                ++count;
        offset[a + 1] = count;
    }
    /* exclusive prefix sum of the counts: write offsets and nnz */
    for (int a = 0; a < nP; ++a)
        offset[a + 1] += offset[a];
    out->nnz = offset[nP];
    out->own = (int32_t *)malloc((size_t)out->nnz * sizeof(int32_t) + 1);
    out->oth = (int32_t *)malloc((size_t)out->nnz * sizeof(int32_t) + 1);
    out->val = (double *)malloc((size_t)out->nnz * sizeof(double) + 1);
    if (!out->own || !out->oth || !out->val) {
        free(offset);
        return ORC_NO_MEMORY;
    }

    /* pass 2: rescan, write kept triples, normalise by the kept sum */
#pragma omp parallel for num_threads(nthreads) schedule(dynamic, 8)
    for (int a = 0; a < nP; ++a) {
        const double *p = P + 3 * (size_t)a;
        int64_t k = offset[a];
        double z = 0.0;
        for (int b = 0; b < nQ; ++b) {
            const double s = similarity(&st[a], cost(p, Q + 3 * (size_t)b));
            if (s >= prm->tau) {
                out->own[k] = a;
                out->oth[k] = b;
                out->val[k] = s;
                z += s;
                ++k;
            }
        }
        for (int64_t t = offset[a]; t < offset[a + 1]; ++t)
            out->val[t] /= z;
    }
    free(offset);
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* symmetrization (Alg. 1 step 3)                                           */
/* ------------------------------------------------------------------------ */

typedef struct {
    int64_t key; /* i*M + j */
    int32_t i, j;
    int32_t dir; /* ORC_ROW or ORC_COL */
    double val;
} stream_item;

static int item_order(const void *pa, const void *pb)
{
    const stream_item *a = (const stream_item *)pa, *b = (const stream_item *)pb;
    if (a->key != b->key)
        return a->key < b->key ? -1 : 1;
    return a->dir - b->dir;
}

/* ------------------------------------------------------------------------ */
/* per-sample result                                                        */
/* ------------------------------------------------------------------------ */

typedef struct orc_result {
    int N, M, L;
    int64_t nnz;
    int32_t *ei, *ej;
    uint8_t *ef;
    double *p_row, *p_col, *p0, *C;
    owner_stats *row, *col;
    double *hist;   /* (2L+1) plans: [0] = P0, [2l-1] after column step l, [2l] after row step l */
    double *colsum; /* L x M: S^l */
    double *rowsum; /* L x N: R^l */
    double loss;
    double *gx, *gy; /* N x 3, M x 3, or NULL */
} orc_result;

void orc_free(orc_result *r)
{
    if (!r)
        return;
    free(r->ei);
    free(r->ej);
    free(r->ef);
    free(r->p_row);
    free(r->p_col);
    free(r->p0);
    free(r->C);
    free(r->row);
    free(r->col);
    free(r->hist);
    free(r->colsum);
    free(r->rowsum);
    free(r->gx);
    free(r->gy);
    free(r);
}

static int valid(int N, int M, const orc_params *p)
{
    if (N < 2 || M < 2 || !p)
        return 0;
    if (!(p->p_min > 0.0 && p->p_min < 1.0))
        return 0;
    if (!(p->p_min * N > 1.0 && p->p_min * M > 1.0)) /* T > 0 needs K p_min > 1 */
        return 0;
    if (!(p->tau >= 0.0 && p->tau <= 1.0) || p->n_iter < 0)
        return 0;
    if (!(p->delta >= 0.0) || !(p->eps_gap > 0.0) || !(p->eps_stab >= 0.0) || !(p->eps_dist >= 0.0))
        return 0;
    if ((unsigned)p->gap_mode > 1u || (unsigned)p->sym_mode > 1u || (unsigned)p->tgrad_mode > 1u ||
        (unsigned)p->select_mode > 1u)
        return 0;
    return 1;
}

/* Gradient of the loss with respect to the cost of one entry, pushed to the
 * two points by Eq. 5: dC/dx = (x - y) / (C + eps_dist), dC/dy = -dC/dx. */
static void push_cost_gradient(const double *x, const double *y, double cbar, double eps_dist,
                               double *gx, double *gy)
{
    const double c = cost(x, y);
    for (int k = 0; k < 3; ++k) {
        const double d = cbar * (x[k] - y[k]) / (c + eps_dist);
        gx[k] += d;
        gy[k] -= d;
    }
}

/* Forward (and, if want_grad, backward with upstream gradient gbar) of one
 * sample. x: N x 3, y: M x 3, both double (the float inputs widened). */
int orc_run(const double *x, const double *y, int N, int M, const orc_params *prm, int want_grad,
            double gbar, int nthreads, orc_result **out)
{
    *out = NULL;
    if (!x || !y || !valid(N, M, prm))
        return ORC_BAD_ARG;
#ifdef _OPENMP
    if (nthreads <= 0)
        nthreads = omp_get_max_threads();
#else
    nthreads = 1;
#endif
    const int L = prm->n_iter;
    orc_result *r = (orc_result *)calloc(1, sizeof(orc_result));
    if (!r)
        return ORC_NO_MEMORY;
    r->N = N;
    r->M = M;
    r->L = L;
    r->row = (owner_stats *)calloc((size_t)N, sizeof(owner_stats));
    r->col = (owner_stats *)calloc((size_t)M, sizeof(owner_stats));
    coo_stream rs = {0}, cs = {0};
    stream_item *items = NULL;
    int rc = ORC_NO_MEMORY;
    if (!r->row || !r->col)
        goto fail;

    /* Alg. 1 step 1: row direction (owners = X, K = M) */
    if ((rc = softmax_direction(x, N, y, M, prm, nthreads, r->row, &rs)) != ORC_OK)
        goto fail;
    /* Alg. 1 step 2: column direction (owners = Y, K = N) */
    if ((rc = softmax_direction(y, M, x, N, prm, nthreads, r->col, &cs)) != ORC_OK)
        goto fail;
    rc = ORC_NO_MEMORY;

    /* Alg. 1 step 3: concatenate, sort by key i*M + j, merge duplicates */
    const int64_t n_items = rs.nnz + cs.nnz;
    items = (stream_item *)malloc((size_t)n_items * sizeof(stream_item) + 1);
    if (!items)
        goto fail;
    for (int64_t t = 0; t < rs.nnz; ++t) {
        stream_item it = {(int64_t)rs.own[t] * M + rs.oth[t], rs.own[t], rs.oth[t], ORC_ROW, rs.val[t]};
        items[t] = it;
    }
    for (int64_t t = 0; t < cs.nnz; ++t) {
        stream_item it = {(int64_t)cs.oth[t] * M + cs.own[t], cs.oth[t], cs.own[t], ORC_COL, cs.val[t]};
        items[rs.nnz + t] = it;
    }
    qsort(items, (size_t)n_items, sizeof(stream_item), item_order);
    int64_t nnz = 0;
    for (int64_t t = 0; t < n_items; ++t)
        if (t == 0 || items[t].key != items[t - 1].key)
            ++nnz;
    r->nnz = nnz;
    r->ei = (int32_t *)malloc((size_t)nnz * sizeof(int32_t) + 1);
    r->ej = (int32_t *)malloc((size_t)nnz * sizeof(int32_t) + 1);
    r->ef = (uint8_t *)calloc((size_t)nnz + 1, 1);
    r->p_row = (double *)calloc((size_t)nnz + 1, sizeof(double));
    r->p_col = (double *)calloc((size_t)nnz + 1, sizeof(double));
    r->p0 = (double *)calloc((size_t)nnz + 1, sizeof(double));
    r->C = (double *)malloc((size_t)nnz * sizeof(double) + 1);
    if (!r->ei || !r->ej || !r->ef || !r->p_row || !r->p_col || !r->p0 || !r->C)
        goto fail;
    for (int64_t t = 0, e = -1; t < n_items; ++t) {
        if (t == 0 || items[t].key != items[t - 1].key) {
            ++e;
            r->ei[e] = items[t].i;
            r->ej[e] = items[t].j;
        }
        r->ef[e] |= (uint8_t)items[t].dir;
        if (items[t].dir == ORC_ROW)
            r->p_row[e] = items[t].val;
        else
            r->p_col[e] = items[t].val;
    }
    for (int64_t t = 0; t < nnz; ++t) {
        if (prm->sym_mode == ORC_SYM_MEAN_DUP && r->ef[t] != (ORC_ROW | ORC_COL))
            r->p0[t] = r->p_row[t] + r->p_col[t]; /* one side present: its value */
        else
            r->p0[t] = 0.5 * (r->p_row[t] + r->p_col[t]); /* initial plan P0 = (P_row + P_col)/2 */
        r->C[t] = cost(x + 3 * (size_t)r->ei[t], y + 3 * (size_t)r->ej[t]);
    }
    free(items);
    items = NULL;
    free(rs.own), free(rs.oth), free(rs.val), free(cs.own), free(cs.oth), free(cs.val);
    memset(&rs, 0, sizeof rs);
    memset(&cs, 0, sizeof cs);

    /* Alg. 1 steps 4-7: Sinkhorn on the COO values, every plan kept */
    r->hist = (double *)malloc((size_t)(2 * L + 1) * (size_t)nnz * sizeof(double) + 1);
    r->colsum = (double *)calloc((size_t)L * M + 1, sizeof(double));
    r->rowsum = (double *)calloc((size_t)L * N + 1, sizeof(double));
    if (!r->hist || !r->colsum || !r->rowsum)
        goto fail;
    memcpy(r->hist, r->p0, (size_t)nnz * sizeof(double));
    const double eps = prm->eps_stab;
    for (int l = 1; l <= L; ++l) {
        const double *prev = r->hist + (size_t)(2 * l - 2) * nnz;
        double *w = r->hist + (size_t)(2 * l - 1) * nnz;
        double *u = r->hist + (size_t)(2 * l) * nnz;
        double *S = r->colsum + (size_t)(l - 1) * M;
        double *R = r->rowsum + (size_t)(l - 1) * N;
        for (int64_t t = 0; t < nnz; ++t) /* column sums into a dense length-M buffer */
            S[r->ej[t]] += prev[t];
        for (int64_t t = 0; t < nnz; ++t) /* Eq. 3 */
            w[t] = prev[t] / (S[r->ej[t]] + eps);
        for (int64_t t = 0; t < nnz; ++t) /* row sums into a dense length-N buffer */
            R[r->ei[t]] += w[t];
        for (int64_t t = 0; t < nnz; ++t) /* Eq. 4 */
            u[t] = w[t] / (R[r->ei[t]] + eps);
    }
    const double *v = r->hist + (size_t)(2 * L) * nnz;

    /* Sec. III-D: loss on the stored pairs */
    double loss = 0.0;
    for (int64_t t = 0; t < nnz; ++t)
        loss += v[t] * r->C[t];
    r->loss = loss;

    if (want_grad) {
        r->gx = (double *)calloc((size_t)N * 3, sizeof(double));
        r->gy = (double *)calloc((size_t)M * 3, sizeof(double));
        double *vbar = (double *)malloc((size_t)nnz * sizeof(double) + 1);
        double *cbar = (double *)malloc((size_t)nnz * sizeof(double) + 1);
        double *rowacc = (double *)calloc((size_t)N, sizeof(double));
        double *colacc = (double *)calloc((size_t)M, sizeof(double));
        double *Tbar_r = (double *)calloc((size_t)N, sizeof(double));
        double *Tbar_c = (double *)calloc((size_t)M, sizeof(double));
        if (!r->gx || !r->gy || !vbar || !cbar || !rowacc || !colacc || !Tbar_r || !Tbar_c) {
            free(vbar), free(cbar), free(rowacc), free(colacc), free(Tbar_r), free(Tbar_c);
            goto fail;
        }
        /* loss = sum v_t C_t: direct terms */
        for (int64_t t = 0; t < nnz; ++t) {
            vbar[t] = gbar * r->C[t];
            cbar[t] = gbar * v[t];
        }
        /* Sinkhorn adjoint, last iteration first. For u = w / (R + eps),
         * R = sum_row w:  wbar = (ubar - sum_row(ubar * u)) / (R + eps). */
        for (int l = L; l >= 1; --l) {
            const double *w = r->hist + (size_t)(2 * l - 1) * nnz;
            const double *u = r->hist + (size_t)(2 * l) * nnz;
            const double *S = r->colsum + (size_t)(l - 1) * M;
            const double *R = r->rowsum + (size_t)(l - 1) * N;
            memset(rowacc, 0, (size_t)N * sizeof(double));
            for (int64_t t = 0; t < nnz; ++t)
                rowacc[r->ei[t]] += vbar[t] * u[t];
            for (int64_t t = 0; t < nnz; ++t) /* adjoint of Eq. 4 */
                vbar[t] = (vbar[t] - rowacc[r->ei[t]]) / (R[r->ei[t]] + eps);
            memset(colacc, 0, (size_t)M * sizeof(double));
            for (int64_t t = 0; t < nnz; ++t)
                colacc[r->ej[t]] += vbar[t] * w[t];
            for (int64_t t = 0; t < nnz; ++t) /* adjoint of Eq. 3 */
                vbar[t] = (vbar[t] - colacc[r->ej[t]]) / (S[r->ej[t]] + eps);
        }
        /* vbar is now dLoss/dP0. P0 = (P_row + P_col)/2 on the union support
         * (or, averaging duplicates literally, the one present value where only
         * one direction keeps the pair): dP0/dP_row = wgt. */
        for (int64_t t = 0; t < nnz; ++t) {
            const double wgt = prm->sym_mode == ORC_SYM_MEAN_DUP && r->ef[t] != (ORC_ROW | ORC_COL) ? 1.0 : 0.5;
            vbar[t] *= wgt; /* from here on: the adjoint of P_row (and of P_col) */
        }
        /* Row softmax adjoint: P_row = s / Z over the kept set, s = exp(-T (C - C1)).
         * abar = P (Pbar - sum P Pbar); Cbar += -T abar; Tbar += -abar (C - C1).
         * A uniform fallback (T = 0) is a constant: nothing flows through it. */
        memset(rowacc, 0, (size_t)N * sizeof(double));
        for (int64_t t = 0; t < nnz; ++t)
            if (r->ef[t] & ORC_ROW)
                rowacc[r->ei[t]] += r->p_row[t] * vbar[t];
        for (int64_t t = 0; t < nnz; ++t)
            if ((r->ef[t] & ORC_ROW) && r->row[r->ei[t]].T != 0.0) {
                const int i = r->ei[t];
                const double a = r->p_row[t] * (vbar[t] - rowacc[i]);
                cbar[t] += -r->row[i].T * a;
                Tbar_r[i] += -a * (r->C[t] - r->row[i].c1);
            }
        /* Column softmax adjoint, the same with roles swapped. */
        memset(colacc, 0, (size_t)M * sizeof(double));
        for (int64_t t = 0; t < nnz; ++t)
            if (r->ef[t] & ORC_COL)
                colacc[r->ej[t]] += r->p_col[t] * vbar[t];
        for (int64_t t = 0; t < nnz; ++t)
            if ((r->ef[t] & ORC_COL) && r->col[r->ej[t]].T != 0.0) {
                const int j = r->ej[t];
                const double a = r->p_col[t] * (vbar[t] - colacc[j]);
                cbar[t] += -r->col[j].T * a;
                Tbar_c[j] += -a * (r->C[t] - r->col[j].c1);
            }
        /* Distance gradient on the stored pairs (Eq. 5). */
        for (int64_t t = 0; t < nnz; ++t)
            push_cost_gradient(x + 3 * (size_t)r->ei[t], y + 3 * (size_t)r->ej[t], cbar[t],
                               prm->eps_dist, r->gx + 3 * (size_t)r->ei[t], r->gy + 3 * (size_t)r->ej[t]);
        /* Temperature adjoint: T = L_K / g, g = C2 - C1 + delta unless clamped.
         * gbar = Tbar dT/dg = -Tbar T / g; it reaches the costs of the minimum
         * (with sign -) and of the second minimum (with sign +). */
        const int detached = prm->tgrad_mode == ORC_TGRAD_DETACHED;
        for (int i = 0; i < N; ++i) {
            const owner_stats *s = &r->row[i];
            if (s->clamped || detached)
                continue;
            const double gb = -Tbar_r[i] * s->T / s->g;
            push_cost_gradient(x + 3 * (size_t)i, y + 3 * (size_t)s->k2, gb, prm->eps_dist,
                               r->gx + 3 * (size_t)i, r->gy + 3 * (size_t)s->k2);
            push_cost_gradient(x + 3 * (size_t)i, y + 3 * (size_t)s->k1, -gb, prm->eps_dist,
                               r->gx + 3 * (size_t)i, r->gy + 3 * (size_t)s->k1);
        }
        for (int j = 0; j < M; ++j) {
            const owner_stats *s = &r->col[j];
            if (s->clamped || detached)
                continue;
            const double gb = -Tbar_c[j] * s->T / s->g;
            push_cost_gradient(x + 3 * (size_t)s->k2, y + 3 * (size_t)j, gb, prm->eps_dist,
                               r->gx + 3 * (size_t)s->k2, r->gy + 3 * (size_t)j);
            push_cost_gradient(x + 3 * (size_t)s->k1, y + 3 * (size_t)j, -gb, prm->eps_dist,
                               r->gx + 3 * (size_t)s->k1, r->gy + 3 * (size_t)j);
        }
        free(vbar), free(cbar), free(rowacc), free(colacc), free(Tbar_r), free(Tbar_c);
    }
    *out = r;
    return ORC_OK;

fail:
    free(items);
    free(rs.own), free(rs.oth), free(rs.val), free(cs.own), free(cs.oth), free(cs.val);
    orc_free(r);
    return rc;
}

/* ------------------------------------------------------------------------ */
/* accessors                                                                */
/* ------------------------------------------------------------------------ */

/* Threads an OpenMP region of the oracle uses when nthreads <= 0. */
int orc_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

int64_t orc_nnz(const orc_result *r) { return r->nnz; }
double orc_loss(const orc_result *r) { return r->loss; }

/* Stored entries in (i, j) order with their flags, P_row, P_col, P0, the
 * final plan v and the cost C. Any output pointer may be NULL. */
void orc_entries(const orc_result *r, int32_t *i, int32_t *j, uint8_t *flags, double *p_row,
                 double *p_col, double *p0, double *v, double *C)
{
    const int64_t n = r->nnz;
    if (i) memcpy(i, r->ei, (size_t)n * sizeof(int32_t));
    if (j) memcpy(j, r->ej, (size_t)n * sizeof(int32_t));
    if (flags) memcpy(flags, r->ef, (size_t)n);
    if (p_row) memcpy(p_row, r->p_row, (size_t)n * sizeof(double));
    if (p_col) memcpy(p_col, r->p_col, (size_t)n * sizeof(double));
    if (p0) memcpy(p0, r->p0, (size_t)n * sizeof(double));
    if (v) memcpy(v, r->hist + (size_t)(2 * r->L) * n, (size_t)n * sizeof(double));
    if (C) memcpy(C, r->C, (size_t)n * sizeof(double));
}

static void export_stats(const owner_stats *s, int n, double *T, double *c1, double *g,
                         int32_t *k1, int32_t *k2, uint8_t *clamped)
{
    for (int a = 0; a < n; ++a) {
        if (T) T[a] = s[a].T;
        if (c1) c1[a] = s[a].c1;
        if (g) g[a] = s[a].g;
        if (k1) k1[a] = s[a].k1;
        if (k2) k2[a] = s[a].k2;
        if (clamped) clamped[a] = s[a].clamped;
    }
}

void orc_row_stats(const orc_result *r, double *T, double *c1, double *g, int32_t *k1, int32_t *k2,
                   uint8_t *clamped)
{
    export_stats(r->row, r->N, T, c1, g, k1, k2, clamped);
}

void orc_col_stats(const orc_result *r, double *T, double *c1, double *g, int32_t *k1, int32_t *k2,
                   uint8_t *clamped)
{
    export_stats(r->col, r->M, T, c1, g, k1, k2, clamped);
}

/* Sums S^L (columns, before the last column scaling) and R^L (rows). */
void orc_last_sums(const orc_result *r, double *colsum, double *rowsum)
{
    if (r->L == 0)
        return;
    if (colsum) memcpy(colsum, r->colsum + (size_t)(r->L - 1) * r->M, (size_t)r->M * sizeof(double));
    if (rowsum) memcpy(rowsum, r->rowsum + (size_t)(r->L - 1) * r->N, (size_t)r->N * sizeof(double));
}

void orc_grads(const orc_result *r, double *gx, double *gy)
{
    if (gx && r->gx) memcpy(gx, r->gx, (size_t)r->N * 3 * sizeof(double));
    if (gy && r->gy) memcpy(gy, r->gy, (size_t)r->M * 3 * sizeof(double));
}

/* ------------------------------------------------------------------------ */
/* sampled owners, for checks at sizes where a full run is too slow         */
/* ------------------------------------------------------------------------ */

/* Statistics and kept-entry count of the listed owners of one direction
 * (owners are points of P, scanned against all of Q). */
int orc_owner_stats(const double *P, int nP, const double *Q, int nQ, const orc_params *prm,
                    const int32_t *owners, int n_owners, int nthreads, double *T, double *c1,
                    double *g, int32_t *k1, int32_t *k2, uint8_t *clamped, int64_t *count)
{
    if (!P || !Q || !owners || !valid(nP, nQ, prm))
        return ORC_BAD_ARG;
#ifdef _OPENMP
    if (nthreads <= 0)
        nthreads = omp_get_max_threads();
#endif
    int bad = 0;
#pragma omp parallel for num_threads(nthreads) schedule(dynamic, 1) reduction(| : bad)
    for (int o = 0; o < n_owners; ++o) {
        const int a = owners[o];
        if (a < 0 || a >= nP) {
            bad = 1;
            continue;
        }
        owner_stats st;
        owner_statistics(P + 3 * (size_t)a, Q, nQ, prm, &st);
        int64_t n = 0;
        for (int b = 0; b < nQ; ++b)
            if (similarity(&st, cost(P + 3 * (size_t)a, Q + 3 * (size_t)b)) >= prm->tau)
                ++n;
        if (T) T[o] = st.T;
        if (c1) c1[o] = st.c1;
        if (g) g[o] = st.g;
        if (k1) k1[o] = st.k1;
        if (k2) k2[o] = st.k2;
        if (clamped) clamped[o] = st.clamped;
        if (count) count[o] = n;
    }
    return bad ? ORC_BAD_ARG : ORC_OK;
}

/* Kept support of one owner: the indices b with s >= tau, their similarity
 * s and their normalised probability, in increasing b. Returns the count,
 * writing at most cap entries. */
int64_t orc_owner_support(const double *P, int nP, const double *Q, int nQ, const orc_params *prm,
                          int owner, int64_t cap, int32_t *idx, double *s_out, double *p_out)
{
    if (!P || !Q || owner < 0 || owner >= nP || !valid(nP, nQ, prm))
        return -1;
    owner_stats st;
    const double *p = P + 3 * (size_t)owner;
    owner_statistics(p, Q, nQ, prm, &st);
    int64_t n = 0;
    double z = 0.0;
    for (int b = 0; b < nQ; ++b) {
        const double s = similarity(&st, cost(p, Q + 3 * (size_t)b));
        if (s >= prm->tau) {
            if (n < cap) {
                if (idx) idx[n] = b;
                if (s_out) s_out[n] = s;
            }
            z += s;
            ++n;
        }
    }
    if (p_out && s_out)
        for (int64_t t = 0; t < n && t < cap; ++t)
            p_out[t] = s_out[t] / z;
    return n;
}
