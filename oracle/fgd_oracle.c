/*
 * fgd_oracle.c -- plain CPU oracle for the Factored Gossip DiLoCo outer step.
 *
 * TEST INFRASTRUCTURE.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg load this library.  It is deliberately slow:
 * single-threaded, scalar, double precision, whole-vector stages in the order
 * the paper gives them, no blocking, no fusion.  It shares no code, header,
 * table or helper with the HIP engine.
 *
 * What it computes (per outer round, for workers m = 0..M-1 over parameters
 * p = 0..P-1; arrays are worker-major [M][ld]):
 *
 *   1. Outer gradient (Sec. 3 DiLoCo equations; Sec. 4.1 factored DiLoCo;
 *      Appendix A, Algorithm 1).  The paper's Delta = y_H - y_0 is handed to
 *      the outer optimizer negated; with theta_prev = y_0 and theta_local =
 *      y_H the gradient given to Nesterov is g0_m = theta_prev_m - theta_local_m.
 *   2. Mix2 of the outer gradient, K2 rounds (Sec. 3 gossip mixing operator:
 *      row m takes sum_n w_{m,n} v_n; Sec. 4.1 factored formulation).
 *   3. Mix1 of the previous outer parameters, K1 rounds, or the exact global
 *      mean (same operator; global averaging is W = 11^T / M).
 *   4. Nesterov outer update in the two-line implementation form of
 *      Appendix B: v' = mu v + g;  theta' = x - lr (g + mu v').  With
 *      Nesterov off, the plain momentum form of the same optimizer:
 *      v' = mu v + g;  theta' = x - lr v'.
 *      Variants (Appendix B, GlobalM1S; Sec. 4.1 and Appendix C, the
 *      Mix2-subset configuration):
 *        - mix1_state: Mix1 is also applied to the momentum v (the outer
 *          optimizer state) before the momentum update.
 *        - Mix2 subset: Mix2 acts only on the parameter indices inside a
 *          list of half-open segments [begin, end); elsewhere it is the
 *          identity, in every round.
 *      Split execution (Appendix A, Algorithm 1: the non-blocking Mix1 is
 *      launched at the start of the round and overlaps the inner loop; the
 *      blocking Mix2 and the outer optimizer run at its end):
 *        - fgdo_mix1_split stores x = Mix1(theta_prev) in the parameter
 *          storage type (and, with the state mixed, v <- Mix1(v));
 *        - fgdo_outer_blocking computes g0, Mix2 and the optimizer from
 *          that stored x, and can write theta' back into theta_local as the
 *          next round's inner starting point.
 *   5. Consensus distance S_m(u) = sum_p (u_m - mean_n u_n)^2 for every
 *      intermediate u (Sec. 4.4 L2 consensus distance; Appendix D.1 uses the
 *      mean of the squared norms, Sec. 4.4 the mean of the norms; both follow
 *      from S_m).
 *
 * Per-round effective weights (mixing under dropped links, which the paper
 * describes only qualitatively as weaker mixing under transient failures):
 *   NONE        the given weights; every mask entry must be 1.
 *   METROPOLIS  on the live graph of that round, d_i = number of live
 *               off-diagonal entries of row i, w_ij = 1 / (1 + max(d_i, d_j))
 *               in double, w_ii = 1 - sum of the row's live off-diagonal
 *               weights (ascending j, double), then every weight is rounded
 *               to float (nearest even).  Dropped entries get weight 0.
 *   SELF        the given weights, with each dropped entry's weight added to
 *               the diagonal of its row (ascending j, double) and rounded to
 *               float.
 * Dropped entries are skipped outright when mixing (a dropped neighbour
 * contributes nothing, even a non-finite value).
 *
 * Storage: theta_prev / theta_local are float32 (dtype 0) or bf16 bit
 * patterns (dtype 1); momentum is float32.  The new theta is rounded from
 * double directly to the storage type (nearest even); the new momentum is
 * rounded to float32.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum { FGDO_OK = 0, FGDO_BAD_ARG = -1, FGDO_NO_MEM = -2 };
enum { FGDO_IDENTITY = 0, FGDO_GLOBAL = 1, FGDO_CSR = 2 };
enum { FGDO_RW_NONE = 0, FGDO_RW_METROPOLIS = 1, FGDO_RW_SELF = 2 };

/* Outer-optimizer settings and step variants. */
typedef struct {
    float lr;              /* outer learning rate gamma */
    float mu;              /* momentum */
    int32_t nesterov;      /* 1: Nesterov form, 0: plain momentum */
    int32_t mix1_state;    /* 1: Mix1 also mixes the momentum before its update */
    int32_t n_seg;         /* Mix2 subset segments (0: Mix2 acts on every index) */
    const int64_t *seg;    /* [n_seg][2] half-open [begin, end), ascending, disjoint */
} fgdo_opts;

typedef struct {
    int32_t kind;           /* FGDO_IDENTITY, FGDO_GLOBAL or FGDO_CSR */
    int32_t rounds;         /* CSR: number of rounds K (0 = identity) */
    const int32_t *row_ptr; /* [M+1] */
    const int32_t *col_idx; /* [nnz], sorted per row, diagonal present */
    const float *weights;   /* [nnz]; may be NULL for METROPOLIS */
    const uint8_t *masks;   /* [rounds][nnz] or NULL (all live) */
    int32_t reweight;       /* FGDO_RW_* */
} fgdo_mix;

/* ---------------------------------------------------------------- bf16 */

/* Round a double to the nearest bf16 (ties to even), straight from double.
 * bf16 has 8 exponent bits and 7 stored mantissa bits, the float32 exponent
 * range and float32's subnormal floor 2^-126 scaled to 7 bits (2^-133). */
uint16_t fgdo_bf16_from_double(double d)
{
    if (isnan(d)) {
        return (uint16_t)(signbit(d) ? 0xFFC0u : 0x7FC0u);
    }
    double a = fabs(d);
    double r;
    /* Largest finite bf16 is (2 - 2^-7) * 2^127; halfway to 2^128 rounds to
     * the even neighbour, which is infinity. */
    if (a >= ldexp(2.0 - ldexp(1.0, -8), 127)) {
        r = INFINITY;
    } else if (a == 0.0) {
        r = 0.0;
    } else {
        int ex;
        frexp(a, &ex);               /* a in [2^(ex-1), 2^ex) */
        int qexp = ex - 1 - 7;       /* spacing of 8-bit significands there */
        if (qexp < -133) qexp = -133; /* subnormal spacing */
        double scaled = ldexp(a, -qexp);
        double n = nearbyint(scaled); /* default rounding mode: nearest even */
        r = ldexp(n, qexp);
    }
    float f = (float)r; /* exact: r is a bf16 value (or inf) */
    uint32_t u;
    memcpy(&u, &f, sizeof u);
    uint16_t h = (uint16_t)(u >> 16);
    if (signbit(d)) h |= 0x8000u;
    return h;
}

double fgdo_bf16_to_double(uint16_t h)
{
    uint32_t u = ((uint32_t)h) << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return (double)f;
}

static double load_param(const void *base, int32_t dtype, int64_t idx)
{
    if (dtype == 0) return (double)((const float *)base)[idx];
    return fgdo_bf16_to_double(((const uint16_t *)base)[idx]);
}

static void store_param(void *base, int32_t dtype, int64_t idx, double val)
{
    if (dtype == 0) ((float *)base)[idx] = (float)val;
    else ((uint16_t *)base)[idx] = fgdo_bf16_from_double(val);
}

/* ------------------------------------------------------------- weights */

static int row_of_diag(const int32_t *row_ptr, const int32_t *col_idx, int32_t i)
{
    for (int32_t e = row_ptr[i]; e < row_ptr[i + 1]; ++e)
        if (col_idx[e] == i) return e;
    return -1;
}

/* Effective weights of one round.  mask: [nnz] or NULL.  Returns FGDO_OK or
 * FGDO_BAD_ARG (missing diagonal, masked diagonal, masks under NONE, missing
 * weights where they are needed). */
int fgdo_round_weights(int32_t M, const int32_t *row_ptr, const int32_t *col_idx, const float *w_in,
                       const uint8_t *mask, int32_t reweight, float *w_out)
{
    if (M <= 0 || !row_ptr || !col_idx || !w_out) return FGDO_BAD_ARG;
    int32_t nnz = row_ptr[M];
    for (int32_t i = 0; i < M; ++i) {
        int e = row_of_diag(row_ptr, col_idx, i);
        if (e < 0) return FGDO_BAD_ARG;
        if (mask && !mask[e]) return FGDO_BAD_ARG;
    }
    if (reweight == FGDO_RW_NONE) {
        if (!w_in) return FGDO_BAD_ARG;
        if (mask)
            for (int32_t e = 0; e < nnz; ++e)
                if (!mask[e]) return FGDO_BAD_ARG;
        for (int32_t e = 0; e < nnz; ++e) w_out[e] = w_in[e];
        return FGDO_OK;
    }
    if (reweight == FGDO_RW_METROPOLIS) {
        int32_t *deg = (int32_t *)calloc((size_t)M, sizeof(int32_t));
        if (!deg) return FGDO_NO_MEM;
        for (int32_t i = 0; i < M; ++i)
            for (int32_t e = row_ptr[i]; e < row_ptr[i + 1]; ++e)
                if (col_idx[e] != i && (!mask || mask[e])) deg[i] += 1;
        for (int32_t i = 0; i < M; ++i) {
            double off = 0.0;
            int32_t diag = -1;
            for (int32_t e = row_ptr[i]; e < row_ptr[i + 1]; ++e) {
                int32_t j = col_idx[e];
                if (j == i) {
                    diag = e;
                    continue;
                }
                if (mask && !mask[e]) {
                    w_out[e] = 0.0f;
                    continue;
                }
                int32_t dmax = deg[i] > deg[j] ? deg[i] : deg[j];
                double w = 1.0 / (1.0 + (double)dmax);
                off += w;
                w_out[e] = (float)w;
            }
            w_out[diag] = (float)(1.0 - off);
        }
        free(deg);
        return FGDO_OK;
    }
    if (reweight == FGDO_RW_SELF) {
        if (!w_in) return FGDO_BAD_ARG;
        for (int32_t i = 0; i < M; ++i) {
            int32_t diag = row_of_diag(row_ptr, col_idx, i);
            double self = (double)w_in[diag];
            for (int32_t e = row_ptr[i]; e < row_ptr[i + 1]; ++e) {
                if (e == diag) continue;
                if (mask && !mask[e]) {
                    self += (double)w_in[e];
                    w_out[e] = 0.0f;
                } else {
                    w_out[e] = w_in[e];
                }
            }
            w_out[diag] = (float)self;
        }
        return FGDO_OK;
    }
    return FGDO_BAD_ARG;
}

/* ---------------------------------------------------------------- mixing */

/* dst_m = sum over live entries e of row m of w[e] * src_{col[e]}, entries in
 * ascending column order, for every parameter p.  src, dst: [M][P] double. */
static void mix_csr_round(int32_t M, int64_t P, const int32_t *row_ptr, const int32_t *col_idx,
                          const float *w, const uint8_t *mask, const double *src, double *dst)
{
    for (int32_t m = 0; m < M; ++m) {
        for (int64_t p = 0; p < P; ++p) {
            double acc = 0.0;
            for (int32_t e = row_ptr[m]; e < row_ptr[m + 1]; ++e) {
                if (mask && !mask[e]) continue;
                acc += (double)w[e] * src[(int64_t)col_idx[e] * P + p];
            }
            dst[(int64_t)m * P + p] = acc;
        }
    }
}

/* dst_m = (1/M) sum_n src_n for every m (global averaging). */
static void mix_global(int32_t M, int64_t P, const double *src, double *dst)
{
    for (int64_t p = 0; p < P; ++p) {
        double s = 0.0;
        for (int32_t n = 0; n < M; ++n) s += src[(int64_t)n * P + p];
        double mean = s / (double)M;
        for (int32_t m = 0; m < M; ++m) dst[(int64_t)m * P + p] = mean;
    }
}

/* S_m(u) = sum_p (u_m,p - mean_n u_n,p)^2, written to S[0..M). */
static void consensus_sq(int32_t M, int64_t P, const double *u, double *S)
{
    for (int32_t m = 0; m < M; ++m) S[m] = 0.0;
    for (int64_t p = 0; p < P; ++p) {
        double s = 0.0;
        for (int32_t n = 0; n < M; ++n) s += u[(int64_t)n * P + p];
        double mean = s / (double)M;
        for (int32_t m = 0; m < M; ++m) {
            double d = u[(int64_t)m * P + p] - mean;
            S[m] += d * d;
        }
    }
}

static int effective_rounds(const fgdo_mix *mx)
{
    if (mx->kind == FGDO_IDENTITY) return 0;
    if (mx->kind == FGDO_GLOBAL) return 1;
    return mx->rounds;
}

static int check_mix(int32_t M, const fgdo_mix *mx)
{
    if (!mx) return FGDO_BAD_ARG;
    if (mx->kind == FGDO_IDENTITY || mx->kind == FGDO_GLOBAL) return FGDO_OK;
    if (mx->kind != FGDO_CSR || mx->rounds < 0) return FGDO_BAD_ARG;
    if (mx->rounds > 0 && (!mx->row_ptr || !mx->col_idx)) return FGDO_BAD_ARG;
    (void)M;
    return FGDO_OK;
}

/* Applies all rounds of one Mix to src (double [M][P]) into dst.  cd, when
 * not NULL, receives S_m of the input and of every round's output:
 * [(rounds_eff + 1) * M].  Returns FGDO_OK or an error. */
/* Puts back the input value at every index outside the subset: there the
 * Mix is the identity, in every round. */
static void restore_outside(int32_t M, int64_t P, const uint8_t *inset, const double *src, double *dst)
{
    if (!inset) return;
    for (int32_t m = 0; m < M; ++m)
        for (int64_t p = 0; p < P; ++p)
            if (!inset[p]) dst[(int64_t)m * P + p] = src[(int64_t)m * P + p];
}

/* One Mix slot on src [M][P] into dst, with consensus rows cd[(K+1)][M]
 * (input, then every round's output; NULL: none).  inset[P] (NULL: every
 * index) marks the indices the Mix acts on. */
int fgdo_mix_apply_subset(int32_t M, int64_t P, const fgdo_mix *mx, const uint8_t *inset, const double *src,
                          double *dst, double *cd)
{
    if (M <= 0 || P < 0 || !src || !dst) return FGDO_BAD_ARG;
    int rc = check_mix(M, mx);
    if (rc) return rc;
    int64_t n = (int64_t)M * P;
    memcpy(dst, src, (size_t)n * sizeof(double));
    if (cd) consensus_sq(M, P, dst, cd);
    int K = effective_rounds(mx);
    if (K == 0) return FGDO_OK;
    double *tmp = (double *)malloc((size_t)(n > 0 ? n : 1) * sizeof(double));
    if (!tmp) return FGDO_NO_MEM;
    if (mx->kind == FGDO_GLOBAL) {
        mix_global(M, P, dst, tmp);
        restore_outside(M, P, inset, src, tmp);
        memcpy(dst, tmp, (size_t)n * sizeof(double));
        if (cd) consensus_sq(M, P, dst, cd + M);
        free(tmp);
        return FGDO_OK;
    }
    int32_t nnz = mx->row_ptr[M];
    float *w = (float *)malloc((size_t)(nnz > 0 ? nnz : 1) * sizeof(float));
    if (!w) {
        free(tmp);
        return FGDO_NO_MEM;
    }
    for (int k = 0; k < K; ++k) {
        const uint8_t *mask = mx->masks ? mx->masks + (int64_t)k * nnz : NULL;
        rc = fgdo_round_weights(M, mx->row_ptr, mx->col_idx, mx->weights, mask, mx->reweight, w);
        if (rc) break;
        mix_csr_round(M, P, mx->row_ptr, mx->col_idx, w, mask, dst, tmp);
        restore_outside(M, P, inset, src, tmp);
        memcpy(dst, tmp, (size_t)n * sizeof(double));
        if (cd) consensus_sq(M, P, dst, cd + (int64_t)(k + 1) * M);
    }
    free(w);
    free(tmp);
    return rc;
}

int fgdo_mix_apply(int32_t M, int64_t P, const fgdo_mix *mx, const double *src, double *dst, double *cd)
{
    return fgdo_mix_apply_subset(M, P, mx, NULL, src, dst, cd);
}

int fgdo_num_cd(const fgdo_mix *mix1, const fgdo_mix *mix2)
{
    return effective_rounds(mix2) + 1 + effective_rounds(mix1) + 1 + 1;
}

/* ------------------------------------------------------------ outer step */

/* One outer step, in place on theta_prev and mom.
 *   theta_prev  [M][ld] storage dtype, in/out
 *   theta_local [M][ld] storage dtype
 *   mom         [M][ld] float32, in/out
 *   cd          [fgdo_num_cd * M] double or NULL
 */
/* Index flags of a Mix2 subset: 1 inside some segment.  Segments must be
 * ascending, disjoint, non-empty and inside [0, P). */
static int subset_flags(int64_t P, int32_t n_seg, const int64_t *seg, uint8_t *inset)
{
    if (n_seg < 0 || (n_seg > 0 && !seg)) return FGDO_BAD_ARG;
    memset(inset, 0, (size_t)(P > 0 ? P : 1));
    int64_t prev_end = 0;
    for (int32_t i = 0; i < n_seg; ++i) {
        int64_t b = seg[2 * i], e = seg[2 * i + 1];
        if (b < prev_end || e <= b || e > P) return FGDO_BAD_ARG;
        for (int64_t p = b; p < e; ++p) inset[p] = 1;
        prev_end = e;
    }
    return FGDO_OK;
}

int fgdo_outer_step(int32_t M, int64_t P, int64_t ld, int32_t dtype, void *theta_prev,
                    const void *theta_local, float *mom, const fgdo_mix *mix1, const fgdo_mix *mix2,
                    const fgdo_opts *opt, double *cd)
{
    if (M <= 0 || P < 0 || ld < P || (dtype != 0 && dtype != 1)) return FGDO_BAD_ARG;
    if (!theta_prev || !theta_local || !mom || !opt) return FGDO_BAD_ARG;
    if (check_mix(M, mix1) || check_mix(M, mix2)) return FGDO_BAD_ARG;
    int64_t n = (int64_t)M * P;
    size_t bytes = (size_t)(n > 0 ? n : 1) * sizeof(double);
    double *g0 = (double *)malloc(bytes);
    double *ghat = (double *)malloc(bytes);
    double *x0 = (double *)malloc(bytes);
    double *x = (double *)malloc(bytes);
    double *v0 = (double *)malloc(bytes);
    double *v = (double *)malloc(bytes);
    double *theta_new = (double *)malloc(bytes);
    uint8_t *inset = opt->n_seg > 0 ? (uint8_t *)malloc((size_t)(P > 0 ? P : 1)) : NULL;
    int K2 = effective_rounds(mix2), K1 = effective_rounds(mix1);
    double *cd2 = (double *)malloc((size_t)(K2 + 1) * M * sizeof(double));
    double *cd1 = (double *)malloc((size_t)(K1 + 1) * M * sizeof(double));
    int rc = FGDO_OK;
    if (!g0 || !ghat || !x0 || !x || !v0 || !v || !theta_new || !cd2 || !cd1 || (opt->n_seg > 0 && !inset)) {
        rc = FGDO_NO_MEM;
        goto done;
    }
    if (inset) {
        rc = subset_flags(P, opt->n_seg, opt->seg, inset);
        if (rc) goto done;
    }

    /* 1. Outer gradient g0 = theta_prev - theta_local (negated paper Delta). */
    for (int32_t m = 0; m < M; ++m)
        for (int64_t p = 0; p < P; ++p) {
            double tp = load_param(theta_prev, dtype, (int64_t)m * ld + p);
            double tl = load_param(theta_local, dtype, (int64_t)m * ld + p);
            x0[(int64_t)m * P + p] = tp;
            g0[(int64_t)m * P + p] = tp - tl;
            v0[(int64_t)m * P + p] = (double)mom[(int64_t)m * ld + p];
        }

    /* 2. Mix2 on the outer gradient (blocking mix), on the subset if any. */
    rc = fgdo_mix_apply_subset(M, P, mix2, inset, g0, ghat, cd2);
    if (rc) goto done;

    /* 3. Mix1 on the previous outer parameters (non-blocking mix), and on
     *    the momentum too when the optimizer state is mixed. */
    rc = fgdo_mix_apply(M, P, mix1, x0, x, cd1);
    if (rc) goto done;
    if (opt->mix1_state) rc = fgdo_mix_apply(M, P, mix1, v0, v, NULL);
    else memcpy(v, v0, bytes);
    if (rc) goto done;

    /* 4. Outer optimizer.  Nesterov, two-line form: v' = mu v + g ;
     *    theta' = x - lr (g + mu v').  Plain momentum: theta' = x - lr v'. */
    {
        double dmu = (double)opt->mu, dlr = (double)opt->lr;
        for (int32_t m = 0; m < M; ++m)
            for (int64_t p = 0; p < P; ++p) {
                int64_t i = (int64_t)m * P + p, j = (int64_t)m * ld + p;
                double g = ghat[i];
                double v_new = dmu * v[i] + g;
                double t_new = opt->nesterov ? x[i] - dlr * (g + dmu * v_new) : x[i] - dlr * v_new;
                mom[j] = (float)v_new;
                store_param(theta_prev, dtype, j, t_new);
                theta_new[i] = load_param(theta_prev, dtype, j); /* as stored */
            }
    }

    /* 5. Consensus distances: g^0..g^K2, x^0..x^K1, stored theta'. */
    if (cd) {
        memcpy(cd, cd2, (size_t)(K2 + 1) * M * sizeof(double));
        memcpy(cd + (int64_t)(K2 + 1) * M, cd1, (size_t)(K1 + 1) * M * sizeof(double));
        consensus_sq(M, P, theta_new, cd + (int64_t)(K2 + K1 + 2) * M);
    }

done:
    free(g0);
    free(ghat);
    free(x0);
    free(x);
    free(v0);
    free(v);
    free(theta_new);
    free(inset);
    free(cd2);
    free(cd1);
    return rc;
}

/* Split execution, first half: x = Mix1(theta_prev) rounded to the
 * parameter storage type into x_out [M][ld]; with mix1_state, the momentum
 * [M][ld] is replaced by Mix1 of itself (rounded to float).  cd: [(K1+1)][M]
 * consensus rows x^0..x^K1 of the unrounded values, or NULL. */
int fgdo_mix1_split(int32_t M, int64_t P, int64_t ld, int32_t dtype, const void *theta_prev, void *x_out,
                    float *mom, const fgdo_mix *mix1, int32_t mix1_state, double *cd)
{
    if (M <= 0 || P < 0 || ld < P || (dtype != 0 && dtype != 1)) return FGDO_BAD_ARG;
    if (!theta_prev || !x_out || (mix1_state && !mom)) return FGDO_BAD_ARG;
    if (check_mix(M, mix1)) return FGDO_BAD_ARG;
    int64_t n = (int64_t)M * P;
    size_t bytes = (size_t)(n > 0 ? n : 1) * sizeof(double);
    double *z = (double *)malloc(bytes), *x = (double *)malloc(bytes);
    int rc = FGDO_OK;
    if (!z || !x) {
        rc = FGDO_NO_MEM;
        goto done;
    }
    for (int32_t m = 0; m < M; ++m)
        for (int64_t p = 0; p < P; ++p) z[(int64_t)m * P + p] = load_param(theta_prev, dtype, (int64_t)m * ld + p);
    rc = fgdo_mix_apply(M, P, mix1, z, x, cd);
    if (rc) goto done;
    for (int32_t m = 0; m < M; ++m)
        for (int64_t p = 0; p < P; ++p) store_param(x_out, dtype, (int64_t)m * ld + p, x[(int64_t)m * P + p]);
    if (mix1_state) {
        for (int32_t m = 0; m < M; ++m)
            for (int64_t p = 0; p < P; ++p) z[(int64_t)m * P + p] = (double)mom[(int64_t)m * ld + p];
        rc = fgdo_mix_apply(M, P, mix1, z, x, NULL);
        if (rc) goto done;
        for (int32_t m = 0; m < M; ++m)
            for (int64_t p = 0; p < P; ++p) mom[(int64_t)m * ld + p] = (float)x[(int64_t)m * P + p];
    }
done:
    free(z);
    free(x);
    return rc;
}

/* Split execution, second half (blocking): from the stored x [M][ld],
 * g0 = theta_prev - theta_local, ghat = Mix2(g0) (on the subset if any), the
 * optimizer update into theta_prev and mom; with write_local, theta_local
 * receives theta' as stored.  cd: [(K2+2)][M] rows g^0..g^K2 and the stored
 * theta', or NULL.  opt->mix1_state is ignored (the state is mixed by the
 * first half). */
int fgdo_outer_blocking(int32_t M, int64_t P, int64_t ld, int32_t dtype, const void *x_in, void *theta_prev,
                        void *theta_local, float *mom, const fgdo_mix *mix2, const fgdo_opts *opt,
                        int32_t write_local, double *cd)
{
    if (M <= 0 || P < 0 || ld < P || (dtype != 0 && dtype != 1)) return FGDO_BAD_ARG;
    if (!x_in || !theta_prev || !theta_local || !mom || !opt) return FGDO_BAD_ARG;
    if (check_mix(M, mix2)) return FGDO_BAD_ARG;
    int64_t n = (int64_t)M * P;
    size_t bytes = (size_t)(n > 0 ? n : 1) * sizeof(double);
    double *g0 = (double *)malloc(bytes), *ghat = (double *)malloc(bytes), *theta_new = (double *)malloc(bytes);
    uint8_t *inset = opt->n_seg > 0 ? (uint8_t *)malloc((size_t)(P > 0 ? P : 1)) : NULL;
    int K2 = effective_rounds(mix2);
    int rc = FGDO_OK;
    if (!g0 || !ghat || !theta_new || (opt->n_seg > 0 && !inset)) {
        rc = FGDO_NO_MEM;
        goto done;
    }
    if (inset) {
        rc = subset_flags(P, opt->n_seg, opt->seg, inset);
        if (rc) goto done;
    }
    for (int32_t m = 0; m < M; ++m)
        for (int64_t p = 0; p < P; ++p)
            g0[(int64_t)m * P + p] = load_param(theta_prev, dtype, (int64_t)m * ld + p) -
                                     load_param(theta_local, dtype, (int64_t)m * ld + p);
    rc = fgdo_mix_apply_subset(M, P, mix2, inset, g0, ghat, cd);
    if (rc) goto done;
    {
        double dmu = (double)opt->mu, dlr = (double)opt->lr;
        for (int32_t m = 0; m < M; ++m)
            for (int64_t p = 0; p < P; ++p) {
                int64_t i = (int64_t)m * P + p, j = (int64_t)m * ld + p;
                double g = ghat[i], x = load_param(x_in, dtype, j);
                double v_new = dmu * (double)mom[j] + g;
                double t_new = opt->nesterov ? x - dlr * (g + dmu * v_new) : x - dlr * v_new;
                mom[j] = (float)v_new;
                store_param(theta_prev, dtype, j, t_new);
                theta_new[i] = load_param(theta_prev, dtype, j);
                if (write_local) store_param(theta_local, dtype, j, t_new);
            }
    }
    if (cd) consensus_sq(M, P, theta_new, cd + (int64_t)(K2 + 1) * M);
done:
    free(g0);
    free(ghat);
    free(theta_new);
    free(inset);
    return rc;
}

/* S_m of a stored [M][ld] array (float32 or bf16 bit patterns). */
int fgdo_consensus(int32_t M, int64_t P, int64_t ld, int32_t dtype, const void *x, double *S)
{
    if (M <= 0 || P < 0 || ld < P || !x || !S || (dtype != 0 && dtype != 1)) return FGDO_BAD_ARG;
    int64_t n = (int64_t)M * P;
    double *u = (double *)malloc((size_t)(n > 0 ? n : 1) * sizeof(double));
    if (!u) return FGDO_NO_MEM;
    for (int32_t m = 0; m < M; ++m)
        for (int64_t p = 0; p < P; ++p) u[(int64_t)m * P + p] = load_param(x, dtype, (int64_t)m * ld + p);
    consensus_sq(M, P, u, S);
    free(u);
    return FGDO_OK;
}
