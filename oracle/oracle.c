/*
 * Brute-force CPU oracle for point sampling of a field of weighted 3D
 * Gaussians (W-VEG), and for its backward pass.
 *
 * TEST INFRASTRUCTURE ONLY. Nothing in the product library links, loads or
 * calls this file; only the tests, the smoke check and the benchmark's CPU
 * baseline do. It shares no code, header or constant table with the GPU
 * path.
 *
 * What it computes (paper Sec. 3.2, Eq. 2 and Eq. 3; Sec. 4.1.1; Sec. 4.1.3;
 * Sec. 5):
 *   G_i(p) = exp(-1/2 Q_i(p)),  Q_i(p) = || S_i^-1 R_i^T (p - mu_i) ||^2
 *   with R_i the rotation of the normalised quaternion (w,x,y,z) and S_i the
 *   diagonal of per-axis standard deviations, so that the inverse covariance
 *   is R S^-2 R^T (Eq. 3 with the paper's R_i read as R(q)^T).
 *   Gaussian i intersects p when its influence G_i(p) is at least the cutoff
 *   tau (Sec. 4.1.1), i.e. Q_i(p) <= T = 2 ln(1/tau).
 *   I(p) = sum_i w_i G_i(p),  V(p) = sum_i w_i v_i G_i(p)  over intersecting i
 *   p is defined when it lies in the closed domain box (Sec. 5, structured
 *   volumes cull samples outside their bounds) and I(p) > tau (Sec. 4.1.3);
 *   then the output is (Phi, I) = (V/I, I), otherwise (0, 0).
 * Every point is tested against every Gaussian; arithmetic is float64 (the
 * parameters and points are passed as float64, normally the exact values of
 * the float32 inputs; finite-difference tests perturb them in float64). The only shortcut is an exact cull: by Cauchy-Schwarz,
 * d_j^2 <= Sigma_jj * Q for every axis j, so a pair with
 * d_j^2 > Sigma_jj * T' has Q > T' and cannot intersect (nor lie in the
 * ambiguity band when T' includes the band). It can be switched off
 * (prune = 0) and the tests check both settings agree.
 *
 * The cell index (Sec. 4.1.1 and Sec. 4.1.2: per-Gaussian AABB of the cutoff
 * ellipsoid on a grid of cells, Gaussian-cell pairs ordered by cell): the
 * boxes in float32, in one fixed order of operations with every operation
 * rounded separately, so the GPU's boxes can be compared bit for bit, and
 * their full cell lists; and, by an exact float64 minimisation of Q over
 * each cell, the cells every Gaussian reaches. A GPU index may list fewer
 * cells than the box (the lists only have to hold the Gaussians that can
 * reach a cell), never fewer than the reached ones.
 *
 * Build: gcc -O2 -fopenmp -ffp-contract=off -shared -fPIC (see build.py).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORC_OK 0
#define ORC_ERR_ARG 1
#define ORC_ERR_CAPACITY 2
#define ORC_ERR_NOMEM 3

/* ambiguous pairs of a point whose a and v are kept one by one */
#define AMB_KEEP 8

/* unit roundoff of float32 */
#define EPS32 (1.0 / 16777216.0)

static void set_threads(int nthreads)
{
#ifdef _OPENMP
    if (nthreads > 0) omp_set_num_threads(nthreads);
#else
    (void)nthreads;
#endif
}

/* ------------------------------------------------------------------------ */
/* Per-Gaussian quantities in float64.                                       */
/* ------------------------------------------------------------------------ */

typedef struct {
    int valid;
    double mu[3];
    double s[3];
    double R[3][3];   /* R(qhat), Hamilton convention, (w,x,y,z) */
    double qhat[4];
    double qnorm;
    double v, w;
    double sig_diag[3]; /* Sigma_jj = sum_k R_jk^2 s_k^2 */
    double kappa;       /* s_max / s_min */
    double e_rel;       /* float32 relative error allowance of G */
    double band;        /* relative half-width of the ambiguity band in Q */
    double C[3][3];     /* upper Cholesky factor of R S^-2 R^T: C^T C = M^T M, M = S^-1 R^T */
} g64;

/* float32 squared norm of the quaternion in the canonical order; a
 * Gaussian whose canonical norm is zero, not finite, or whose other
 * parameters are not finite or whose scales are not positive is invalid
 * and contributes nothing. */
static int gauss_valid_f(const float *mu, const float *s, const float *q, float v, float w)
{
    for (int j = 0; j < 3; j++) {
        if (!isfinite(mu[j]) || !isfinite(s[j]) || !(s[j] > 0.0f)) return 0;
    }
    for (int j = 0; j < 4; j++)
        if (!isfinite(q[j])) return 0;
    if (!isfinite(v) || !isfinite(w)) return 0;
    volatile float a = q[0] * q[0];
    volatile float b = q[1] * q[1];
    volatile float c = q[2] * q[2];
    volatile float d = q[3] * q[3];
    volatile float ab = a + b;
    volatile float abc = ab + c;
    volatile float n2 = abc + d;
    if (!(n2 > 0.0f) || !isfinite(n2)) return 0;
    return 1;
}

/* the same predicate for float64 parameters, judged on their float32
 * roundings (exact when the parameters are float32 values) */
static int gauss_valid_d(const double *mu, const double *s, const double *q, double v, double w)
{
    float muf[3], sf[3], qf[4];
    for (int j = 0; j < 3; j++) {
        if (!isfinite(mu[j]) || !isfinite(s[j]) || !(s[j] > 0.0)) return 0;
        muf[j] = (float)mu[j];
        sf[j] = (float)s[j];
    }
    for (int j = 0; j < 4; j++) {
        if (!isfinite(q[j])) return 0;
        qf[j] = (float)q[j];
    }
    return gauss_valid_f(muf, sf, qf, (float)v, (float)w);
}

/* Rotation matrix of a unit quaternion (w,x,y,z), Hamilton product
 * convention: it maps the Gaussian's local axes to world axes. */
static void quat_to_rot(const double q[4], double R[3][3])
{
    double w = q[0], x = q[1], y = q[2], z = q[3];
    R[0][0] = 1.0 - 2.0 * (y * y + z * z);
    R[0][1] = 2.0 * (x * y - w * z);
    R[0][2] = 2.0 * (x * z + w * y);
    R[1][0] = 2.0 * (x * y + w * z);
    R[1][1] = 1.0 - 2.0 * (x * x + z * z);
    R[1][2] = 2.0 * (y * z - w * x);
    R[2][0] = 2.0 * (x * z - w * y);
    R[2][1] = 2.0 * (y * z + w * x);
    R[2][2] = 1.0 - 2.0 * (x * x + y * y);
}

static void prepare(int64_t i, const double *mean, const double *scale, const double *rot,
                    const double *value, const double *weight, double T, g64 *g)
{
    const double *mu = mean + 3 * i, *s = scale + 3 * i, *q = rot + 4 * i;
    memset(g, 0, sizeof(*g));
    g->valid = gauss_valid_d(mu, s, q, value[i], weight[i]);
    if (!g->valid) return;
    double qn = sqrt(q[0] * q[0] + q[1] * q[1] + q[2] * q[2] + q[3] * q[3]);
    g->qnorm = qn;
    for (int k = 0; k < 4; k++) g->qhat[k] = q[k] / qn;
    quat_to_rot(g->qhat, g->R);
    double smax = 0.0, smin = INFINITY;
    for (int k = 0; k < 3; k++) {
        g->mu[k] = mu[k];
        g->s[k] = s[k];
        if (g->s[k] > smax) smax = g->s[k];
        if (g->s[k] < smin) smin = g->s[k];
    }
    for (int j = 0; j < 3; j++) {
        double acc = 0.0;
        for (int k = 0; k < 3; k++) acc += g->R[j][k] * g->R[j][k] * g->s[k] * g->s[k];
        g->sig_diag[j] = acc;
    }
    /* Sigma^-1 = R S^-2 R^T and its upper triangular factor (Cholesky, row
     * by row): |C d|^2 = |S^-1 R^T d|^2 = Q for every d */
    double A[3][3];
    for (int j = 0; j < 3; j++)
        for (int l = 0; l < 3; l++) {
            double acc = 0.0;
            for (int k = 0; k < 3; k++) acc += g->R[j][k] * g->R[l][k] / (g->s[k] * g->s[k]);
            A[j][l] = acc;
        }
    for (int r = 0; r < 3; r++) {
        double dg = A[r][r];
        for (int m = 0; m < r; m++) dg -= g->C[m][r] * g->C[m][r];
        g->C[r][r] = sqrt(dg);
        for (int c = r + 1; c < 3; c++) {
            double off = A[r][c];
            for (int m = 0; m < r; m++) off -= g->C[m][r] * g->C[m][c];
            g->C[r][c] = off / g->C[r][r];
        }
    }
    g->v = value[i];
    g->w = weight[i];
    g->kappa = smax / smin;
    /* first-order float32 bound on the relative error of G: 9 eps T kappa
     * from the whitening (Q = |u|^2 with u = S^-1 R^T d), plus a few ulps
     * for exp and the products */
    g->e_rel = EPS32 * (9.0 * T * g->kappa + 8.0);
    g->band = ldexp(1.0, -18) * (g->kappa > 1.0 ? g->kappa : 1.0);
}

/* u = S^-1 R^T d and Q = |u|^2 */
static double whiten(const g64 *g, const double d[3], double u[3])
{
    double Q = 0.0;
    for (int k = 0; k < 3; k++) {
        double t = g->R[0][k] * d[0] + g->R[1][k] * d[1] + g->R[2][k] * d[2];
        u[k] = t / g->s[k];
        Q += u[k] * u[k];
    }
    return Q;
}

/* exact cull: 1 if some axis proves Q > Tlim */
static int culled(const g64 *g, const double d[3], double Tlim)
{
    for (int j = 0; j < 3; j++)
        if (d[j] * d[j] > g->sig_diag[j] * Tlim) return 1;
    return 0;
}

static int in_box_d(const double *p, const float lo[3], const float hi[3])
{
    for (int j = 0; j < 3; j++)
        if (!(p[j] >= (double)lo[j]) || !(p[j] <= (double)hi[j])) return 0;
    return 1;
}

static g64 *prepare_all(int64_t n, const double *mean, const double *scale, const double *rot,
                        const double *value, const double *weight, double T)
{
    g64 *gs = (g64 *)malloc(sizeof(g64) * (size_t)(n > 0 ? n : 1));
    if (!gs) return NULL;
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; i++) prepare(i, mean, scale, rot, value, weight, T, &gs[i]);
    return gs;
}

/* ------------------------------------------------------------------------ */
/* Forward (Eq. 2, Eq. 3, Sec. 4.1.3).                                       */
/* ------------------------------------------------------------------------ */

/*
 * For each point: phi, inf (the output pair, (0,0) when undefined), defined
 * flag, number of intersecting Gaussians, and the data the tests need to
 * accept the results that float32 may legitimately produce:
 *   namb          number of pairs with |Q - T| <= T * band_i
 *   i_base/v_base sums over intersecting pairs that are not ambiguous
 *   amb_a/amb_v   a = w G and v of the first AMB_KEEP ambiguous pairs
 *   amb_tot       per point: the sum of a over all its ambiguous pairs and
 *                 the least and largest v among them (0, 0, 0 when none)
 *   b_phi/b_inf   conditioning allowances sum a_i e_i |v_i - Phi| / I and
 *                 sum a_i e_i over intersecting pairs
 * Any output pointer may be NULL.
 */
int orc_forward(int64_t n, const double *mean, const double *scale, const double *rot,
                const double *value, const double *weight, const float lo[3], const float hi[3],
                float tau, int64_t npts, const double *pts, int prune, int nthreads,
                double *phi, double *inf, int32_t *defined, int32_t *ncontrib, int32_t *namb,
                double *i_base, double *v_base, double *amb_a, double *amb_v, double *amb_tot,
                double *b_phi, double *b_inf)
{
    if (n < 0 || npts < 0 || !(tau > 0.0f) || !(tau < 1.0f)) return ORC_ERR_ARG;
    set_threads(nthreads);
    const double T = 2.0 * log(1.0 / (double)tau);
    const double tauD = (double)tau;
    g64 *gs = prepare_all(n, mean, scale, rot, value, weight, T);
    if (!gs) return ORC_ERR_NOMEM;
    int err = 0;
#pragma omp parallel
    {
        size_t cap = 256, cnt = 0;
        double *ca = (double *)malloc(cap * sizeof(double));
        double *ce = (double *)malloc(cap * sizeof(double));
        double *cv = (double *)malloc(cap * sizeof(double));
        if (!ca || !ce || !cv) {
#pragma omp atomic write
            err = 1;
        }
#pragma omp for schedule(dynamic, 16)
        for (int64_t p = 0; p < npts; p++) {
            if (err) continue;
            const double *pp = pts + 3 * p;
            double I = 0.0, V = 0.0, Ib = 0.0, Vb = 0.0;
            int K = 0, A = 0;
            double aa[AMB_KEEP] = {0}, av[AMB_KEEP] = {0};
            double asum = 0.0, avlo = INFINITY, avhi = -INFINITY;
            cnt = 0;
            int inside = in_box_d(pp, lo, hi);
            if (inside) {
                for (int64_t i = 0; i < n; i++) {
                    const g64 *g = &gs[i];
                    if (!g->valid) continue;
                    double d[3] = {pp[0] - g->mu[0], pp[1] - g->mu[1], pp[2] - g->mu[2]};
                    double Tband = T * (1.0 + g->band);
                    if (prune && culled(g, d, Tband * (1.0 + 1e-9))) continue;
                    double u[3];
                    double Q = whiten(g, d, u);
                    int amb = fabs(Q - T) <= T * g->band;
                    if (amb) {
                        const double a = g->w * exp(-0.5 * Q);
                        if (A < AMB_KEEP) {
                            aa[A] = a;
                            av[A] = g->v;
                        }
                        asum += a;
                        avlo = g->v < avlo ? g->v : avlo;
                        avhi = g->v > avhi ? g->v : avhi;
                        A++;
                    }
                    if (Q <= T) {
                        double a = g->w * exp(-0.5 * Q);
                        I += a;
                        V += a * g->v;
                        K++;
                        if (!amb) {
                            Ib += a;
                            Vb += a * g->v;
                        }
                        if (cnt == cap) {
                            cap *= 2;
                            double *na = (double *)realloc(ca, cap * sizeof(double));
                            double *ne = (double *)realloc(ce, cap * sizeof(double));
                            double *nv = (double *)realloc(cv, cap * sizeof(double));
                            if (!na || !ne || !nv) {
#pragma omp atomic write
                                err = 1;
                                break;
                            }
                            ca = na;
                            ce = ne;
                            cv = nv;
                        }
                        ca[cnt] = a;
                        ce[cnt] = g->e_rel;
                        cv[cnt] = g->v;
                        cnt++;
                    }
                }
            }
            int def = inside && (I > tauD);
            double ph = def ? V / I : 0.0;
            double bi = 0.0, bp = 0.0;
            for (size_t c = 0; c < cnt; c++) {
                bi += ca[c] * ce[c];
                bp += ca[c] * ce[c] * fabs(cv[c] - ph);
            }
            if (phi) phi[p] = ph;
            if (inf) inf[p] = def ? I : 0.0;
            if (defined) defined[p] = def;
            if (ncontrib) ncontrib[p] = K;
            if (namb) namb[p] = A;
            if (i_base) i_base[p] = Ib;
            if (v_base) v_base[p] = Vb;
            if (amb_a)
                for (int k = 0; k < AMB_KEEP; k++) amb_a[AMB_KEEP * p + k] = aa[k];
            if (amb_v)
                for (int k = 0; k < AMB_KEEP; k++) amb_v[AMB_KEEP * p + k] = av[k];
            if (amb_tot) {
                amb_tot[3 * p] = asum;
                amb_tot[3 * p + 1] = A ? avlo : 0.0;
                amb_tot[3 * p + 2] = A ? avhi : 0.0;
            }
            if (b_inf) b_inf[p] = bi;
            if (b_phi) b_phi[p] = def ? bp / I : 0.0;
        }
        free(ca);
        free(ce);
        free(cv);
    }
    free(gs);
    return err ? ORC_ERR_NOMEM : ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Backward (Sec. 4.1.4: gradients of the loss flow from dL/dPhi and dL/dI   */
/* of every sample to the parameters mu, S, R, v, w of the Gaussians that     */
/* influenced it; Sec. 4.2: R comes from a normalised quaternion).           */
/* ------------------------------------------------------------------------ */

/*
 * Exact derivative of the smooth piece: the set of intersecting pairs and
 * the definedness of every point are held fixed (taken from the forward
 * outputs phi/inf passed in, which the caller computes with orc_forward).
 *
 * For a defined point p with cotangents (gPhi, gI), Phi = V/I gives
 *   dL/dV = gPhi / I,  dL/dI = gI - gPhi * Phi / I
 * and for an intersecting Gaussian with a = w G:
 *   dL/da = gPhi (v - Phi) / I + gI
 *   dL/dv = gPhi a / I,  dL/dw = dL/da * G,  dL/dQ = -1/2 a dL/da
 *   u = S^-1 R^T d, Q = |u|^2, d = p - mu:
 *   dL/dmu_j = -sum_k dL/dQ 2 u_k R_jk / s_k
 *   dL/ds_k  = -dL/dQ 2 u_k^2 / s_k
 *   dL/dR_jk =  dL/dQ 2 u_k d_j / s_k
 * then through R(qhat) to qhat, and through qhat = q/|q| to q:
 *   dL/dq = (dL/dqhat - qhat (qhat . dL/dqhat)) / |q|.
 * Output per selected Gaussian, 12 values: dmu[3], ds[3], dq[4], dv, dw;
 * abs_out holds the sum over pairs of the absolute per-pair terms, with
 * dL/da counted as the sum of the magnitudes of its parts (see below).
 * Points with zero_mask[p] != 0 contribute nothing (their cotangents are
 * taken as zero). sel == NULL selects every Gaussian. npairs (optional)
 * receives each selected Gaussian's number of intersecting pairs at the
 * defined points taken into account, and mom_abs (optional, [nsel][9])
 * the sums over those pairs of |dL/dQ| C_k and |dL/dQ| C_m C_k (m <= k:
 * 00 01 02 11 12 22), with C_k = sum_j |C_kj d_j| the size of the parts of
 * c_k = (C d)_k, C the upper Cholesky factor of Sigma^-1 (so |c|^2 = Q),
 * and |dL/dQ| taken at the size of dL/da's parts: the magnitudes of the
 * sums an implementation that whitens with the triangular factor
 * accumulates. term_abs (optional, [nsel][10]) receives the sums over the
 * pairs of the absolute values of the exact per-pair terms of dmu, ds, dq
 * for that same |dL/dQ|: what a relative error of G scales.
 */
int orc_backward(int64_t n, const double *mean, const double *scale, const double *rot,
                 const double *value, const double *weight, const float lo[3], const float hi[3],
                 float tau, int64_t npts, const double *pts, const double *phi, const double *inf,
                 const double *g_phi, const double *g_inf, const uint8_t *zero_mask,
                 int64_t nsel, const int64_t *sel, int prune, int nthreads,
                 double *grad, double *abs_out, int64_t *npairs, double *mom_abs, double *term_abs)
{
    if (n < 0 || npts < 0 || !(tau > 0.0f) || !(tau < 1.0f)) return ORC_ERR_ARG;
    if (!sel) nsel = n;
    set_threads(nthreads);
    const double T = 2.0 * log(1.0 / (double)tau);
    const double tauD = (double)tau;
#pragma omp parallel for schedule(dynamic, 4)
    for (int64_t t = 0; t < nsel; t++) {
        int64_t i = sel ? sel[t] : t;
        double acc[12], aab[12], mab[9], tab[10];
        int64_t K = 0;
        memset(tab, 0, sizeof(tab));
        memset(acc, 0, sizeof(acc));
        memset(aab, 0, sizeof(aab));
        memset(mab, 0, sizeof(mab));
        g64 g;
        if (i >= 0 && i < n) prepare(i, mean, scale, rot, value, weight, T, &g);
        else g.valid = 0;
        if (g.valid) {
            for (int64_t p = 0; p < npts; p++) {
                if (zero_mask && zero_mask[p]) continue;
                const double *pp = pts + 3 * p;
                if (!in_box_d(pp, lo, hi) || !(inf[p] > tauD)) continue;
                double d[3] = {pp[0] - g.mu[0], pp[1] - g.mu[1], pp[2] - g.mu[2]};
                if (prune && culled(&g, d, T * (1.0 + 1e-9))) continue;
                double u[3];
                double Q = whiten(&g, d, u);
                if (!(Q <= T)) continue;
                K++;
                double I = inf[p], Ph = phi[p];
                double gP = g_phi[p], gI = g_inf[p];
                double G = exp(-0.5 * Q);
                double a = g.w * G;
                double dLda = gP * (g.v - Ph) / I + gI;
                /* the size of dL/da as its two parts gPhi v / I and
                 * gI - gPhi Phi / I: what an evaluation in float32 rounds,
                 * for the tolerance sums (dL/da itself can cancel to ~0) */
                double dLdaMag = fabs(gP * g.v / I) + fabs(gP * Ph / I) + fabs(gI);
                double term[12];
                /* every term but dv is linear in dL/dQ: form them for a unit
                 * dL/dQ, then scale by the pair's value and by its size */
                double dLdQ = 1.0;
                for (int j = 0; j < 3; j++) {
                    double s_ = 0.0;
                    for (int k = 0; k < 3; k++) s_ += dLdQ * 2.0 * u[k] * g.R[j][k] / g.s[k];
                    term[j] = -s_;
                }
                for (int k = 0; k < 3; k++) term[3 + k] = -dLdQ * 2.0 * u[k] * u[k] / g.s[k];
                double dR[3][3];
                for (int j = 0; j < 3; j++)
                    for (int k = 0; k < 3; k++) dR[j][k] = dLdQ * 2.0 * u[k] * d[j] / g.s[k];
                double w = g.qhat[0], x = g.qhat[1], y = g.qhat[2], z = g.qhat[3];
                /* derivative of each R entry w.r.t. (w,x,y,z), summed against dR */
                double dqh[4];
                dqh[0] = 2.0 * (-z * dR[0][1] + y * dR[0][2] + z * dR[1][0] - x * dR[1][2] - y * dR[2][0] + x * dR[2][1]);
                dqh[1] = 2.0 * (y * dR[0][1] + z * dR[0][2] + y * dR[1][0] - 2.0 * x * dR[1][1] - w * dR[1][2] +
                                z * dR[2][0] + w * dR[2][1] - 2.0 * x * dR[2][2]);
                dqh[2] = 2.0 * (-2.0 * y * dR[0][0] + x * dR[0][1] + w * dR[0][2] + x * dR[1][0] + z * dR[1][2] -
                                w * dR[2][0] + z * dR[2][1] - 2.0 * y * dR[2][2]);
                dqh[3] = 2.0 * (-2.0 * z * dR[0][0] - w * dR[0][1] + x * dR[0][2] + w * dR[1][0] - 2.0 * z * dR[1][1] +
                                y * dR[1][2] + x * dR[2][0] + y * dR[2][1]);
                double dot = w * dqh[0] + x * dqh[1] + y * dqh[2] + z * dqh[3];
                for (int k = 0; k < 4; k++) term[6 + k] = (dqh[k] - g.qhat[k] * dot) / g.qnorm;
                /* the size of the quaternion terms before they cancel: each
                 * component is a signed sum of dL/dR entries (exactly zero
                 * for a spherical Gaussian), so float arithmetic rounds it at
                 * the size of those entries, not at its own */
                const double aw = fabs(w), ax = fabs(x), ay = fabs(y), az = fabs(z);
                /* u_k itself is a sum of three products R_jk d_j / s_k, which
                 * cancel for points near a principal plane: U_k is the size
                 * at which any evaluation rounds it */
                double U[3];
                for (int k = 0; k < 3; k++) {
                    U[k] = 0.0;
                    for (int j = 0; j < 3; j++) U[k] += fabs(g.R[j][k] * d[j]) / g.s[k];
                }
                double A_[3][3];
                for (int j = 0; j < 3; j++)
                    for (int k = 0; k < 3; k++) A_[j][k] = 2.0 * U[k] * fabs(d[j]) / g.s[k];
                double mq[4];
                mq[0] = 2.0 * (az * A_[0][1] + ay * A_[0][2] + az * A_[1][0] + ax * A_[1][2] + ay * A_[2][0] +
                               ax * A_[2][1]);
                mq[1] = 2.0 * (ay * A_[0][1] + az * A_[0][2] + ay * A_[1][0] + 2.0 * ax * A_[1][1] + aw * A_[1][2] +
                               az * A_[2][0] + aw * A_[2][1] + 2.0 * ax * A_[2][2]);
                mq[2] = 2.0 * (2.0 * ay * A_[0][0] + ax * A_[0][1] + aw * A_[0][2] + ax * A_[1][0] + az * A_[1][2] +
                               aw * A_[2][0] + az * A_[2][1] + 2.0 * ay * A_[2][2]);
                mq[3] = 2.0 * (2.0 * az * A_[0][0] + aw * A_[0][1] + ax * A_[0][2] + aw * A_[1][0] +
                               2.0 * az * A_[1][1] + ay * A_[1][2] + ax * A_[2][0] + ay * A_[2][1]);
                const double mdot = aw * mq[0] + ax * mq[1] + ay * mq[2] + az * mq[3];
                double mag[10];
                /* the mean terms -2 (M^T u)_j likewise: three products that
                 * cancel where d lies along a principal direction of the
                 * covariance (at the ellipsoid's axis-extreme points); the
                 * scale terms -2 u_k^2 / s_k at the size of u_k's parts */
                for (int j = 0; j < 3; j++) {
                    double m = 0.0;
                    for (int k = 0; k < 3; k++) m += 2.0 * U[k] * fabs(g.R[j][k]) / g.s[k];
                    mag[j] = m;
                }
                for (int k = 0; k < 3; k++) mag[3 + k] = 2.0 * U[k] * U[k] / g.s[k];
                for (int k = 0; k < 4; k++) mag[6 + k] = (mq[k] + fabs(g.qhat[k]) * mdot) / g.qnorm;
                const double dLdQv = -0.5 * a * dLda, dLdQm = 0.5 * a * dLdaMag;
                for (int k = 0; k < 10; k++) {
                    acc[k] += term[k] * dLdQv;
                    aab[k] += mag[k] * dLdQm;
                    tab[k] += fabs(term[k]) * dLdQm;
                }
                /* the sizes of the triangular-frame moments sum |dL/dQ| c
                 * and sum |dL/dQ| c c^T, c = C d, at the size of c's parts */
                double Cp[3];
                for (int a_ = 0; a_ < 3; a_++) {
                    Cp[a_] = 0.0;
                    for (int b_ = a_; b_ < 3; b_++) Cp[a_] += fabs(g.C[a_][b_] * d[b_]);
                }
                for (int k = 0; k < 3; k++) mab[k] += dLdQm * Cp[k];
                mab[3] += dLdQm * Cp[0] * Cp[0];
                mab[4] += dLdQm * Cp[0] * Cp[1];
                mab[5] += dLdQm * Cp[0] * Cp[2];
                mab[6] += dLdQm * Cp[1] * Cp[1];
                mab[7] += dLdQm * Cp[1] * Cp[2];
                mab[8] += dLdQm * Cp[2] * Cp[2];
                term[10] = gP * a / I;
                acc[10] += term[10];
                aab[10] += fabs(term[10]);
                acc[11] += dLda * G;
                aab[11] += dLdaMag * G;
            }
        }
        for (int k = 0; k < 12; k++) {
            grad[12 * t + k] = acc[k];
            if (abs_out) abs_out[12 * t + k] = aab[k];
        }
        if (npairs) npairs[t] = K;
        if (mom_abs)
            for (int k = 0; k < 9; k++) mom_abs[9 * t + k] = mab[k];
        if (term_abs)
            for (int k = 0; k < 10; k++) term_abs[10 * t + k] = tab[k];
    }
    return ORC_OK;
}

/*
 * touched[p] = 1 when some selected Gaussian has Q <= T (1 + band) at p and
 * p lies in the box: only those points can carry gradient to the selection.
 */
int orc_support(int64_t n, const double *mean, const double *scale, const double *rot,
                const double *value, const double *weight, const float lo[3], const float hi[3],
                float tau, int64_t npts, const double *pts, int64_t nsel, const int64_t *sel,
                int nthreads, uint8_t *touched)
{
    if (n < 0 || npts < 0 || nsel < 0 || !(tau > 0.0f) || !(tau < 1.0f)) return ORC_ERR_ARG;
    set_threads(nthreads);
    const double T = 2.0 * log(1.0 / (double)tau);
    g64 *gs = (g64 *)malloc(sizeof(g64) * (size_t)(nsel > 0 ? nsel : 1));
    if (!gs) return ORC_ERR_NOMEM;
    for (int64_t t = 0; t < nsel; t++) {
        if (sel[t] >= 0 && sel[t] < n) prepare(sel[t], mean, scale, rot, value, weight, T, &gs[t]);
        else gs[t].valid = 0;
    }
#pragma omp parallel for schedule(static)
    for (int64_t p = 0; p < npts; p++) {
        const double *pp = pts + 3 * p;
        uint8_t hit = 0;
        if (in_box_d(pp, lo, hi)) {
            for (int64_t t = 0; t < nsel && !hit; t++) {
                const g64 *g = &gs[t];
                if (!g->valid) continue;
                double d[3] = {pp[0] - g->mu[0], pp[1] - g->mu[1], pp[2] - g->mu[2]};
                double Tb = T * (1.0 + g->band);
                if (culled(g, d, Tb * (1.0 + 1e-9))) continue;
                double u[3];
                if (whiten(g, d, u) <= Tb) hit = 1;
            }
        }
        touched[p] = hit;
    }
    free(gs);
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Queries.                                                                  */
/* ------------------------------------------------------------------------ */

/* Canonical float32 voxel centre of voxel id (x fastest) of a dims grid
 * spanning [lo, hi]: c_j = lo_j + (i_j + 1/2) * ((hi_j - lo_j) / dims_j),
 * each operation rounded separately. */
int orc_voxel_centers(const int32_t dims[3], const float lo[3], const float hi[3], int64_t nids,
                      const uint32_t *ids, float *out)
{
    for (int j = 0; j < 3; j++)
        if (dims[j] <= 0) return ORC_ERR_ARG;
    float vs[3];
    for (int j = 0; j < 3; j++) {
        volatile float ext = hi[j] - lo[j];
        vs[j] = ext / (float)dims[j];
    }
    int64_t nx = dims[0], ny = dims[1];
    for (int64_t t = 0; t < nids; t++) {
        int64_t id = ids ? (int64_t)ids[t] : t;
        int64_t c[3] = {id % nx, (id / nx) % ny, id / (nx * ny)};
        for (int j = 0; j < 3; j++) {
            volatile float f = (float)c[j] + 0.5f;
            volatile float m = f * vs[j];
            out[3 * t + j] = lo[j] + m;
        }
    }
    return ORC_OK;
}

/* Training sample positions (the structured training of Sec. 4.2.2: a random
 * position in each voxel every iteration): voxel (i, j, k) of ids[t] (or t
 * when ids is NULL) with the caller's offsets u = u[3t .. 3t + 2] lies at
 * lo + (i + u) * ((hi - lo) / dims) per axis, in float32 with each operation
 * rounded (u = 1/2 gives the voxel centre above). */
int orc_jitter_positions(const int32_t dims[3], const float lo[3], const float hi[3], int64_t nids,
                         const uint32_t *ids, const float *u, float *out)
{
    for (int j = 0; j < 3; j++)
        if (dims[j] <= 0) return ORC_ERR_ARG;
    float vs[3];
    for (int j = 0; j < 3; j++) {
        volatile float ext = hi[j] - lo[j];
        vs[j] = ext / (float)dims[j];
    }
    int64_t nx = dims[0], ny = dims[1];
    for (int64_t t = 0; t < nids; t++) {
        int64_t id = ids ? (int64_t)ids[t] : t;
        int64_t c[3] = {id % nx, (id / nx) % ny, id / (nx * ny)};
        for (int j = 0; j < 3; j++) {
            volatile float f = (float)c[j] + u[3 * t + j];
            volatile float m = f * vs[j];
            out[3 * t + j] = lo[j] + m;
        }
    }
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* Cell index (Sec. 4.1.1, Sec. 4.1.2), canonical float32.                   */
/* ------------------------------------------------------------------------ */

/* Half-extent factor of the index boxes: the cutoff radius sqrt(2 ln(1/tau))
 * enlarged by 2^-10 so the box also holds every point whose float32 Q falls
 * at the cutoff; computed in float64 and rounded once to float32. */
static float index_radius(float tau)
{
    double rc = sqrt(2.0 * log(1.0 / (double)tau));
    return (float)(rc * (1.0 + 1.0 / 1024.0));
}

/* Cell box of one Gaussian; returns the number of cells (0 when the box
 * misses the grid or the Gaussian is invalid). Every float32 operation is
 * rounded separately, in this order. */
static int64_t cell_box(const float *mu, const float *s, const float *q, float v, float w,
                        const float lo[3], const float invc[3], const int32_t cells[3], float RCI,
                        int32_t box[6])
{
    for (int j = 0; j < 6; j++) box[j] = -1;
    if (!gauss_valid_f(mu, s, q, v, w)) return 0;
    volatile float t0 = q[0] * q[0], t1 = q[1] * q[1], t2 = q[2] * q[2], t3 = q[3] * q[3];
    volatile float n2a = t0 + t1;
    volatile float n2b = n2a + t2;
    volatile float n2 = n2b + t3;
    volatile float rt = sqrtf(n2);
    volatile float inv = 1.0f / rt;
    volatile float qw = q[0] * inv, qx = q[1] * inv, qy = q[2] * inv, qz = q[3] * inv;
    float R[3][3];
    {
        volatile float yy = qy * qy, zz = qz * qz, xx = qx * qx;
        volatile float xy = qx * qy, wz = qw * qz, xz = qx * qz, wy = qw * qy, yz = qy * qz, wx = qw * qx;
        volatile float s00 = yy + zz, s11 = xx + zz, s22 = xx + yy;
        volatile float d01 = xy - wz, d02 = xz + wy, d10 = xy + wz, d12 = yz - wx, d20 = xz - wy, d21 = yz + wx;
        volatile float m00 = 2.0f * s00, m11 = 2.0f * s11, m22 = 2.0f * s22;
        R[0][0] = 1.0f - m00;
        R[0][1] = 2.0f * d01;
        R[0][2] = 2.0f * d02;
        R[1][0] = 2.0f * d10;
        R[1][1] = 1.0f - m11;
        R[1][2] = 2.0f * d12;
        R[2][0] = 2.0f * d20;
        R[2][1] = 2.0f * d21;
        R[2][2] = 1.0f - m22;
    }
    int64_t count = 1;
    int32_t b[6];
    for (int j = 0; j < 3; j++) {
        volatile float a0 = R[j][0] * s[0], a1 = R[j][1] * s[1], a2 = R[j][2] * s[2];
        volatile float p0 = a0 * a0, p1 = a1 * a1, p2 = a2 * a2;
        volatile float va = p0 + p1;
        volatile float var = va + p2;
        volatile float sq = sqrtf(var);
        volatile float h = RCI * sq;
        volatile float lo_ = mu[j] - h, hi_ = mu[j] + h;
        volatile float dl = lo_ - lo[j], dh = hi_ - lo[j];
        volatile float tl = dl * invc[j], th = dh * invc[j];
        float fl = floorf(tl), fh = floorf(th);
        float cmax = (float)(cells[j] - 1);
        if (!isfinite(h) || !isfinite(fl) || !isfinite(fh) || !(fh >= 0.0f) || !(fl <= cmax)) return 0;
        b[j] = (int32_t)(fl > 0.0f ? fl : 0.0f);
        b[3 + j] = (int32_t)(fh < cmax ? fh : cmax);
        count *= (int64_t)(b[3 + j] - b[j] + 1);
    }
    memcpy(box, b, sizeof(b));
    return count;
}

static void grid_invc(const float lo[3], const float hi[3], const int32_t cells[3], float invc[3])
{
    for (int j = 0; j < 3; j++) {
        volatile float ext = hi[j] - lo[j];
        invc[j] = (float)cells[j] / ext;
    }
}

static int grid_ok(const float lo[3], const float hi[3], const int32_t cells[3])
{
    int64_t nc = 1;
    for (int j = 0; j < 3; j++) {
        if (cells[j] <= 0 || !(hi[j] > lo[j]) || !isfinite(lo[j]) || !isfinite(hi[j])) return 0;
        nc *= cells[j];
    }
    return nc < ((int64_t)1 << 31);
}

/* box[n][6] = (cx_lo, cy_lo, cz_lo, cx_hi, cy_hi, cz_hi) or -1 (the cells
 * of the cutoff ellipsoid's axis-aligned box, Sec. 4.1.1) and count[n] (its
 * number of cells); either output may be NULL. Returns the total number of
 * cells over all boxes (or -1 on bad arguments). */
int64_t orc_index_boxes(int64_t n, const float *mean, const float *scale, const float *rot,
                        const float *value, const float *weight, const float lo[3], const float hi[3],
                        const int32_t cells[3], float tau, int32_t *box, int64_t *count)
{
    if (n < 0 || !grid_ok(lo, hi, cells) || !(tau > 0.0f) || !(tau < 1.0f)) return -1;
    float invc[3];
    grid_invc(lo, hi, cells, invc);
    float RCI = index_radius(tau);
    int64_t total = 0;
    for (int64_t i = 0; i < n; i++) {
        int32_t b[6];
        int64_t c = cell_box(mean + 3 * i, scale + 3 * i, rot + 4 * i, value[i], weight[i], lo, invc, cells, RCI, b);
        if (box) memcpy(box + 6 * i, b, sizeof(b));
        if (count) count[i] = c;
        total += c;
    }
    return total;
}

/*
 * Gaussian-cell pairs (key = cx + Cx (cy + Cy cz), gid) of every cell of
 * every box (Sec. 4.1.2's block intersection lists), in lexicographic
 * (key, gid) order, and cell_offsets[k] = number of pairs with key < k for
 * k = 0..ncells. Written by counting: offsets from per-cell counts, then
 * Gaussians in increasing id append to the lists of the cells in their box.
 * Returns ORC_ERR_CAPACITY (with *n_pairs set) when capacity is too small.
 */
int orc_index(int64_t n, const float *mean, const float *scale, const float *rot,
              const float *value, const float *weight, const float lo[3], const float hi[3],
              const int32_t cells[3], float tau, uint32_t *keys, uint32_t *gids, int64_t capacity,
              uint32_t *cell_offsets, int64_t *n_pairs)
{
    if (n < 0 || !grid_ok(lo, hi, cells) || !(tau > 0.0f) || !(tau < 1.0f)) return ORC_ERR_ARG;
    int64_t ncells = (int64_t)cells[0] * cells[1] * cells[2];
    const size_t nn = (size_t)(n > 0 ? n : 1);
    int32_t *box = (int32_t *)malloc(sizeof(int32_t) * 6 * nn);
    int64_t *cursor = (int64_t *)calloc((size_t)ncells + 1, sizeof(int64_t));
    if (!box || !cursor) {
        free(box);
        free(cursor);
        return ORC_ERR_NOMEM;
    }
    int64_t P = orc_index_boxes(n, mean, scale, rot, value, weight, lo, hi, cells, tau, box, NULL);
    *n_pairs = P;
    if (P > capacity || P >= ((int64_t)1 << 32)) {
        free(box);
        free(cursor);
        return ORC_ERR_CAPACITY;
    }
    int64_t Cx = cells[0], Cy = cells[1];
    /* two sweeps over the listed cells: count per cell, then place (key, gid) */
    for (int sweep = 0; sweep < 2; sweep++) {
        if (sweep == 1) {
            for (int64_t k = 0; k < ncells; k++) cursor[k + 1] += cursor[k];
            for (int64_t k = 0; k <= ncells; k++) cell_offsets[k] = (uint32_t)cursor[k];
        }
        for (int64_t i = 0; i < n; i++) {
            const int32_t *b = box + 6 * i;
            if (b[0] < 0) continue;
            for (int64_t z = b[2]; z <= b[5]; z++)
                for (int64_t y = b[1]; y <= b[4]; y++)
                    for (int64_t x = b[0]; x <= b[3]; x++) {
                        int64_t key = x + Cx * (y + Cy * z);
                        if (sweep == 0) {
                            cursor[key + 1]++;
                        } else {
                            int64_t at = cursor[key]++;
                            keys[at] = (uint32_t)key;
                            gids[at] = (uint32_t)i;
                        }
                    }
        }
    }
    free(box);
    free(cursor);
    return ORC_OK;
}

/* ------------------------------------------------------------------------ */
/* The cells a Gaussian reaches (Sec. 4.1.1: a block needs a Gaussian in its  */
/* list exactly when the Gaussian's cutoff region overlaps it).              */
/* ------------------------------------------------------------------------ */

/*
 * Minimum of the convex quadratic f(d) = d^T A d (A symmetric positive
 * definite) over the box L <= d <= U, in float64.
 *
 * The minimiser lies in the relative interior of exactly one face of the
 * box (the box itself, one of its 6 facets, 12 edges or 8 vertices). On
 * the affine hull of a face some coordinates are fixed at a bound and the
 * others are free; there f is a convex quadratic in the free coordinates
 * whose minimiser solves A_FF d_F = -A_FX d_X. Every face whose such
 * minimiser satisfies the free coordinates' bounds gives an attained value
 * of f on the box, and the face holding the true minimiser is among them,
 * so the least of those values is the minimum. The free systems have at
 * most 3 unknowns and are solved by Cramer's rule.
 */
static double box_min_quadratic(const double A[3][3], const double L[3], const double U[3])
{
    double best = INFINITY;
    /* state per axis: 0 free, 1 fixed at L, 2 fixed at U */
    for (int code = 0; code < 27; code++) {
        int st[3] = {code % 3, (code / 3) % 3, code / 9};
        int fr[3], nf = 0;
        double d[3] = {0.0, 0.0, 0.0};
        for (int j = 0; j < 3; j++) {
            if (st[j] == 0)
                fr[nf++] = j;
            else
                d[j] = st[j] == 1 ? L[j] : U[j];
        }
        /* right-hand side b_F = -A_FX d_X */
        double b[3] = {0.0, 0.0, 0.0};
        for (int a = 0; a < nf; a++)
            for (int j = 0; j < 3; j++)
                if (st[j] != 0) b[a] -= A[fr[a]][j] * d[j];
        if (nf == 1) {
            d[fr[0]] = b[0] / A[fr[0]][fr[0]];
        } else if (nf == 2) {
            const double a00 = A[fr[0]][fr[0]], a01 = A[fr[0]][fr[1]], a11 = A[fr[1]][fr[1]];
            const double det = a00 * a11 - a01 * a01;
            if (!(det > 0.0)) continue;
            d[fr[0]] = (b[0] * a11 - a01 * b[1]) / det;
            d[fr[1]] = (a00 * b[1] - a01 * b[0]) / det;
        } else if (nf == 3) {
            /* the unconstrained minimiser d = 0 */
            d[0] = d[1] = d[2] = 0.0;
        }
        int ok = 1;
        for (int a = 0; a < nf; a++) {
            const int j = fr[a];
            if (!(d[j] >= L[j] && d[j] <= U[j])) ok = 0;
        }
        if (!ok) continue;
        double f = 0.0;
        for (int j = 0; j < 3; j++)
            for (int k = 0; k < 3; k++) f += d[j] * A[j][k] * d[k];
        if (f < best) best = f;
    }
    return best;
}

/*
 * For the selected Gaussians (sel[0..nsel), or all when sel is NULL): the
 * cells of the index grid that hold a point within the Gaussian's cutoff
 * Q <= T = 2 ln(1/tau), each cell taken as its box widened by margin cell
 * widths on every side (margin >= 0; 0 gives the cells the cutoff region
 * itself overlaps). Q over a cell is minimised exactly in float64
 * (box_min_quadratic on the inverse covariance A = R S^-2 R^T). Only cells
 * of the Gaussian's canonical box (orc_index_boxes) are examined; by
 * Cauchy-Schwarz no point outside the cutoff's own axis-aligned extent is
 * within the cutoff, and that box holds the extent with a margin.
 * count[a] = number of such cells of Gaussian sel[a]; when keys is non-NULL
 * their keys follow Gaussian after Gaussian (in increasing key) in
 * keys[0 .. sum count), at most capacity of them (ORC_ERR_CAPACITY
 * beyond). Invalid Gaussians reach no cell.
 */
int orc_reached_cells(int64_t n, const float *mean, const float *scale, const float *rot,
                      const float *value, const float *weight, const float lo[3], const float hi[3],
                      const int32_t cells[3], float tau, double margin, int64_t nsel, const int64_t *sel,
                      int nthreads, int64_t *count, uint32_t *keys, int64_t capacity)
{
    if (n < 0 || nsel < 0 || !grid_ok(lo, hi, cells) || !(tau > 0.0f) || !(tau < 1.0f) || !(margin >= 0.0))
        return ORC_ERR_ARG;
    set_threads(nthreads);
    const double T = 2.0 * log(1.0 / (double)tau);
    float invc[3];
    grid_invc(lo, hi, cells, invc);
    const float RCI = index_radius(tau);
    double width[3];
    for (int j = 0; j < 3; j++) width[j] = ((double)hi[j] - (double)lo[j]) / (double)cells[j];
    const int64_t m = sel ? nsel : n;
    int err = 0;
    for (int pass = 0; pass < (keys ? 2 : 1); pass++) {
        int64_t *start = NULL;
        if (pass == 1) {
            start = (int64_t *)malloc(sizeof(int64_t) * (size_t)(m + 1));
            if (!start) return ORC_ERR_NOMEM;
            start[0] = 0;
            for (int64_t a = 0; a < m; a++) start[a + 1] = start[a] + count[a];
            if (start[m] > capacity) {
                free(start);
                return ORC_ERR_CAPACITY;
            }
        }
#pragma omp parallel for schedule(dynamic, 8)
        for (int64_t a = 0; a < m; a++) {
            const int64_t i = sel ? sel[a] : a;
            if (i < 0 || i >= n) {
#pragma omp atomic write
                err = 1;
                continue;
            }
            int32_t b[6];
            int64_t c = cell_box(mean + 3 * i, scale + 3 * i, rot + 4 * i, value[i], weight[i], lo, invc, cells,
                                 RCI, b);
            int64_t got = 0;
            if (c > 0) {
                const double q[4] = {rot[4 * i], rot[4 * i + 1], rot[4 * i + 2], rot[4 * i + 3]};
                const double qn = sqrt(q[0] * q[0] + q[1] * q[1] + q[2] * q[2] + q[3] * q[3]);
                const double qh[4] = {q[0] / qn, q[1] / qn, q[2] / qn, q[3] / qn};
                double R[3][3], A[3][3];
                quat_to_rot(qh, R);
                for (int j = 0; j < 3; j++)
                    for (int k = 0; k < 3; k++) {
                        double acc = 0.0;
                        for (int t = 0; t < 3; t++)
                            acc += R[j][t] * R[k][t] / ((double)scale[3 * i + t] * (double)scale[3 * i + t]);
                        A[j][k] = acc;
                    }
                for (int64_t z = b[2]; z <= b[5]; z++)
                    for (int64_t y = b[1]; y <= b[4]; y++)
                        for (int64_t x = b[0]; x <= b[3]; x++) {
                            const int64_t cc[3] = {x, y, z};
                            double L[3], U[3];
                            for (int j = 0; j < 3; j++) {
                                L[j] = ((double)lo[j] + ((double)cc[j] - margin) * width[j]) - (double)mean[3 * i + j];
                                U[j] = ((double)lo[j] + ((double)cc[j] + 1.0 + margin) * width[j]) -
                                       (double)mean[3 * i + j];
                            }
                            if (box_min_quadratic(A, L, U) <= T) {
                                if (pass == 1) keys[start[a] + got] = (uint32_t)(x + (int64_t)cells[0] *
                                                                                   (y + (int64_t)cells[1] * z));
                                got++;
                            }
                        }
            }
            if (pass == 0) count[a] = got;
        }
        free(start);
    }
    return err ? ORC_ERR_ARG : ORC_OK;
}
