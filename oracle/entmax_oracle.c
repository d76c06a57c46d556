/*
 * entmax_oracle.c -- plain fp64 CPU reference for alpha-entmax attention.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the oracle that the GPU path is
 * checked against.  Only the test suite, the smoke check and the bench's CPU
 * baseline may load it; the product path never calls it and shares no code,
 * header or constant with it.
 *
 * What it computes (AdaSplash, arXiv 2502.12082), one attention head at a
 * time, everything in double precision:
 *
 *   x_ij  = (alpha-1) * scale * <q_i, k_j>              scores in the
 *                                                       coordinates of Eq. 2
 *   tau_i = the unique root of f(tau) = sum_j [x_ij - tau]_+^gamma - 1
 *           (Eq. 3), gamma = 1/(alpha-1), found by long bisection (Eq. 4)
 *           on the bracket [max_j x_ij - 1, max_j x_ij - n_i^(1-alpha)]
 *           that Algorithm 1 initialises with
 *   p_ij  = [x_ij - tau_i]_+^gamma                      (Eq. 2)
 *   u_ij  = [x_ij - tau_i]_+^(gamma-1) on x_ij > tau_i, 0 elsewhere
 *           (= p^(2-alpha), the sparse Jacobian of Sec. 3.2.2, App. A.2)
 *   O_i   = sum_j p_ij v_j                              (App. A.1)
 *   O2_i  = sum_j u_ij v_j / sum_j u_ij                 (App. A.2, O^(2))
 *   delta_i = <dO_i, O2_i>                              (App. A.2)
 *   dS_ij = u_ij (<dO_i, v_j> - delta_i)                (App. A.2)
 *   dQ_i  = scale * sum_j dS_ij k_j,  dK_j = scale * sum_i dS_ij q_i,
 *   dV_j  = sum_i p_ij dO_i                             (Eq. 11-13, App. A.2)
 *   margin_IJ = max over valid (i in I, j in J) of (x_ij - tau_i), with
 *           64-row / 64-column blocks; the block mask of Eq. 8 is
 *           margin_IJ > 0 (some probability in the block is positive).
 *
 * "Valid" pairs: all j < n, or j <= i when causal (top-left aligned).
 * n_i is the number of valid keys of row i.
 *
 * The Halley-bisection iterates of Algorithm 1 are also provided in fp64
 * (eo_halley_bisection_trace) as a diagnostic of the paper's solver; the
 * attention outputs above use the exact root, not those iterates.
 *
 * Work is split over rows (or columns) with POSIX threads; every output
 * element is produced by exactly one thread in a fixed order, so results do
 * not depend on the thread count.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define EO_BLOCK 64

/* ---------------------------------------------------------------- helpers */

/* Neumaier (compensated) summation state. */
typedef struct {
    double sum, comp;
} eo_acc;

static void acc_add(eo_acc* a, double v) {
    double t = a->sum + v;
    if (fabs(a->sum) >= fabs(v))
        a->comp += (a->sum - t) + v;
    else
        a->comp += (v - t) + a->sum;
    a->sum = t;
}

static double acc_value(const eo_acc* a) { return a->sum + a->comp; }

static double dot(const double* a, const double* b, int d) {
    double s = 0.0;
    for (int t = 0; t < d; ++t) s += a[t] * b[t];
    return s;
}

/* Number of keys row i may attend to. */
static int valid_keys(int n, int causal, int i) { return causal ? i + 1 : n; }

/* Eq. 3 with compensated summation: f(tau) = sum_j [x_j - tau]_+^gamma - 1. */
static double root_function(const double* x, int n, double gamma, double tau) {
    eo_acc a = {0.0, 0.0};
    for (int j = 0; j < n; ++j) {
        double z = x[j] - tau;
        if (z > 0.0) acc_add(&a, pow(z, gamma));
    }
    return acc_value(&a) - 1.0;
}

/* ------------------------------------------------------- threshold (tau) */

/*
 * Exact threshold of alpha-entmax for one score row x (already in Eq. 2
 * coordinates, i.e. multiplied by alpha-1).  Bracket of Algorithm 1; bisection
 * rule of Eq. 4, taking the "otherwise" branch when f(tau) == 0; iterate until
 * the midpoint can no longer be distinguished from an end point in fp64.
 */
double eo_entmax_threshold(const double* x, int n, double alpha) {
    const double gamma = 1.0 / (alpha - 1.0);
    double m = x[0];
    for (int j = 1; j < n; ++j)
        if (x[j] > m) m = x[j];
    double lo = m - 1.0;
    double hi = m - pow((double)n, 1.0 - alpha);
    for (int it = 0; it < 200; ++it) {
        double mid = 0.5 * (lo + hi);
        if (mid <= lo || mid >= hi) break;
        if (root_function(x, n, gamma, mid) < 0.0)
            hi = mid;
        else
            lo = mid;
    }
    return 0.5 * (lo + hi);
}

/* alpha-entmax of one row (Eq. 2): p_j = [x_j - tau]_+^gamma; returns tau. */
double eo_entmax_row(const double* x, int n, double alpha, double* p) {
    const double gamma = 1.0 / (alpha - 1.0);
    double tau = eo_entmax_threshold(x, n, alpha);
    for (int j = 0; j < n; ++j) {
        double z = x[j] - tau;
        p[j] = z > 0.0 ? pow(z, gamma) : 0.0;
    }
    return tau;
}

/*
 * Gradient of sum_j g_j p_j with respect to x / (alpha-1) for one row, where
 * p = alpha-entmax(x) with threshold tau (Sec. 3.2.2): with u_j = [x_j -
 * tau]_+^(gamma-1) on the strict support z > 0 (0 elsewhere), the Jacobian is
 * Diag(u) - u u^T / sum(u), so out_j = u_j (g_j - <u, g> / sum(u)).  The
 * (alpha-1) of the input scaling cancels gamma's factor, as in the attention
 * backward.
 */
void eo_entmax_row_bwd(const double* x, int n, double alpha, double tau, const double* g,
                       double* out) {
    const double gamma = 1.0 / (alpha - 1.0);
    eo_acc su = {0.0, 0.0}, sug = {0.0, 0.0};
    for (int j = 0; j < n; ++j) {
        const double z = x[j] - tau;
        const double u = z > 0.0 ? pow(z, gamma - 1.0) : 0.0;
        out[j] = u;
        acc_add(&su, u);
        acc_add(&sug, u * g[j]);
    }
    const double mean = acc_value(&su) > 0.0 ? acc_value(&sug) / acc_value(&su) : 0.0;
    for (int j = 0; j < n; ++j) out[j] = out[j] * (g[j] - mean);
}

/*
 * Algorithm 1 (Halley-bisection) run in fp64 on one row x in Eq. 2
 * coordinates, for the iterations-versus-error diagnostic.  Writes the tau
 * held before each of the T updates and after the last one (T+1 values) into
 * trace.  One iteration = evaluate f, f', f'' (Eq. 3, 6, 7) at tau, update the
 * bracket with B_f (Eq. 4), then accept the Halley value H_f (Eq. 5) if it is
 * finite and inside [lo, hi], else take the bracket midpoint.  Sums run over
 * the strict support x_j > tau only.
 */
void eo_halley_bisection_trace(const double* x, int n, double alpha, int T, double* trace) {
    const double gamma = 1.0 / (alpha - 1.0);
    double m = x[0];
    for (int j = 1; j < n; ++j)
        if (x[j] > m) m = x[j];
    double lo = m - 1.0;
    double hi = m - pow((double)n, 1.0 - alpha);
    double tau = 0.5 * (lo + hi);
    for (int it = 0; it < T; ++it) {
        trace[it] = tau;
        double s0 = 0.0, s1 = 0.0, s2 = 0.0;
        for (int j = 0; j < n; ++j) {
            double z = x[j] - tau;
            if (z > 0.0) {
                s0 += pow(z, gamma);
                s1 += pow(z, gamma - 1.0);
                s2 += pow(z, gamma - 2.0);
            }
        }
        double f = s0 - 1.0;
        double f1 = -gamma * s1;                   /* Eq. 6 */
        double f2 = gamma * (gamma - 1.0) * s2;    /* Eq. 7: (2-a)/(a-1)^2 */
        if (f < 0.0)
            hi = tau;
        else
            lo = tau;
        double th = tau - 2.0 * f * f1 / (2.0 * f1 * f1 - f * f2);
        if (isfinite(th) && th >= lo && th <= hi)
            tau = th;
        else
            tau = 0.5 * (lo + hi);
    }
    trace[T] = tau;
}

/* ------------------------------------------------------- threaded drivers */

typedef struct {
    /* problem */
    int n, d, causal;
    double alpha, scale;
    const double *q, *k, *v, *dout, *tau, *delta;
    /* work list: either an explicit index list or the range [lo, hi) */
    const int32_t* idx;
    int count, lo;
    /* outputs */
    double *tau_out, *o, *o2, *dq, *dk, *dv, *margin;
    /* threading */
    int tid, nthreads;
} eo_job;

typedef void (*eo_worker)(eo_job* job, int item);

typedef struct {
    eo_job* job;
    eo_worker fn;
} eo_thread_arg;

static void* thread_main(void* p) {
    eo_thread_arg* a = (eo_thread_arg*)p;
    eo_job* job = a->job;
    for (int t = job->tid; t < job->count; t += job->nthreads) {
        int item = job->idx ? job->idx[t] : job->lo + t;
        a->fn(job, item);
    }
    return NULL;
}

static void run_parallel(eo_job* proto, eo_worker fn, int nthreads) {
    if (nthreads < 1) nthreads = 1;
    if (nthreads > 256) nthreads = 256;
    eo_job jobs[256];
    eo_thread_arg args[256];
    pthread_t th[256];
    for (int t = 0; t < nthreads; ++t) {
        jobs[t] = *proto;
        jobs[t].tid = t;
        jobs[t].nthreads = nthreads;
        args[t].job = &jobs[t];
        args[t].fn = fn;
    }
    for (int t = 1; t < nthreads; ++t) pthread_create(&th[t], NULL, thread_main, &args[t]);
    thread_main(&args[0]);
    for (int t = 1; t < nthreads; ++t) pthread_join(th[t], NULL);
}

/* Score row i in Eq. 2 coordinates over its valid keys; returns n_i. */
static int score_row(const eo_job* J, int i, double* x) {
    int ni = valid_keys(J->n, J->causal, i);
    const double* qi = J->q + (size_t)i * J->d;
    double c = (J->alpha - 1.0) * J->scale;
    for (int j = 0; j < ni; ++j) x[j] = c * dot(qi, J->k + (size_t)j * J->d, J->d);
    return ni;
}

static void tau_worker(eo_job* J, int i) {
    double* x = (double*)malloc(sizeof(double) * (size_t)J->n);
    int ni = score_row(J, i, x);
    J->tau_out[i] = eo_entmax_threshold(x, ni, J->alpha);
    free(x);
}

static void fwd_worker(eo_job* J, int i) {
    const int d = J->d;
    const double gamma = 1.0 / (J->alpha - 1.0);
    double* x = (double*)malloc(sizeof(double) * (size_t)J->n);
    int ni = score_row(J, i, x);
    double ti = J->tau[i];
    double* o = J->o ? J->o + (size_t)i * d : NULL;
    double* o2 = J->o2 ? J->o2 + (size_t)i * d : NULL;
    if (o) memset(o, 0, sizeof(double) * d);
    if (o2) memset(o2, 0, sizeof(double) * d);
    double usum = 0.0;
    for (int j = 0; j < ni; ++j) {
        double z = x[j] - ti;
        if (z <= 0.0) continue;
        double p = pow(z, gamma);
        double u = pow(z, gamma - 1.0);
        const double* vj = J->v + (size_t)j * d;
        usum += u;
        for (int t = 0; t < d; ++t) {
            if (o) o[t] += p * vj[t];
            if (o2) o2[t] += u * vj[t];
        }
    }
    if (o2)
        for (int t = 0; t < d; ++t) o2[t] /= usum;
    free(x);
}

static void dq_worker(eo_job* J, int i) {
    const int d = J->d;
    const double gamma = 1.0 / (J->alpha - 1.0);
    double* x = (double*)malloc(sizeof(double) * (size_t)J->n);
    int ni = score_row(J, i, x);
    double ti = J->tau[i], di = J->delta[i];
    const double* doi = J->dout + (size_t)i * d;
    double* dq = J->dq + (size_t)i * d;
    memset(dq, 0, sizeof(double) * d);
    for (int j = 0; j < ni; ++j) {
        double z = x[j] - ti;
        if (z <= 0.0) continue;
        double u = pow(z, gamma - 1.0);
        double ds = u * (dot(doi, J->v + (size_t)j * d, d) - di);
        const double* kj = J->k + (size_t)j * d;
        for (int t = 0; t < d; ++t) dq[t] += ds * kj[t];
    }
    for (int t = 0; t < d; ++t) dq[t] *= J->scale;
    free(x);
}

static void dkdv_worker(eo_job* J, int j) {
    const int d = J->d;
    const double gamma = 1.0 / (J->alpha - 1.0);
    const double c = (J->alpha - 1.0) * J->scale;
    const double* kj = J->k + (size_t)j * d;
    const double* vj = J->v + (size_t)j * d;
    double* dk = J->dk + (size_t)j * d;
    double* dv = J->dv + (size_t)j * d;
    memset(dk, 0, sizeof(double) * d);
    memset(dv, 0, sizeof(double) * d);
    int i0 = J->causal ? j : 0; /* rows that may attend to key j */
    for (int i = i0; i < J->n; ++i) {
        const double* qi = J->q + (size_t)i * d;
        double z = c * dot(qi, kj, d) - J->tau[i];
        if (z <= 0.0) continue;
        double p = pow(z, gamma);
        double u = pow(z, gamma - 1.0);
        const double* doi = J->dout + (size_t)i * d;
        double ds = u * (dot(doi, vj, d) - J->delta[i]);
        for (int t = 0; t < d; ++t) {
            dk[t] += ds * qi[t];
            dv[t] += p * doi[t];
        }
    }
    for (int t = 0; t < d; ++t) dk[t] *= J->scale;
}

static void margin_worker(eo_job* J, int I) {
    /* one 64-row query block I: margin over every 64-column key block J */
    const int n = J->n, T = (n + EO_BLOCK - 1) / EO_BLOCK;
    double* x = (double*)malloc(sizeof(double) * (size_t)n);
    double* row = J->margin + (size_t)I * T;
    for (int b = 0; b < T; ++b) row[b] = -INFINITY;
    int iend = (I + 1) * EO_BLOCK < n ? (I + 1) * EO_BLOCK : n;
    for (int i = I * EO_BLOCK; i < iend; ++i) {
        int ni = score_row(J, i, x);
        for (int j = 0; j < ni; ++j) {
            double z = x[j] - J->tau[i];
            if (z > row[j / EO_BLOCK]) row[j / EO_BLOCK] = z;
        }
    }
    free(x);
}

/* ------------------------------------------------------------ public API */
/*
 * All matrices are row-major [n, d] fp64 for ONE head.  `rows` / `cols` is an
 * optional int32 index list (NULL: all of 0..n-1).  Outputs are indexed by the
 * absolute row / column, so the caller passes full-size [n] / [n, d] buffers
 * and only the listed entries are written.
 */

void eo_tau(int n, int d, const double* q, const double* k, double alpha, double scale,
            int causal, const int32_t* rows, int nrows, double* tau, int nthreads) {
    eo_job J;
    memset(&J, 0, sizeof J);
    J.n = n; J.d = d; J.causal = causal; J.alpha = alpha; J.scale = scale;
    J.q = q; J.k = k; J.idx = rows; J.count = rows ? nrows : n; J.tau_out = tau;
    run_parallel(&J, tau_worker, nthreads);
}

void eo_forward_rows(int n, int d, const double* q, const double* k, const double* v,
                     double alpha, double scale, int causal, const double* tau,
                     const int32_t* rows, int nrows, double* o, double* o2, int nthreads) {
    eo_job J;
    memset(&J, 0, sizeof J);
    J.n = n; J.d = d; J.causal = causal; J.alpha = alpha; J.scale = scale;
    J.q = q; J.k = k; J.v = v; J.tau = tau; J.idx = rows; J.count = rows ? nrows : n;
    J.o = o; J.o2 = o2;
    run_parallel(&J, fwd_worker, nthreads);
}

/* margin[I*T + J] for the listed 64-row query blocks I (NULL: all T), every
 * key block J; reads tau of the rows of those blocks only. */
void eo_block_margin(int n, int d, const double* q, const double* k, double alpha,
                     double scale, int causal, const double* tau, const int32_t* brows,
                     int nbrows, double* margin, int nthreads) {
    eo_job J;
    memset(&J, 0, sizeof J);
    J.n = n; J.d = d; J.causal = causal; J.alpha = alpha; J.scale = scale;
    J.q = q; J.k = k; J.tau = tau; J.margin = margin;
    J.idx = brows;
    J.count = brows ? nbrows : (n + EO_BLOCK - 1) / EO_BLOCK;
    run_parallel(&J, margin_worker, nthreads);
}

/* delta_i = <dO_i, O2_i> for the listed rows (O2 from eo_forward_rows). */
void eo_delta_rows(int n, int d, const double* dout, const double* o2, const int32_t* rows,
                   int nrows, double* delta) {
    int count = rows ? nrows : n;
    for (int t = 0; t < count; ++t) {
        int i = rows ? rows[t] : t;
        delta[i] = dot(dout + (size_t)i * d, o2 + (size_t)i * d, d);
    }
}

void eo_dq_rows(int n, int d, const double* q, const double* k, const double* v,
                const double* dout, double alpha, double scale, int causal, const double* tau,
                const double* delta, const int32_t* rows, int nrows, double* dq, int nthreads) {
    eo_job J;
    memset(&J, 0, sizeof J);
    J.n = n; J.d = d; J.causal = causal; J.alpha = alpha; J.scale = scale;
    J.q = q; J.k = k; J.v = v; J.dout = dout; J.tau = tau; J.delta = delta;
    J.idx = rows; J.count = rows ? nrows : n; J.dq = dq;
    run_parallel(&J, dq_worker, nthreads);
}

/* dK_j, dV_j for the listed columns; reads tau and delta of every row that
 * may attend to those columns (all rows, or rows >= j when causal). */
void eo_dkdv_cols(int n, int d, const double* q, const double* k, const double* v,
                  const double* dout, double alpha, double scale, int causal,
                  const double* tau, const double* delta, const int32_t* cols, int ncols,
                  double* dk, double* dv, int nthreads) {
    eo_job J;
    memset(&J, 0, sizeof J);
    J.n = n; J.d = d; J.causal = causal; J.alpha = alpha; J.scale = scale;
    J.q = q; J.k = k; J.v = v; J.dout = dout; J.tau = tau; J.delta = delta;
    J.idx = cols; J.count = cols ? ncols : n; J.dk = dk; J.dv = dv;
    run_parallel(&J, dkdv_worker, nthreads);
}
