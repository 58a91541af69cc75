/*
 * mesa_oracle.c -- plain fp64 CPU reference of the Mesa layer.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path (libmesa, its kernels
 * or its Python binding) may include, link or call this file.  Only the test
 * suite, the smoke check and the benchmark's CPU-baseline leg use it.  It
 * shares no code, header, table or helper with the HIP path.
 *
 * What it computes (MesaNet, arXiv 2506.05233):
 *   For each (batch, head) independently, starting from H_0 = G_0 = 0:
 *     H_t = gamma_t H_{t-1} + beta_t k_t k_t^T          (Sec. 2, state recurrences;
 *     G_t = gamma_t G_{t-1} + beta_t v_t k_t^T           App. E, gated form)
 *     q*_t = (H_t + Lambda)^{-1} q_t                     (Eq. mesa-layer-final)
 *     o_t  = G_t q*_t                                    (App. D, Eq. app-mesa-dynamics)
 *   The solve is either
 *     - fixed-step conjugate gradients following App. C, Alg. 1 with tolerance
 *       zero: Jacobi-scaled start x0 = q / diag(H_t + Lambda) (App. C text),
 *       one matrix-vector product for the first residual, then n_cg loop
 *       iterations, or
 *     - an exact Cholesky solve (the closed form of Eq. mesa-layer-objective).
 *   Nothing is chunked: this is the sequential recurrence, token by token.
 *
 * Readings adopted where the paper is ambiguous:
 *   - the Jacobi diagonal is that of the system being solved, H_t + Lambda;
 *   - n_cg counts loop iterations, so a solve does n_cg + 1 products;
 *   - the loop stops, after updating x, when the new residual meets Alg. 1's
 *     relative test |r_{k+1}| <= eps |r_0| (squared: delta_new <= eps^2 delta_0;
 *     with eps = 0 that is a residual of exactly zero); it also stops, keeping
 *     x, when the squared residual is zero before a step or when p^T A p <= 0
 *     (guards for q = 0 and breakdown).  "Zero" is read in floating point: in
 *     exact arithmetic CG reaches a zero residual within n steps, but the
 *     recursively updated residual of a floating-point run keeps shrinking past
 *     the attainable accuracy and finally underflows, where alpha = delta / p^T A p
 *     loses all precision.  So a squared residual at or below 2^-200 |b|^2 counts
 *     as zero (x then changes by less than 2^-100 relative per step);
 *   - beta enters once: H += beta k k^T, G += beta v k^T;
 *   - decode updates the state with the new token first, then solves.
 *
 * Backward pass (App. D, "Mesa layer backward pass"), given e_t = dL/do_t:
 *     u_t  = G_t^T e_t,  e*_t = (H_t + Lambda)^{-1} u_t  (same solver as q*_t)
 *     dL/dq_t = e*_t,   dL/dLambda_a = -sum_t q*_{t,a} e*_{t,a}
 *   and, with the adjoints of the states accumulated backwards in time,
 *     DG_s = sum_{t>=s} zeta_{t,s} e_t q*_t^T  = e_s q*_s^T + gamma_{s+1} DG_{s+1}
 *     DH_s = -sum_{t>=s} zeta_{t,s} e*_t q*_t^T = -e*_s q*_s^T + gamma_{s+1} DH_{s+1},
 *     dL/dv_s     = beta_s DG_s k_s
 *     dL/dk_s     = beta_s (DG_s^T v_s + (DH_s + DH_s^T) k_s)
 *     dL/dbeta_s  = v_s^T DG_s k_s + k_s^T DH_s k_s
 *     dL/dgamma_s = <DG_s, G_{s-1}> + <DH_s, H_{s-1}>   (Frobenius products).
 *   This is the gradient of the layer with q*_t taken as the exact solution
 *   (the paper's implicit differentiation; CG approximates both solves).  The
 *   paper writes its sums without the input gate and with e*_t in the value term
 *   of dL/dk_s; differentiating e_t^T G_t q*_t with respect to k_s gives
 *   beta_s zeta_{t,s} q*_t (e_t^T v_s), the reading taken here.
 *
 * All arrays are dense, row-major, fp64, host memory, owned by the caller.
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum { ORACLE_SOLVE_CG = 0, ORACLE_SOLVE_CHOLESKY = 1 };
enum { ORACLE_INIT_JACOBI = 0, ORACLE_INIT_QUERY = 1 };

/* CG on the SPD system A x = b (App. C, Alg. 1): at most n_cg loop iterations,
 * relative tolerance eps >= 0 (eps = 0: the fixed-step solve).
 * init = ORACLE_INIT_JACOBI: x0 = b / diag(A)  (the paper's choice);
 * init = ORACLE_INIT_QUERY : x0 = b            (the "zero CG steps gives GLA"
 *                                               remark of Sec. 3; tests only).
 * work must hold 3n doubles.  Returns the number of loop iterations that
 * updated x. */
int oracle_cg(const double* A, const double* b, int64_t n, int n_cg, int init, double eps,
              double* x, double* work)
{
    double* r = work;
    double* p = work + n;
    double* w = work + 2 * n;
    for (int64_t i = 0; i < n; ++i)
        x[i] = (init == ORACLE_INIT_QUERY) ? b[i] : b[i] / A[i * n + i];
    double delta = 0.0, bb = 0.0;
    for (int64_t i = 0; i < n; ++i) {
        double ax = 0.0;
        for (int64_t j = 0; j < n; ++j) ax += A[i * n + j] * x[j];
        r[i] = b[i] - ax;
        p[i] = r[i];
        delta += r[i] * r[i];
        bb += b[i] * b[i];
    }
    const double delta0 = delta;  /* |r_0|^2, the reference of the relative test */
    const double zero = ldexp(bb, -200);  /* squared residuals at or below this are zero */
    int it = 0;
    for (; it < n_cg; ++it) {
        if (!(delta > zero)) break;
        double pw = 0.0;
        for (int64_t i = 0; i < n; ++i) {
            double s = 0.0;
            for (int64_t j = 0; j < n; ++j) s += A[i * n + j] * p[j];
            w[i] = s;
            pw += p[i] * s;
        }
        if (!(pw > 0.0)) break;
        double alpha = delta / pw;
        double delta_new = 0.0;
        for (int64_t i = 0; i < n; ++i) {
            x[i] += alpha * p[i];
            r[i] -= alpha * w[i];
            delta_new += r[i] * r[i];
        }
        if (delta_new <= eps * eps * delta0 || delta_new <= zero) { ++it; break; }
        double beta_cg = delta_new / delta;
        for (int64_t i = 0; i < n; ++i) p[i] = r[i] + beta_cg * p[i];
        delta = delta_new;
    }
    return it;
}

/* Exact solve of the SPD system A x = b by Cholesky, A = L L^T.
 * work must hold n*n doubles.  Returns 0, or -1 if A is not positive definite. */
int oracle_cholesky_solve(const double* A, const double* b, int64_t n, double* x, double* work)
{
    double* L = work;
    memset(L, 0, (size_t)(n * n) * sizeof(double));
    for (int64_t j = 0; j < n; ++j) {
        double d = A[j * n + j];
        for (int64_t m = 0; m < j; ++m) d -= L[j * n + m] * L[j * n + m];
        if (!(d > 0.0)) return -1;
        double ljj = sqrt(d);
        L[j * n + j] = ljj;
        for (int64_t i = j + 1; i < n; ++i) {
            double s = A[i * n + j];
            for (int64_t m = 0; m < j; ++m) s -= L[i * n + m] * L[j * n + m];
            L[i * n + j] = s / ljj;
        }
    }
    /* forward: L y = b (y stored in x) */
    for (int64_t i = 0; i < n; ++i) {
        double s = b[i];
        for (int64_t m = 0; m < i; ++m) s -= L[i * n + m] * x[m];
        x[i] = s / L[i * n + i];
    }
    /* backward: L^T x = y */
    for (int64_t i = n - 1; i >= 0; --i) {
        double s = x[i];
        for (int64_t m = i + 1; m < n; ++m) s -= L[m * n + i] * x[m];
        x[i] = s / L[i * n + i];
    }
    return 0;
}

/* One token of the recurrence on one (batch, head): update, solve, read out.
 * H [dk*dk], G [dv*dk] are updated in place.  A_work holds dk*dk, solve_work
 * holds max(3*dk, dk*dk), xq holds dk (returns q*).  Returns 0 or -1. */
static int mesa_token(double* H, double* G, const double* q, const double* k, const double* v,
                      double gamma, double beta, const double* lambda, int64_t dk, int64_t dv,
                      int n_cg, int solver, int init, double eps, double* o, double* xq,
                      int32_t* steps, double* A_work, double* solve_work)
{
    for (int64_t a = 0; a < dk; ++a)
        for (int64_t b = 0; b < dk; ++b)
            H[a * dk + b] = gamma * H[a * dk + b] + beta * k[a] * k[b];
    for (int64_t a = 0; a < dv; ++a)
        for (int64_t b = 0; b < dk; ++b)
            G[a * dk + b] = gamma * G[a * dk + b] + beta * v[a] * k[b];
    for (int64_t a = 0; a < dk; ++a)
        for (int64_t b = 0; b < dk; ++b)
            A_work[a * dk + b] = H[a * dk + b] + (a == b ? lambda[a] : 0.0);
    if (solver == ORACLE_SOLVE_CHOLESKY) {
        if (oracle_cholesky_solve(A_work, q, dk, xq, solve_work) != 0) return -1;
    } else {
        const int it = oracle_cg(A_work, q, dk, n_cg, init, eps, xq, solve_work);
        if (steps) *steps = it;
    }
    for (int64_t a = 0; a < dv; ++a) {
        double s = 0.0;
        for (int64_t b = 0; b < dk; ++b) s += G[a * dk + b] * xq[b];
        o[a] = s;
    }
    return 0;
}

typedef struct {
    const double *q, *k, *v, *gamma, *beta, *lambda;
    int64_t B, Hh, T, dk, dv;
    int n_cg, solver, init;
    double eps;
    int32_t* steps;
    double *out, *qstar, *final_H, *final_G;
    double *state_H, *state_G;   /* decode: in/out states; forward: NULL */
    int n_threads, tid;
    int status;
} oracle_job;

static void* forward_worker(void* arg)
{
    oracle_job* j = (oracle_job*)arg;
    const int64_t dk = j->dk, dv = j->dv, T = j->T;
    double* H = (double*)malloc((size_t)(dk * dk) * sizeof(double));
    double* G = (double*)malloc((size_t)(dv * dk) * sizeof(double));
    double* A = (double*)malloc((size_t)(dk * dk) * sizeof(double));
    double* sw = (double*)malloc((size_t)(dk * dk + 3 * dk) * sizeof(double));
    double* xq = (double*)malloc((size_t)dk * sizeof(double));
    j->status = 0;
    for (int64_t bh = j->tid; bh < j->B * j->Hh; bh += j->n_threads) {
        const int64_t h = bh % j->Hh;
        memset(H, 0, (size_t)(dk * dk) * sizeof(double));
        memset(G, 0, (size_t)(dv * dk) * sizeof(double));
        for (int64_t t = 0; t < T; ++t) {
            const int64_t tok = bh * T + t;
            if (mesa_token(H, G, j->q + tok * dk, j->k + tok * dk, j->v + tok * dv,
                           j->gamma[tok], j->beta[tok], j->lambda + h * dk, dk, dv,
                           j->n_cg, j->solver, j->init, j->eps, j->out + tok * dv, xq,
                           j->steps ? j->steps + tok : NULL, A, sw) != 0)
                j->status = -1;
            if (j->qstar) memcpy(j->qstar + tok * dk, xq, (size_t)dk * sizeof(double));
        }
        if (j->final_H) memcpy(j->final_H + bh * dk * dk, H, (size_t)(dk * dk) * sizeof(double));
        if (j->final_G) memcpy(j->final_G + bh * dv * dk, G, (size_t)(dv * dk) * sizeof(double));
    }
    free(H); free(G); free(A); free(sw); free(xq);
    return NULL;
}

static void* decode_worker(void* arg)
{
    oracle_job* j = (oracle_job*)arg;
    const int64_t dk = j->dk, dv = j->dv;
    double* A = (double*)malloc((size_t)(dk * dk) * sizeof(double));
    double* sw = (double*)malloc((size_t)(dk * dk + 3 * dk) * sizeof(double));
    double* xq = (double*)malloc((size_t)dk * sizeof(double));
    j->status = 0;
    for (int64_t bh = j->tid; bh < j->B * j->Hh; bh += j->n_threads) {
        const int64_t h = bh % j->Hh;
        if (mesa_token(j->state_H + bh * dk * dk, j->state_G + bh * dv * dk,
                       j->q + bh * dk, j->k + bh * dk, j->v + bh * dv,
                       j->gamma[bh], j->beta[bh], j->lambda + h * dk, dk, dv,
                       j->n_cg, j->solver, j->init, j->eps, j->out + bh * dv, xq,
                       j->steps ? j->steps + bh : NULL, A, sw) != 0)
            j->status = -1;
        if (j->qstar) memcpy(j->qstar + bh * dk, xq, (size_t)dk * sizeof(double));
    }
    free(A); free(sw); free(xq);
    return NULL;
}

static int run_jobs(oracle_job* proto, void* (*fn)(void*), int n_threads)
{
    const int64_t units = proto->B * proto->Hh;
    if (n_threads < 1) n_threads = 1;
    if (n_threads > units) n_threads = (int)(units > 0 ? units : 1);
    oracle_job* jobs = (oracle_job*)malloc((size_t)n_threads * sizeof(oracle_job));
    pthread_t* th = (pthread_t*)malloc((size_t)n_threads * sizeof(pthread_t));
    for (int i = 0; i < n_threads; ++i) {
        jobs[i] = *proto;
        jobs[i].n_threads = n_threads;
        jobs[i].tid = i;
    }
    for (int i = 1; i < n_threads; ++i) pthread_create(&th[i], NULL, fn, &jobs[i]);
    fn(&jobs[0]);
    int status = jobs[0].status;
    for (int i = 1; i < n_threads; ++i) {
        pthread_join(th[i], NULL);
        if (jobs[i].status != 0) status = jobs[i].status;
    }
    free(jobs);
    free(th);
    return status;
}

/* Whole-sequence forward.  q,k [B,Hh,T,dk]; v [B,Hh,T,dv]; gamma,beta [B,Hh,T];
 * lambda [Hh,dk]; CG tolerance eps (0: fixed steps); out [B,Hh,T,dv]; optional
 * (may be NULL): qstar [B,Hh,T,dk], final_H [B,Hh,dk,dk], final_G [B,Hh,dv,dk],
 * steps [B,Hh,T] (CG iterations per token).  Returns 0, or -1 if a Cholesky
 * solve met a non-positive pivot. */
int oracle_forward(const double* q, const double* k, const double* v, const double* gamma,
                   const double* beta, const double* lambda, int64_t B, int64_t Hh, int64_t T,
                   int64_t dk, int64_t dv, int n_cg, int solver, int init, double eps, double* out,
                   double* qstar, double* final_H, double* final_G, int32_t* steps, int n_threads)
{
    oracle_job proto;
    memset(&proto, 0, sizeof(proto));
    proto.q = q; proto.k = k; proto.v = v; proto.gamma = gamma; proto.beta = beta;
    proto.lambda = lambda; proto.B = B; proto.Hh = Hh; proto.T = T; proto.dk = dk; proto.dv = dv;
    proto.n_cg = n_cg; proto.solver = solver; proto.init = init; proto.out = out;
    proto.qstar = qstar; proto.final_H = final_H; proto.final_G = final_G;
    proto.eps = eps; proto.steps = steps;
    return run_jobs(&proto, forward_worker, n_threads);
}

/* One recurrent decode step from the given states (updated in place).
 * state_H [N,Hh,dk,dk]; state_G [N,Hh,dv,dk]; q,k [N,Hh,dk]; v [N,Hh,dv];
 * gamma,beta [N,Hh]; lambda [Hh,dk]; CG tolerance eps; out [N,Hh,dv];
 * qstar [N,Hh,dk] and steps [N,Hh] may be NULL. */
int oracle_decode_step(double* state_H, double* state_G, const double* q, const double* k,
                       const double* v, const double* gamma, const double* beta,
                       const double* lambda, int64_t N, int64_t Hh, int64_t dk, int64_t dv,
                       int n_cg, int solver, int init, double eps, double* out, double* qstar,
                       int32_t* steps, int n_threads)
{
    oracle_job proto;
    memset(&proto, 0, sizeof(proto));
    proto.q = q; proto.k = k; proto.v = v; proto.gamma = gamma; proto.beta = beta;
    proto.lambda = lambda; proto.B = N; proto.Hh = Hh; proto.T = 1; proto.dk = dk; proto.dv = dv;
    proto.n_cg = n_cg; proto.solver = solver; proto.init = init; proto.out = out;
    proto.qstar = qstar; proto.state_H = state_H; proto.state_G = state_G;
    proto.eps = eps; proto.steps = steps;
    return run_jobs(&proto, decode_worker, n_threads);
}

/* ------------------------------------------------------------------ backward */

typedef struct {
    const double *q, *k, *v, *gamma, *beta, *lambda, *dout;
    int64_t B, Hh, T, dk, dv;
    int n_cg, solver, init;
    double *dq, *dk_out, *dv_out, *dgamma, *dbeta, *dlam_part; /* dlam_part [B*Hh, dk] */
    double *qstar, *estar;                                      /* may be NULL */
    int n_threads, tid;
    int status;
} oracle_bwd_job;

enum { BWD_BLOCK = 64 };  /* tokens between state checkpoints */

/* A x = b with the job's solver; x and work as for mesa_token. */
static int bwd_solve(const oracle_bwd_job* j, const double* A, const double* b, double* x, double* sw)
{
    if (j->solver == ORACLE_SOLVE_CHOLESKY) return oracle_cholesky_solve(A, b, j->dk, x, sw);
    oracle_cg(A, b, j->dk, j->n_cg, j->init, 0.0, x, sw);
    return 0;
}

static void state_step(double* H, double* G, const double* k, const double* v, double gamma, double beta,
                       int64_t dk, int64_t dv)
{
    for (int64_t a = 0; a < dk; ++a)
        for (int64_t b = 0; b < dk; ++b) H[a * dk + b] = gamma * H[a * dk + b] + beta * k[a] * k[b];
    for (int64_t a = 0; a < dv; ++a)
        for (int64_t b = 0; b < dk; ++b) G[a * dk + b] = gamma * G[a * dk + b] + beta * v[a] * k[b];
}

static void* backward_worker(void* arg)
{
    oracle_bwd_job* j = (oracle_bwd_job*)arg;
    const int64_t dk = j->dk, dv = j->dv, T = j->T;
    const int64_t nH = dk * dk, nG = dv * dk, nblk = (T + BWD_BLOCK - 1) / BWD_BLOCK;
    double* H = (double*)malloc((size_t)nH * sizeof(double));
    double* G = (double*)malloc((size_t)nG * sizeof(double));
    double* A = (double*)malloc((size_t)nH * sizeof(double));
    double* sw = (double*)malloc((size_t)(nH + 3 * dk) * sizeof(double));
    double* u = (double*)malloc((size_t)dk * sizeof(double));
    double* xs = (double*)malloc((size_t)(T > 0 ? T : 1) * dk * sizeof(double));  /* q*_t */
    double* es = (double*)malloc((size_t)(T > 0 ? T : 1) * dk * sizeof(double));  /* e*_t */
    double* ckH = (double*)malloc((size_t)(nblk > 0 ? nblk : 1) * nH * sizeof(double));
    double* ckG = (double*)malloc((size_t)(nblk > 0 ? nblk : 1) * nG * sizeof(double));
    double* bH = (double*)malloc((size_t)(BWD_BLOCK + 1) * nH * sizeof(double));
    double* bG = (double*)malloc((size_t)(BWD_BLOCK + 1) * nG * sizeof(double));
    double* DH = (double*)malloc((size_t)nH * sizeof(double));
    double* DG = (double*)malloc((size_t)nG * sizeof(double));
    j->status = 0;
    for (int64_t bh = j->tid; bh < j->B * j->Hh; bh += j->n_threads) {
        const int64_t h = bh % j->Hh;
        const double* lam = j->lambda + h * dk;
        double* dlam = j->dlam_part + bh * dk;
        memset(dlam, 0, (size_t)dk * sizeof(double));
        /* forward in time: states, q*_t, u_t = G_t^T e_t, e*_t; checkpoints of the
         * state entering every block */
        memset(H, 0, (size_t)nH * sizeof(double));
        memset(G, 0, (size_t)nG * sizeof(double));
        for (int64_t t = 0; t < T; ++t) {
            const int64_t tok = bh * T + t;
            if (t % BWD_BLOCK == 0) {
                memcpy(ckH + (t / BWD_BLOCK) * nH, H, (size_t)nH * sizeof(double));
                memcpy(ckG + (t / BWD_BLOCK) * nG, G, (size_t)nG * sizeof(double));
            }
            state_step(H, G, j->k + tok * dk, j->v + tok * dv, j->gamma[tok], j->beta[tok], dk, dv);
            for (int64_t a = 0; a < dk; ++a)
                for (int64_t b = 0; b < dk; ++b) A[a * dk + b] = H[a * dk + b] + (a == b ? lam[a] : 0.0);
            if (bwd_solve(j, A, j->q + tok * dk, xs + t * dk, sw) != 0) j->status = -1;
            const double* e = j->dout + tok * dv;
            for (int64_t b = 0; b < dk; ++b) {
                double acc = 0.0;
                for (int64_t a = 0; a < dv; ++a) acc += G[a * dk + b] * e[a];
                u[b] = acc;
            }
            if (bwd_solve(j, A, u, es + t * dk, sw) != 0) j->status = -1;
            for (int64_t a = 0; a < dk; ++a) {
                j->dq[tok * dk + a] = es[t * dk + a];
                dlam[a] -= xs[t * dk + a] * es[t * dk + a];
            }
            if (j->qstar) memcpy(j->qstar + tok * dk, xs + t * dk, (size_t)dk * sizeof(double));
            if (j->estar) memcpy(j->estar + tok * dk, es + t * dk, (size_t)dk * sizeof(double));
        }
        /* backward in time, block by block: recompute the block's states from its
         * checkpoint (bH[i] = state after token c0 + i - 1), then walk s downwards */
        memset(DH, 0, (size_t)nH * sizeof(double));
        memset(DG, 0, (size_t)nG * sizeof(double));
        double gamma_next = 0.0;  /* gamma_{s+1}; no token after the last */
        for (int64_t blk = nblk - 1; blk >= 0; --blk) {
            const int64_t c0 = blk * BWD_BLOCK;
            const int64_t c1 = c0 + BWD_BLOCK < T ? c0 + BWD_BLOCK : T;
            memcpy(bH, ckH + blk * nH, (size_t)nH * sizeof(double));
            memcpy(bG, ckG + blk * nG, (size_t)nG * sizeof(double));
            for (int64_t t = c0; t < c1; ++t) {
                const int64_t tok = bh * T + t, i = t - c0;
                memcpy(bH + (i + 1) * nH, bH + i * nH, (size_t)nH * sizeof(double));
                memcpy(bG + (i + 1) * nG, bG + i * nG, (size_t)nG * sizeof(double));
                state_step(bH + (i + 1) * nH, bG + (i + 1) * nG, j->k + tok * dk, j->v + tok * dv,
                           j->gamma[tok], j->beta[tok], dk, dv);
            }
            for (int64_t s = c1 - 1; s >= c0; --s) {
                const int64_t tok = bh * T + s, i = s - c0;
                const double* ks = j->k + tok * dk;
                const double* vs = j->v + tok * dv;
                const double* e = j->dout + tok * dv;
                const double* xq = xs + s * dk;
                const double* xe = es + s * dk;
                for (int64_t a = 0; a < dv; ++a)
                    for (int64_t b = 0; b < dk; ++b) DG[a * dk + b] = gamma_next * DG[a * dk + b] + e[a] * xq[b];
                for (int64_t a = 0; a < dk; ++a)
                    for (int64_t b = 0; b < dk; ++b) DH[a * dk + b] = gamma_next * DH[a * dk + b] - xe[a] * xq[b];
                const double beta = j->beta[tok];
                double db = 0.0, dg = 0.0;
                for (int64_t a = 0; a < dv; ++a) {
                    double s1 = 0.0;
                    for (int64_t b = 0; b < dk; ++b) s1 += DG[a * dk + b] * ks[b];
                    j->dv_out[tok * dv + a] = beta * s1;
                    db += vs[a] * s1;
                }
                for (int64_t b = 0; b < dk; ++b) {
                    double s1 = 0.0;
                    for (int64_t a = 0; a < dv; ++a) s1 += DG[a * dk + b] * vs[a];
                    for (int64_t a = 0; a < dk; ++a) s1 += (DH[b * dk + a] + DH[a * dk + b]) * ks[a];
                    j->dk_out[tok * dk + b] = beta * s1;
                }
                for (int64_t a = 0; a < dk; ++a) {
                    double s1 = 0.0;
                    for (int64_t b = 0; b < dk; ++b) s1 += DH[a * dk + b] * ks[b];
                    db += ks[a] * s1;
                }
                const double* Hp = bH + i * nH;  /* H_{s-1} */
                const double* Gp = bG + i * nG;  /* G_{s-1} */
                for (int64_t x = 0; x < nG; ++x) dg += DG[x] * Gp[x];
                for (int64_t x = 0; x < nH; ++x) dg += DH[x] * Hp[x];
                j->dbeta[tok] = db;
                j->dgamma[tok] = dg;
                gamma_next = j->gamma[tok];
            }
        }
    }
    free(H); free(G); free(A); free(sw); free(u); free(xs); free(es);
    free(ckH); free(ckG); free(bH); free(bG); free(DH); free(DG);
    return NULL;
}

/* Gradients of L with dL/do_t = dout_t [B,Hh,T,dv].  Inputs as oracle_forward;
 * outputs dq, dk [B,Hh,T,dk], dv [B,Hh,T,dv], dgamma, dbeta [B,Hh,T],
 * dlam_part [B*Hh, dk] (per-sequence sums; the caller sums over the batch);
 * qstar, estar [B,Hh,T,dk] may be NULL.  Returns 0, or -1 if a Cholesky solve
 * met a non-positive pivot. */
int oracle_backward(const double* q, const double* k, const double* v, const double* gamma,
                    const double* beta, const double* lambda, const double* dout, int64_t B,
                    int64_t Hh, int64_t T, int64_t dk, int64_t dv, int n_cg, int solver, int init,
                    double* dq, double* dk_out, double* dv_out, double* dgamma, double* dbeta,
                    double* dlam_part, double* qstar, double* estar, int n_threads)
{
    const int64_t units = B * Hh;
    if (n_threads < 1) n_threads = 1;
    if (n_threads > units) n_threads = (int)(units > 0 ? units : 1);
    oracle_bwd_job* jobs = (oracle_bwd_job*)malloc((size_t)n_threads * sizeof(oracle_bwd_job));
    pthread_t* th = (pthread_t*)malloc((size_t)n_threads * sizeof(pthread_t));
    for (int i = 0; i < n_threads; ++i) {
        oracle_bwd_job* j = &jobs[i];
        memset(j, 0, sizeof(*j));
        j->q = q; j->k = k; j->v = v; j->gamma = gamma; j->beta = beta; j->lambda = lambda;
        j->dout = dout; j->B = B; j->Hh = Hh; j->T = T; j->dk = dk; j->dv = dv;
        j->n_cg = n_cg; j->solver = solver; j->init = init;
        j->dq = dq; j->dk_out = dk_out; j->dv_out = dv_out; j->dgamma = dgamma; j->dbeta = dbeta;
        j->dlam_part = dlam_part; j->qstar = qstar; j->estar = estar;
        j->n_threads = n_threads; j->tid = i;
    }
    for (int i = 1; i < n_threads; ++i) pthread_create(&th[i], NULL, backward_worker, &jobs[i]);
    backward_worker(&jobs[0]);
    int status = jobs[0].status;
    for (int i = 1; i < n_threads; ++i) {
        pthread_join(th[i], NULL);
        if (jobs[i].status != 0) status = jobs[i].status;
    }
    free(jobs);
    free(th);
    return status;
}
