/*
 * CPU oracle for the Mamba-3 SSM layer: the plain sequential recurrence in
 * fp64.  TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the CPU
 * baseline of the benchmark call it; the library never does.  It shares no
 * code, header or constant with the HIP path.
 *
 * What it computes, per (batch, head) slice, independently:
 *
 *   Exponential-trapezoidal step (Sec. 3.1, Prop. "Exponential-Trapezoidal
 *   Discretization", eq. mamba3-recurrence):
 *       alpha_t = exp(dt_t A_t)
 *       beta_t  = (1 - lambda_t) dt_t alpha_t        (current step's values)
 *       gamma_t = lambda_t dt_t
 *   Complex state as a real block-rotation (Sec. 3.2, Prop. "Complex-to-Real
 *   SSM Equivalence"; App. proof of the RoPE-trick/trapezoid proposition,
 *   eq. trap-real-rot): the previous state and the previous input term are
 *   both rotated by R_t, the current input term is not:
 *       h_t = alpha_t R_t h_{t-1} + beta_t R_t B_{t-1} X_{t-1}^T
 *             + gamma_t B_t X_t^T
 *   MIMO (Sec. 3.3 and App. "MIMO for Mamba-3"): B_t, C_t are N x R and
 *   X_t is P x R, so B X^T is an N x P matrix product, the output is
 *       Y_t = h_t^T C_t + D X_t                        (P x R)
 *   The D skip is a per-head scalar times X (not in the paper; the usual
 *   Mamba convention).
 *
 * Conventions (readings of the paper):
 *   - the N reals pair up as (i, i + N/2): the paper stacks [B; B_hat] and
 *     [C; -C_hat], real parts first.  R(phi) acts on (u_i, u_{i+N/2}) as
 *     [[cos, -sin], [sin, cos]].
 *   - theta[t][i] is the per-step angle (already Delta_t times the frequency).
 *   - h_{-1} = 0 and B_{-1} X_{-1}^T = 0 unless an initial state / carry is
 *     given (Sec. 3.1.2: the unrolled state starts from gamma_0 B_0 x_0).
 *
 * Layouts (all contiguous fp64, one slice after another):
 *   x [S][L][R][P], B and C [S][L][R][N], dt, A, lam [S][L],
 *   theta [S][L][N/2], D [S], state [S][N][P] (rows n, columns p),
 *   carryB [S][R][N], carryX [S][R][P], y [S][L][R][P].
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* One recurrence step on one slice, updating h, Bp, Xp in place. */
static void step_slice(int64_t N, int64_t P, int64_t R,
                       const double *X, const double *B, const double *C,
                       double dt, double A, double lam, const double *theta,
                       double D, double *h, double *Bp, double *Xp,
                       double *y, double *u)
{
    const int64_t H = N / 2;
    const double alpha = exp(dt * A);
    const double beta = (1.0 - lam) * dt * alpha;
    const double gamma = lam * dt;

    /* u = alpha h + beta Bp Xp^T  (both get rotated by R_t next) */
    for (int64_t n = 0; n < N; ++n)
        for (int64_t p = 0; p < P; ++p) {
            double s = 0.0;
            for (int64_t r = 0; r < R; ++r)
                s += Bp[r * N + n] * Xp[r * P + p];
            u[n * P + p] = alpha * h[n * P + p] + beta * s;
        }
    /* h = R_t u */
    for (int64_t i = 0; i < H; ++i) {
        const double c = cos(theta[i]), s = sin(theta[i]);
        for (int64_t p = 0; p < P; ++p) {
            const double re = u[i * P + p], im = u[(i + H) * P + p];
            h[i * P + p] = c * re - s * im;
            h[(i + H) * P + p] = s * re + c * im;
        }
    }
    /* h += gamma B X^T */
    for (int64_t n = 0; n < N; ++n)
        for (int64_t p = 0; p < P; ++p) {
            double s = 0.0;
            for (int64_t r = 0; r < R; ++r)
                s += B[r * N + n] * X[r * P + p];
            h[n * P + p] += gamma * s;
        }
    /* Y = h^T C + D X */
    for (int64_t r = 0; r < R; ++r)
        for (int64_t p = 0; p < P; ++p) {
            double s = 0.0;
            for (int64_t n = 0; n < N; ++n)
                s += h[n * P + p] * C[r * N + n];
            y[r * P + p] = s + D * X[r * P + p];
        }
    memcpy(Bp, B, sizeof(double) * (size_t)(R * N));
    memcpy(Xp, X, sizeof(double) * (size_t)(R * P));
}

/*
 * Full scan over S slices of length L.  init_state / init_B / init_X may be
 * NULL (zero).  state, carryB, carryX receive h_{L-1}, B_{L-1}, X_{L-1}
 * (or the initial values when L == 0).  nthreads <= 0 means the OpenMP
 * default.  Returns the number of threads used.
 */
int m3o_scan(int64_t S, int64_t L, int64_t N, int64_t P, int64_t R,
             const double *x, const double *B, const double *C,
             const double *dt, const double *A, const double *lam,
             const double *theta, const double *D,
             const double *init_state, const double *init_B,
             const double *init_X,
             double *y, double *state, double *carryB, double *carryX,
             int nthreads)
{
    int used = 1;
#ifdef _OPENMP
    if (nthreads <= 0) nthreads = omp_get_max_threads();
    #pragma omp parallel for schedule(dynamic, 1) num_threads(nthreads)
#endif
    for (int64_t s = 0; s < S; ++s) {
#ifdef _OPENMP
        if (s == 0) used = omp_get_num_threads();
#endif
        double *h = state + s * N * P;
        double *Bp = carryB + s * R * N;
        double *Xp = carryX + s * R * P;
        double *u = (double *)malloc(sizeof(double) * (size_t)(N * P));
        if (init_state) memcpy(h, init_state + s * N * P, sizeof(double) * (size_t)(N * P));
        else memset(h, 0, sizeof(double) * (size_t)(N * P));
        if (init_B) {
            memcpy(Bp, init_B + s * R * N, sizeof(double) * (size_t)(R * N));
            memcpy(Xp, init_X + s * R * P, sizeof(double) * (size_t)(R * P));
        } else {
            memset(Bp, 0, sizeof(double) * (size_t)(R * N));
            memset(Xp, 0, sizeof(double) * (size_t)(R * P));
        }
        for (int64_t t = 0; t < L; ++t) {
            const int64_t st = s * L + t;
            step_slice(N, P, R, x + st * R * P, B + st * R * N, C + st * R * N,
                       dt[st], A[st], lam[st], theta + st * (N / 2), D[s],
                       h, Bp, Xp, y + st * R * P, u);
        }
        free(u);
    }
    return used;
}

/* One decode step on S slices (state and carry updated in place). */
int m3o_step(int64_t S, int64_t N, int64_t P, int64_t R,
             double *state, double *carryB, double *carryX,
             const double *x, const double *B, const double *C,
             const double *dt, const double *A, const double *lam,
             const double *theta, const double *D, double *y, int nthreads)
{
    int used = 1;
#ifdef _OPENMP
    if (nthreads <= 0) nthreads = omp_get_max_threads();
    #pragma omp parallel for schedule(static) num_threads(nthreads)
#endif
    for (int64_t s = 0; s < S; ++s) {
#ifdef _OPENMP
        if (s == 0) used = omp_get_num_threads();
#endif
        double *u = (double *)malloc(sizeof(double) * (size_t)(N * P));
        step_slice(N, P, R, x + s * R * P, B + s * R * N, C + s * R * N,
                   dt[s], A[s], lam[s], theta + s * (N / 2), D[s],
                   state + s * N * P, carryB + s * R * N, carryX + s * R * P,
                   y + s * R * P, u);
        free(u);
    }
    return used;
}

/*
 * Reverse mode of the sequential recurrence (the gradient of a scalar loss
 * J(y, final state) with respect to every input), fp64, per slice:
 * the forward loop above is run once storing every state h_t, then the
 * chain rule is applied to each step in reverse order, from the step's own
 * definitions:
 *     alpha = exp(dt A), beta = (1 - lambda) dt alpha, gamma = lambda dt
 *     u   = alpha h_{t-1} + beta B_{t-1} X_{t-1}^T       (N x P)
 *     h_t = R(theta_t) u + gamma B_t X_t^T
 *     Y_t = h_t^T C_t + D X_t
 * With dh = dJ/dh_t (starting from dJ/dh_{L-1} = dfinal):
 *     dC_t = h_t dY_t,  dh += C_t dY_t^T,  dX_t += D dY_t,  dD += <X_t, dY_t>
 *     dgamma = <dh, B_t X_t^T>,  dB_t += gamma dh X_t,  dX_t += gamma dh^T B_t
 *     dtheta_t[i] = sum_p (dh[i+N/2][p] K[i][p] - dh[i][p] K[i+N/2][p]),  K = R(theta_t) u
 *     du = R(theta_t)^T dh
 *     dalpha = <du, h_{t-1}>,  dbeta = <du, B_{t-1} X_{t-1}^T>
 *     dB_{t-1} += beta du X_{t-1},  dX_{t-1} += beta du^T B_{t-1},  dJ/dh_{t-1} = alpha du
 *     then through alpha, beta, gamma to dt_t, A_t, lambda_t.
 * B_{-1} X_{-1}^T is zero (no initial carry); dinit = dJ/dh_{-1}.
 * Outputs have the layouts of the inputs: dx [S][L][R][P], dB and dC
 * [S][L][R][N], ddt, dA, dlam [S][L] (dA per token), dtheta [S][L][N/2],
 * dD [S], dinit [S][N][P] (may be NULL).  dy [S][L][R][P]; dfinal [S][N][P]
 * or NULL (zero).  Returns the number of threads used.
 */
int m3o_scan_bwd(int64_t S, int64_t L, int64_t N, int64_t P, int64_t R,
                 const double *x, const double *B, const double *C,
                 const double *dt, const double *A, const double *lam,
                 const double *theta, const double *D, const double *init_state,
                 const double *dy, const double *dfinal,
                 double *dx, double *dB, double *dC, double *ddt, double *dA,
                 double *dlam, double *dtheta, double *dD, double *dinit,
                 int nthreads)
{
    int used = 1;
    const int64_t H = N / 2, NP = N * P;
#ifdef _OPENMP
    if (nthreads <= 0) nthreads = omp_get_max_threads();
    #pragma omp parallel for schedule(dynamic, 1) num_threads(nthreads)
#endif
    for (int64_t s = 0; s < S; ++s) {
#ifdef _OPENMP
        if (s == 0) used = omp_get_num_threads();
#endif
        /* forward: hs[t+1] = h_t, hs[0] = h_{-1} */
        double *hs = (double *)malloc(sizeof(double) * (size_t)((L + 1) * NP));
        double *u = (double *)malloc(sizeof(double) * (size_t)NP);
        double *dh = (double *)malloc(sizeof(double) * (size_t)NP);
        double *du = (double *)malloc(sizeof(double) * (size_t)NP);
        double *Bp = (double *)calloc((size_t)(R * N), sizeof(double));
        double *Xp = (double *)calloc((size_t)(R * P), sizeof(double));
        double *yt = (double *)malloc(sizeof(double) * (size_t)(R * P));
        if (init_state) memcpy(hs, init_state + s * NP, sizeof(double) * (size_t)NP);
        else memset(hs, 0, sizeof(double) * (size_t)NP);
        for (int64_t t = 0; t < L; ++t) {
            const int64_t st = s * L + t;
            memcpy(hs + (t + 1) * NP, hs + t * NP, sizeof(double) * (size_t)NP);
            step_slice(N, P, R, x + st * R * P, B + st * R * N, C + st * R * N,
                       dt[st], A[st], lam[st], theta + st * H, D[s],
                       hs + (t + 1) * NP, Bp, Xp, yt, u);
        }
        /* reverse */
        if (dfinal) memcpy(dh, dfinal + s * NP, sizeof(double) * (size_t)NP);
        else memset(dh, 0, sizeof(double) * (size_t)NP);
        dD[s] = 0.0;
        memset(dx + s * L * R * P, 0, sizeof(double) * (size_t)(L * R * P));
        memset(dB + s * L * R * N, 0, sizeof(double) * (size_t)(L * R * N));
        for (int64_t t = L - 1; t >= 0; --t) {
            const int64_t st = s * L + t;
            const double *Xt = x + st * R * P, *Bt = B + st * R * N, *Ct = C + st * R * N;
            const double *dYt = dy + st * R * P;
            const double *ht = hs + (t + 1) * NP, *hm = hs + t * NP;
            const double *Bm1 = t > 0 ? B + (st - 1) * R * N : NULL;
            const double *Xm1 = t > 0 ? x + (st - 1) * R * P : NULL;
            double *dXt = dx + st * R * P, *dBt = dB + st * R * N, *dCt = dC + st * R * N;
            const double alpha = exp(dt[st] * A[st]);
            const double beta = (1.0 - lam[st]) * dt[st] * alpha;
            const double gamma = lam[st] * dt[st];
            /* output: Y = h^T C + D X */
            for (int64_t r = 0; r < R; ++r)
                for (int64_t n = 0; n < N; ++n) {
                    double v = 0.0;
                    for (int64_t p = 0; p < P; ++p) v += ht[n * P + p] * dYt[r * P + p];
                    dCt[r * N + n] = v;
                }
            for (int64_t n = 0; n < N; ++n)
                for (int64_t p = 0; p < P; ++p) {
                    double v = 0.0;
                    for (int64_t r = 0; r < R; ++r) v += Ct[r * N + n] * dYt[r * P + p];
                    dh[n * P + p] += v;
                }
            for (int64_t e = 0; e < R * P; ++e) {
                dXt[e] += D[s] * dYt[e];
                dD[s] += Xt[e] * dYt[e];
            }
            /* current input term gamma B_t X_t^T */
            double dgamma = 0.0;
            for (int64_t n = 0; n < N; ++n)
                for (int64_t p = 0; p < P; ++p) {
                    double bx = 0.0;
                    for (int64_t r = 0; r < R; ++r) bx += Bt[r * N + n] * Xt[r * P + p];
                    dgamma += dh[n * P + p] * bx;
                }
            for (int64_t r = 0; r < R; ++r) {
                for (int64_t n = 0; n < N; ++n) {
                    double v = 0.0;
                    for (int64_t p = 0; p < P; ++p) v += dh[n * P + p] * Xt[r * P + p];
                    dBt[r * N + n] += gamma * v;
                }
                for (int64_t p = 0; p < P; ++p) {
                    double v = 0.0;
                    for (int64_t n = 0; n < N; ++n) v += dh[n * P + p] * Bt[r * N + n];
                    dXt[r * P + p] += gamma * v;
                }
            }
            /* u = alpha h_{t-1} + beta B_{t-1} X_{t-1}^T, recomputed from its
               definition; K = R(theta) u; du = R^T dh */
            for (int64_t n = 0; n < N; ++n)
                for (int64_t p = 0; p < P; ++p) {
                    double bx = 0.0;
                    if (t > 0)
                        for (int64_t r = 0; r < R; ++r) bx += Bm1[r * N + n] * Xm1[r * P + p];
                    u[n * P + p] = alpha * hm[n * P + p] + beta * bx;
                }
            for (int64_t i = 0; i < H; ++i) {
                const double c = cos(theta[st * H + i]), sn = sin(theta[st * H + i]);
                double dth = 0.0;
                for (int64_t p = 0; p < P; ++p) {
                    const double ure = u[i * P + p], uim = u[(i + H) * P + p];
                    const double kre = c * ure - sn * uim, kim = sn * ure + c * uim;
                    const double gre = dh[i * P + p], gim = dh[(i + H) * P + p];
                    dth += gim * kre - gre * kim;
                    du[i * P + p] = c * gre + sn * gim;
                    du[(i + H) * P + p] = -sn * gre + c * gim;
                }
                dtheta[st * H + i] = dth;
            }
            /* u = alpha h_{t-1} + beta B_{t-1} X_{t-1}^T */
            double dalpha = 0.0, dbeta = 0.0;
            for (int64_t n = 0; n < NP; ++n) dalpha += du[n] * hm[n];
            if (t > 0) {
                for (int64_t n = 0; n < N; ++n)
                    for (int64_t p = 0; p < P; ++p) {
                        double bx = 0.0;
                        for (int64_t r = 0; r < R; ++r) bx += Bm1[r * N + n] * Xm1[r * P + p];
                        dbeta += du[n * P + p] * bx;
                    }
                double *dBm1 = dB + (st - 1) * R * N, *dXm1 = dx + (st - 1) * R * P;
                for (int64_t r = 0; r < R; ++r) {
                    for (int64_t n = 0; n < N; ++n) {
                        double v = 0.0;
                        for (int64_t p = 0; p < P; ++p) v += du[n * P + p] * Xm1[r * P + p];
                        dBm1[r * N + n] += beta * v;
                    }
                    for (int64_t p = 0; p < P; ++p) {
                        double v = 0.0;
                        for (int64_t n = 0; n < N; ++n) v += du[n * P + p] * Bm1[r * N + n];
                        dXm1[r * P + p] += beta * v;
                    }
                }
            }
            for (int64_t n = 0; n < NP; ++n) dh[n] = alpha * du[n];
            /* scalars: beta = (1 - lam) dt alpha, gamma = lam dt, alpha = exp(dt A) */
            const double dal = dalpha + dbeta * (1.0 - lam[st]) * dt[st];
            ddt[st] = dal * alpha * A[st] + dbeta * (1.0 - lam[st]) * alpha + dgamma * lam[st];
            dA[st] = dal * alpha * dt[st];
            dlam[st] = -dbeta * dt[st] * alpha + dgamma * dt[st];
        }
        if (dinit) memcpy(dinit + s * NP, dh, sizeof(double) * (size_t)NP);
        free(hs); free(u); free(dh); free(du); free(Bp); free(Xp); free(yt);
    }
    return used;
}
