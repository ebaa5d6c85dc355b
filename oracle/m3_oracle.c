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
