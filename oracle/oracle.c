/*
 * Float64 CPU oracle for the FlashConv hot path of "Hungry Hungry Hippos"
 * (Fu, Dao et al., arXiv 2212.14052).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product library links, loads or
 * calls this file; only the test-suite, the smoke check and the CPU-baseline
 * leg of the benchmark do.  It shares no code, header or table with the HIP
 * path.
 *
 * Every routine is the plain definition of what the fast path computes,
 * written for clarity, not speed:
 *   - ZOH discretisation of a diagonal SSM,
 *   - the SSM convolution kernel f = [CB, CAB, CA^2B, ...]     (Sec. 2.1),
 *   - the direct O(L^2) causal convolution y = f * u + D u     (Sec. 2.1),
 *     and its gradients du, df, dD by their definitions (backward-pass
 *     appendix),
 *   - the explicit recurrence x_i = A x_{i-1} + B u_i,
 *     y_i = C x_i + D u_i                                       (Sec. 2.1),
 *   - the state-passing algorithm (Sec. 4.2, Algorithm 2), used only to pin
 *     the oracle against Proposition 2,
 *   - the shift SSM (Sec. 3.2), evaluated as the literal shift-matrix
 *     recurrence.
 *
 * Conventions (float64 throughout, complex values as interleaved re/im):
 *   - a diagonal SSM has m complex modes per channel; its real output is
 *     y_t = 2 Re(sum_n C_n x_{t,n}) + D u_t, i.e. each complex mode stands for
 *     a conjugate pair of real modes, so the impulse response of the
 *     recurrence is exactly k_t = 2 Re sum_n C_n Bbar_n Abar_n^t (+ D at t=0);
 *   - rows are (batch, channel) pairs, row r = b*H + h, contiguous length L;
 *   - the state after input t is x_t; x_{-1} = x0 (the initial condition).
 */
#include <complex.h>
#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

typedef double complex cplx;

static inline cplx ld(const double *p, long i) { return p[2 * i] + I * p[2 * i + 1]; }
static inline void st(double *p, long i, cplx v) { p[2 * i] = creal(v); p[2 * i + 1] = cimag(v); }

/*
 * Zero-order-hold discretisation of the diagonal continuous-time SSM
 * x' = A x + B u (Sec. 2.1): with the input held constant over one step dt,
 * Abar = exp(dt A), Bbar = A^{-1} (exp(dt A) - 1) B, elementwise per mode.
 * A, B, Abar, Bbar: (H, m) complex.  dt: (H).
 */
void oracle_zoh(const double *A, const double *B, const double *dt, int H, int m,
                double *Abar, double *Bbar)
{
    for (int h = 0; h < H; ++h)
        for (int n = 0; n < m; ++n) {
            long i = (long)h * m + n;
            cplx a = ld(A, i), b = ld(B, i);
            cplx e = cexp(dt[h] * a);
            st(Abar, i, e);
            st(Bbar, i, (e - 1.0) / a * b);
        }
}

/*
 * SSM convolution kernel of a diagonal SSM given in discrete form (Sec. 2.1:
 * f = [CB, CAB, CA^2B, ...]):  k[h,t] = 2 Re sum_n C[h,n] Bbar[h,n] Abar[h,n]^t.
 * Each power is evaluated directly as exp(t log Abar), not by repeated
 * multiplication.  k: (H, L).
 */
void oracle_ssm_kernel_discrete(const double *Abar, const double *Bbar, const double *C,
                                int H, int m, int L, double *k)
{
#pragma omp parallel for schedule(static)
    for (int h = 0; h < H; ++h)
        for (int t = 0; t < L; ++t) {
            cplx s = 0;
            for (int n = 0; n < m; ++n) {
                long i = (long)h * m + n;
                cplx p = cexp((double)t * clog(ld(Abar, i)));
                s += ld(C, i) * ld(Bbar, i) * p;
            }
            k[(long)h * L + t] = 2.0 * creal(s);
        }
}

/*
 * The same kernel from the continuous parameters, with the ZOH step folded
 * in: Abar^t = exp(t dt A), so k[h,t] = 2 Re sum_n C Bbar exp(t dt_h A_n).
 */
void oracle_ssm_kernel(const double *A, const double *B, const double *C, const double *dt,
                       int H, int m, int L, double *k)
{
#pragma omp parallel for schedule(static)
    for (int h = 0; h < H; ++h) {
        for (int t = 0; t < L; ++t) {
            cplx s = 0;
            for (int n = 0; n < m; ++n) {
                long i = (long)h * m + n;
                cplx a = ld(A, i);
                cplx bbar = (cexp(dt[h] * a) - 1.0) / a * ld(B, i);
                s += ld(C, i) * bbar * cexp((double)t * dt[h] * a);
            }
            k[(long)h * L + t] = 2.0 * creal(s);
        }
    }
}

/*
 * Direct causal (linear, not circular) convolution plus skip term (Sec. 2.1,
 * "y = f * u + D u"):  y[r,t] = sum_{j=0}^{t} k[h,j] u[r,t-j] + D[h] u[r,t],
 * with h = r mod H.  The sum includes j = t (the current input meets f_0 = CB).
 * u, y: (R, L) with R = B*H; k: (H, L); D: (H) or NULL (no skip).
 */
void oracle_causal_conv(const double *u, const double *k, const double *D,
                        int R, int H, int L, double *y)
{
#pragma omp parallel for schedule(dynamic, 1)
    for (int r = 0; r < R; ++r) {
        int h = r % H;
        const double *ur = u + (long)r * L;
        const double *kh = k + (long)h * L;
        double *yr = y + (long)r * L;
        for (int t = 0; t < L; ++t) {
            double s = 0.0;
            for (int j = 0; j <= t; ++j) s += kh[j] * ur[t - j];
            if (D) s += D[h] * ur[t];
            yr[t] = s;
        }
    }
}

/*
 * Gradients of the causal convolution y = f * u + D u (the backward pass of
 * the appendix on FlashConv's backward), by their definitions: for a loss
 * with output gradient dy,
 *   du[r,t] = sum_{s=t}^{L-1} k[h,s-t] dy[r,s] + D[h] dy[r,t],
 *   dk[h,j] = sum_{b} sum_{t=j}^{L-1} dy[b,h,t] u[b,h,t-j],
 *   dD[h]   = sum_{b} sum_{t} dy[b,h,t] u[b,h,t],
 * with rows r = b*H + h, R = B*H.  D may be NULL (no skip term in du); each
 * of du, dk, dD may be NULL (not computed).
 */
void oracle_causal_conv_bwd(const double *u, const double *k, const double *D, const double *dy,
                            int R, int H, int L, double *du, double *dk, double *dD)
{
    const int B = R / H;
    if (du) {
#pragma omp parallel for schedule(dynamic, 1)
        for (int r = 0; r < R; ++r) {
            int h = r % H;
            const double *kh = k + (long)h * L, *g = dy + (long)r * L;
            for (int t = 0; t < L; ++t) {
                double s = 0.0;
                for (int q = t; q < L; ++q) s += kh[q - t] * g[q];
                if (D) s += D[h] * g[t];
                du[(long)r * L + t] = s;
            }
        }
    }
    if (dk || dD) {
#pragma omp parallel for schedule(dynamic, 1)
        for (int h = 0; h < H; ++h) {
            for (int j = 0; j < L; ++j) {
                if (!dk && j > 0) break;
                double s = 0.0;
                for (int b = 0; b < B; ++b) {
                    const double *ur = u + ((long)b * H + h) * L, *g = dy + ((long)b * H + h) * L;
                    for (int t = j; t < L; ++t) s += g[t] * ur[t - j];
                }
                if (dk) dk[(long)h * L + j] = s;
                if (j == 0 && dD) dD[h] = s;
            }
        }
    }
}

/*
 * Explicit recurrence of the diagonal SSM (Sec. 2.1, discrete form):
 *   x_t = Abar x_{t-1} + Bbar u_t,   y_t = 2 Re(C . x_t) + D u_t,
 * with x_{-1} = x0 (NULL: zero).  Modes are independent, so "Abar x" is the
 * elementwise product.  u, y: (R, L); Abar, Bbar, C: (H, m) complex; D: (H) or NULL (no skip);
 * x0, x_final: (R, m) complex (x_final = x_{L-1}; may be NULL).
 */
void oracle_ssm_recurrence(const double *u, const double *Abar, const double *Bbar,
                           const double *C, const double *D, const double *x0,
                           int R, int H, int L, int m, double *y, double *x_final)
{
#pragma omp parallel for schedule(dynamic, 1)
    for (int r = 0; r < R; ++r) {
        int h = r % H;
        cplx *x = (cplx *)malloc(sizeof(cplx) * (size_t)m);
        for (int n = 0; n < m; ++n) x[n] = x0 ? ld(x0, (long)r * m + n) : 0;
        for (int t = 0; t < L; ++t) {
            double ut = u[(long)r * L + t];
            cplx s = 0;
            for (int n = 0; n < m; ++n) {
                long i = (long)h * m + n;
                x[n] = ld(Abar, i) * x[n] + ld(Bbar, i) * ut;
                s += ld(C, i) * x[n];
            }
            y[(long)r * L + t] = 2.0 * creal(s) + (D ? D[h] * ut : 0.0);
        }
        if (x_final)
            for (int n = 0; n < m; ++n) st(x_final, (long)r * m + n, x[n]);
        free(x);
    }
}

/*
 * State-passing algorithm (Sec. 4.2, Algorithm 2), batched over rows.
 * The sequence is split into C = L/N' chunks.  With the state carried into a
 * chunk written x (the state after the previous chunk's last input):
 *   precompute  A^{N'};  M_ux[n,i] = Abar_n^{N'-1-i} Bbar_n;
 *               M_xy[t,n] = C_n Abar_n^{t+1}     (t, i = 0..N'-1),
 *   per chunk:  y^(c) = 2 Re(M_xy x) + f * u^(c) + D u^(c),
 *               x     = A^{N'} x + M_ux u^(c),
 * where f is the length-N' SSM kernel and "f * u^(c)" is the direct causal
 * convolution of the chunk (oracle_causal_conv on one row).  The exponent t+1
 * in M_xy and N'-1-i in M_ux are the 0-indexed forms that make the result
 * equal to the recurrence (Proposition 2).
 * Shapes as oracle_ssm_recurrence; chunk must divide L.
 */
void oracle_statepass(const double *u, const double *Abar, const double *Bbar,
                      const double *C, const double *D, const double *x0,
                      int R, int H, int L, int m, int chunk, double *y, double *x_final)
{
    int nc = L / chunk;
    double *f = (double *)malloc(sizeof(double) * (size_t)H * chunk);
    oracle_ssm_kernel_discrete(Abar, Bbar, C, H, m, chunk, f);
#pragma omp parallel for schedule(dynamic, 1)
    for (int r = 0; r < R; ++r) {
        int h = r % H;
        cplx *x = (cplx *)malloc(sizeof(cplx) * (size_t)m);
        cplx *AN = (cplx *)malloc(sizeof(cplx) * (size_t)m);
        cplx *Mux = (cplx *)malloc(sizeof(cplx) * (size_t)m * chunk);
        cplx *Mxy = (cplx *)malloc(sizeof(cplx) * (size_t)m * chunk);
        double *conv = (double *)malloc(sizeof(double) * (size_t)chunk);
        for (int n = 0; n < m; ++n) {
            long i = (long)h * m + n;
            cplx la = clog(ld(Abar, i));
            AN[n] = cexp((double)chunk * la);
            for (int t = 0; t < chunk; ++t) {
                Mux[(long)n * chunk + t] = cexp((double)(chunk - 1 - t) * la) * ld(Bbar, i);
                Mxy[(long)n * chunk + t] = ld(C, i) * cexp((double)(t + 1) * la);
            }
            x[n] = x0 ? ld(x0, (long)r * m + n) : 0;
        }
        for (int c = 0; c < nc; ++c) {
            const double *uc = u + (long)r * L + (long)c * chunk;
            double *yc = y + (long)r * L + (long)c * chunk;
            oracle_causal_conv(uc, f + (long)h * chunk, NULL, 1, 1, chunk, conv);
            for (int t = 0; t < chunk; ++t) {
                cplx s = 0;
                for (int n = 0; n < m; ++n) s += Mxy[(long)n * chunk + t] * x[n];
                yc[t] = 2.0 * creal(s) + conv[t] + (D ? D[h] * uc[t] : 0.0);
            }
            for (int n = 0; n < m; ++n) {
                cplx s = 0;
                for (int t = 0; t < chunk; ++t) s += Mux[(long)n * chunk + t] * uc[t];
                x[n] = AN[n] * x[n] + s;
            }
        }
        if (x_final)
            for (int n = 0; n < m; ++n) st(x_final, (long)r * m + n, x[n]);
        free(x); free(AN); free(Mux); free(Mxy); free(conv);
    }
    free(f);
}

/*
 * Shift SSM (Sec. 3.2): A is the m x m down-shift matrix (A[i][j] = 1 iff
 * i - 1 = j), B = e_1, so the state is updated as x_t = [u_t, x_{t-1}[0..m-2]]
 * and y_t = Cs . x_t + Ds u_t.  Evaluated literally as that recurrence.
 * u, y: (R, L); Cs: (H, m) real; Ds: (H) or NULL.
 */
void oracle_shift_ssm(const double *u, const double *Cs, const double *Ds,
                      int R, int H, int L, int m, double *y)
{
#pragma omp parallel for schedule(dynamic, 1)
    for (int r = 0; r < R; ++r) {
        int h = r % H;
        double *x = (double *)calloc((size_t)m, sizeof(double));
        for (int t = 0; t < L; ++t) {
            for (int i = m - 1; i > 0; --i) x[i] = x[i - 1];   /* x <- A x   */
            x[0] = u[(long)r * L + t];                           /*   + B u_t  */
            double s = 0.0;
            for (int i = 0; i < m; ++i) s += Cs[(long)h * m + i] * x[i];
            if (Ds) s += Ds[h] * u[(long)r * L + t];
            y[(long)r * L + t] = s;
        }
        free(x);
    }
}

/* Number of OpenMP threads the oracle runs with (for the CPU-baseline report). */
int oracle_num_threads(void)
{
    int n = 1;
#ifdef _OPENMP
#pragma omp parallel
    {
#pragma omp single
        n = omp_get_num_threads();
    }
#endif
    return n;
}
