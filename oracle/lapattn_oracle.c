/*
 * lapattn_oracle.c -- plain fp64 reference of Nystrom-approximated Laplacian-kernel
 * attention, forward and backward.
 *
 * TEST INFRASTRUCTURE ONLY (see lapattn_oracle.h).  Plain loops in the order the
 * paper states the method; OpenMP only splits independent output rows across
 * threads, every sum runs sequentially in index order.  No blocking, no fusion.
 *
 * What each step follows:
 *   kernel             k(x,y) = exp(-||x-y||_1/lambda)            Sec. 1, Sec. 4.1, Eq. (8)
 *   landmarks          segment means of consecutive tokens        Sec. 4.2 "Sampling strategies" (R5),
 *                      or means of r x r windows of the H' x W' token map (average
 *                      pooling with kernel r and stride r, the same passage)
 *   K_LL, K_QL, K_LK   Algorithm 1 (kernel on sampled points, cross-kernel),
 *                      in the orientation K_QL * X * K_LK           (R1)
 *   Newton-Schulz      Algorithm 2: W += eps*I, X0 = W^T/c, X <- X(2I - W X)
 *                      with c = ||W||_1 ||W||_inf                  (R2, R3, R9, R10)
 *   key summary        sum_j phi(k_j)^T v_j and sum_j phi(k_j)^T   Sec. 3.2, Eq. (3)
 *   normalisation      z_ij = g_ij - mean_j' g_ij' + 1/n           Eq. (4) with Sigma^{-1/2} = I (R4)
 *   m-space option     z_il = w_l (a_il - mean_l' a_il') + 1/m,   Appendix B, Eq. (13) with the
 *                      Out_i = z_i^T M[:, :d]                     offline diagonal w (R15)
 *   output             Z V                                        Eq. (7)
 *   DWC(V)             the depth-wise convolution term of Eq. (7)  (R14), a separate
 *                      function: the caller adds it to Z V
 *   backward           chain rule through all of the above; kernel gradient
 *                      dk/dx = -(1/lambda) sign(x-y) k            App. A (R8), the sign
 *                      decided with the landmark mean y rounded to fp32 (R16)
 */
#include "lapattn_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

int lapattn_oracle_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

static double sgn(double x) { return (double)((x > 0) - (x < 0)); }

/* R16: the backward decides sign(x - y) of the kernel gradient (App. A) with the landmark
 * mean y rounded to fp32, the precision in which the kernels hold the landmarks (the paper
 * fixes none).  The sign is a decision taken by floating point: where a token coordinate lies
 * within the rounding of a landmark mean, the two choices are the two one-sided derivatives,
 * and both sides must take the same one.  Every other step stays in fp64. */
static double lm32(double y) { return (double)(float)y; }

double lapattn_oracle_kernel(const double* x, const double* y, int d, double lambda) {
    double dist = 0.0;
    for (int c = 0; c < d; ++c) dist += fabs(x[c] - y[c]);
    return exp(-dist / lambda);
}

int lapattn_oracle_segments(int n, int m, int* starts) {
    if (n < 1 || m < 1 || m > n) return 1;
    for (int l = 0; l <= m; ++l) starts[l] = (int)(((long long)l * n) / m);
    return 0;
}

int lapattn_oracle_windows(int n, int m, int grid_w, int r, int* starts, int* members) {
    if (grid_w == 0 && r == 0) {
        if (lapattn_oracle_segments(n, m, starts)) return 1;
        for (int i = 0; i < n; ++i) members[i] = i;
        return 0;
    }
    /* tokens in row-major order on an H' x W' map, W' = grid_w; r must divide H' and W' */
    if (grid_w < 1 || r < 1 || n % grid_w) return 1;
    const int hp = n / grid_w;
    if (hp % r || grid_w % r || m != (hp / r) * (grid_w / r)) return 1;
    const int mw = grid_w / r;
    for (int l = 0; l < m; ++l) {
        const int wy = l / mw, wx = l % mw;
        starts[l] = l * r * r;
        for (int t = 0; t < r * r; ++t) members[l * r * r + t] = (wy * r + t / r) * grid_w + wx * r + t % r;
    }
    starts[m] = m * r * r;
    return 0;
}

/* C = A * B for m x p times p x q, all row-major. */
static void matmul(const double* A, const double* Bm, double* C, int m, int p, int q) {
    for (int i = 0; i < m; ++i)
        for (int j = 0; j < q; ++j) {
            double s = 0.0;
            for (int k = 0; k < p; ++k) s += A[i * p + k] * Bm[k * q + j];
            C[i * q + j] = s;
        }
}

static void transpose(const double* A, double* At, int m, int q) {
    for (int i = 0; i < m; ++i)
        for (int j = 0; j < q; ++j) At[j * m + i] = A[i * q + j];
}

/* Induced norms of Algorithm 2's start (R2): ||W||_1 = max column abs-sum,
 * ||W||_inf = max row abs-sum.  Also report the first maximising column/row. */
static void induced_norms(const double* W, int m, double* n1, int* bstar, double* ninf, int* astar) {
    *n1 = -1.0; *ninf = -1.0; *bstar = 0; *astar = 0;
    for (int b = 0; b < m; ++b) {
        double s = 0.0;
        for (int a = 0; a < m; ++a) s += fabs(W[a * m + b]);
        if (s > *n1) { *n1 = s; *bstar = b; }
    }
    for (int a = 0; a < m; ++a) {
        double s = 0.0;
        for (int b = 0; b < m; ++b) s += fabs(W[a * m + b]);
        if (s > *ninf) { *ninf = s; *astar = a; }
    }
}

double lapattn_oracle_ns(const double* W_in, int m, int T, double eps, double* Xs) {
    size_t mm = (size_t)m * m;
    double* W = (double*)malloc(mm * sizeof(double));
    double* WX = (double*)malloc(mm * sizeof(double));
    memcpy(W, W_in, mm * sizeof(double));
    /* Algorithm 2: W <- W + eps I */
    for (int a = 0; a < m; ++a) W[a * m + a] += eps;
    double n1, ninf; int bs, as;
    induced_norms(W, m, &n1, &bs, &ninf, &as);
    double c = n1 * ninf;
    if (c == 0.0) {
        /* R10: the start scale vanishes only for W = 0, whose pseudoinverse is 0. */
        memset(Xs, 0, (size_t)(T + 1) * mm * sizeof(double));
    } else {
        /* X0 = W^T / c */
        for (int a = 0; a < m; ++a)
            for (int b = 0; b < m; ++b) Xs[a * m + b] = W[b * m + a] / c;
        /* X_{t+1} = X_t (2I - W X_t) */
        for (int t = 0; t < T; ++t) {
            const double* X = Xs + (size_t)t * mm;
            double* Xn = Xs + (size_t)(t + 1) * mm;
            matmul(W, X, WX, m, m, m);
            for (int a = 0; a < m; ++a)
                for (int b = 0; b < m; ++b) WX[a * m + b] = (a == b ? 2.0 : 0.0) - WX[a * m + b];
            matmul(X, WX, Xn, m, m, m);
        }
    }
    free(W); free(WX);
    return c;
}

/* Everything one head's forward produces; the backward reuses it. */
typedef struct {
    int n, d, m, T, dv;            /* dv = d + 1: values with the ones column */
    int* starts;                   /* m + 1: landmark l averages members[starts[l] .. starts[l+1]) */
    int* members;                  /* n token indices, grouped by landmark */
    double *qt, *kt;               /* m x d */
    double *Wk;                    /* m x m, kernel part plus eps on the diagonal */
    double *Xs;                    /* (T+1) x m x m */
    double c;                      /* X0 scale */
    double *Bm;                    /* m x n   K_LK */
    double *U;                     /* m x dv  K_LK [V|1] */
    double *M;                     /* m x dv  X_T U */
    double *A;                     /* n x m   K_QL */
    double *Y;                     /* n x dv  K_QL M */
    double *vbar;                  /* d */
} head_state;

static void head_alloc(head_state* s, int n, int d, int m, int T, int grid_w, int r) {
    s->n = n; s->d = d; s->m = m; s->T = T; s->dv = d + 1;
    s->starts = (int*)malloc((size_t)(m + 1) * sizeof(int));
    s->members = (int*)malloc((size_t)n * sizeof(int));
    lapattn_oracle_windows(n, m, grid_w, r, s->starts, s->members);   /* validated by the caller */
    s->qt = (double*)malloc((size_t)m * d * sizeof(double));
    s->kt = (double*)malloc((size_t)m * d * sizeof(double));
    s->Wk = (double*)malloc((size_t)m * m * sizeof(double));
    s->Xs = (double*)malloc((size_t)(T + 1) * m * m * sizeof(double));
    s->Bm = (double*)malloc((size_t)m * n * sizeof(double));
    s->U = (double*)malloc((size_t)m * (d + 1) * sizeof(double));
    s->M = (double*)malloc((size_t)m * (d + 1) * sizeof(double));
    s->A = (double*)malloc((size_t)n * m * sizeof(double));
    s->Y = (double*)malloc((size_t)n * (d + 1) * sizeof(double));
    s->vbar = (double*)malloc((size_t)d * sizeof(double));
}

static void head_free(head_state* s) {
    free(s->starts); free(s->members); free(s->qt); free(s->kt); free(s->Wk); free(s->Xs); free(s->Bm);
    free(s->U); free(s->M); free(s->A); free(s->Y); free(s->vbar);
}

/* One head of the forward: q, k, v are n x d; out is n x d. */
static void head_forward(const double* q, const double* k, const double* v, double* out,
                         double lambda, int norm, double eps, const double* wl, head_state* s) {
    const int n = s->n, d = s->d, m = s->m, T = s->T, dv = s->dv;

    /* Landmarks (R5): means of the balanced segments [floor(l n/m), floor((l+1) n/m)), or of
     * the r x r windows of the token map (Sec. 4.2), members in window row-major order. */
    for (int l = 0; l < m; ++l) {
        int a0 = s->starts[l], a1 = s->starts[l + 1];
        for (int c = 0; c < d; ++c) {
            double sq = 0.0, sk = 0.0;
            for (int t = a0; t < a1; ++t) {
                const int i = s->members[t];
                sq += q[(size_t)i * d + c];
                sk += k[(size_t)i * d + c];
            }
            s->qt[l * d + c] = sq / (a1 - a0);
            s->kt[l * d + c] = sk / (a1 - a0);
        }
    }

    /* Algorithm 1, kernel matrix on the sampled points: K_LL[a][b] = k(qt_a, kt_b) (R1). */
    for (int a = 0; a < m; ++a)
        for (int b = 0; b < m; ++b)
            s->Wk[a * m + b] = lapattn_oracle_kernel(s->qt + a * d, s->kt + b * d, d, lambda);

    /* Algorithm 2. */
    s->c = lapattn_oracle_ns(s->Wk, m, T, eps, s->Xs);
    for (int a = 0; a < m; ++a) s->Wk[a * m + a] += eps;

    /* Key-side summary: K_LK[a][j] = k(qt_a, k_j), U = K_LK [V | 1]. */
#pragma omp parallel for schedule(static)
    for (int a = 0; a < m; ++a) {
        for (int j = 0; j < n; ++j)
            s->Bm[(size_t)a * n + j] = lapattn_oracle_kernel(s->qt + a * d, k + (size_t)j * d, d, lambda);
        for (int c = 0; c < dv; ++c) {
            double acc = 0.0;
            for (int j = 0; j < n; ++j)
                acc += s->Bm[(size_t)a * n + j] * (c < d ? v[(size_t)j * d + c] : 1.0);
            s->U[a * dv + c] = acc;
        }
    }

    /* M = X_T U. */
    matmul(s->Xs + (size_t)T * m * m, s->U, s->M, m, m, dv);

    /* vbar = mean_j v_j. */
    for (int c = 0; c < d; ++c) {
        double acc = 0.0;
        for (int j = 0; j < n; ++j) acc += v[(size_t)j * d + c];
        s->vbar[c] = acc / n;
    }

    /* Query side: K_QL[i][l] = k(q_i, kt_l) (Eq. (8)), Y = K_QL M, then the
     * normalisation.  Y[i][d] = (G^ 1)_i = s_i. */
#pragma omp parallel for schedule(static)
    for (int i = 0; i < n; ++i) {
        for (int l = 0; l < m; ++l)
            s->A[(size_t)i * m + l] = lapattn_oracle_kernel(q + (size_t)i * d, s->kt + l * d, d, lambda);
        for (int c = 0; c < dv; ++c) {
            double acc = 0.0;
            for (int l = 0; l < m; ++l) acc += s->A[(size_t)i * m + l] * s->M[l * dv + c];
            s->Y[(size_t)i * dv + c] = acc;
        }
        double si = s->Y[(size_t)i * dv + d];
        if (norm == ORACLE_NORM_MSPACE) {
            /* Appendix B: the query's landmark kernel vector a_i, centred by its mean over the
             * landmarks, whitened by the diagonal w, plus 1/m; it weights the rows of M. */
            double abar = 0.0;
            for (int l = 0; l < m; ++l) abar += s->A[(size_t)i * m + l];
            abar /= m;
            for (int c = 0; c < d; ++c) {
                double o = 0.0;
                for (int l = 0; l < m; ++l) {
                    const double z = (wl ? wl[l] : 1.0) * (s->A[(size_t)i * m + l] - abar) + 1.0 / m;
                    o += z * s->M[l * dv + c];
                }
                out[(size_t)i * d + c] = o;
            }
            continue;
        }
        for (int c = 0; c < d; ++c) {
            double y = s->Y[(size_t)i * dv + c];
            double o;
            if (norm == ORACLE_NORM_INLINE)
                /* sum_j z_ij v_j with z_ij = g_ij - s_i/n + 1/n (Eq. (4), R4) */
                o = y + (1.0 - si) * s->vbar[c];
            else if (norm == ORACLE_NORM_ROWSUM)
                /* Eq. (3): numerator over denominator */
                o = y / si;
            else
                o = y;
            out[(size_t)i * d + c] = o;
        }
    }
}

static int check_args(int B, int H, int n, int d, int m, double lambda, int T, int norm) {
    if (B < 1 || H < 1 || n < 1 || d < 1 || m < 1 || m > n) return 2;
    if (!(lambda > 0.0) || !isfinite(lambda)) return 3;
    if (T < 0) return 3;
    if (norm < 0 || norm > 3) return 3;
    return 0;
}

static int check_windows(int n, int m, int grid_w, int r) {
    int* st = (int*)malloc((size_t)(m + 1) * sizeof(int));
    int* mem = (int*)malloc((size_t)n * sizeof(int));
    const int rc = lapattn_oracle_windows(n, m, grid_w, r, st, mem);
    free(st); free(mem);
    return rc ? 4 : 0;
}

int lapattn_oracle_forward(const double* Q, const double* K, const double* V, double* Out,
                           int B, int H, int n, int d, int m, double lambda, int T,
                           int norm, double eps, int grid_w, int r,
                           double* Qt, double* Kt, double* Wk, double* Xs,
                           double* U, double* M, double* Y, double* vbar, const double* whiten) {
    if (!Q || !K || !V || !Out) return 1;
    int rc = check_args(B, H, n, d, m, lambda, T, norm);
    if (rc) return rc;
    if ((rc = check_windows(n, m, grid_w, r))) return rc;
    const int BH = B * H, dv = d + 1;
    const size_t hs = (size_t)n * d;
    for (int h = 0; h < BH; ++h) {
        head_state s;
        head_alloc(&s, n, d, m, T, grid_w, r);
        const double* wl = whiten ? whiten + (size_t)(h % H) * m : NULL;
        head_forward(Q + h * hs, K + h * hs, V + h * hs, Out + h * hs, lambda, norm, eps, wl, &s);
        if (Qt) memcpy(Qt + (size_t)h * m * d, s.qt, (size_t)m * d * sizeof(double));
        if (Kt) memcpy(Kt + (size_t)h * m * d, s.kt, (size_t)m * d * sizeof(double));
        if (Wk) memcpy(Wk + (size_t)h * m * m, s.Wk, (size_t)m * m * sizeof(double));
        if (Xs) memcpy(Xs + (size_t)h * (T + 1) * m * m, s.Xs, (size_t)(T + 1) * m * m * sizeof(double));
        if (U) memcpy(U + (size_t)h * m * dv, s.U, (size_t)m * dv * sizeof(double));
        if (M) memcpy(M + (size_t)h * m * dv, s.M, (size_t)m * dv * sizeof(double));
        if (Y) memcpy(Y + (size_t)h * n * dv, s.Y, (size_t)n * dv * sizeof(double));
        if (vbar) memcpy(vbar + (size_t)h * d, s.vbar, (size_t)d * sizeof(double));
        head_free(&s);
    }
    return 0;
}

/* Reverse mode through Algorithm 2.  G holds dL/dX_T on entry; on exit dW holds
 * dL/dW (W including eps on the diagonal, whose gradient equals that of the
 * kernel matrix).  X_{t+1} = 2 X_t - X_t W X_t gives
 *   dW   -= X_t^T G X_t^T
 *   dX_t  = 2 G - G X_t^T W^T - W^T X_t^T G
 * and X0 = W^T / c with c = ||W||_1 ||W||_inf gives
 *   dW  += G0^T / c  -  (<G0, W^T> / c^2) * dc/dW,
 *   dc/dW[a][b] = ||W||_inf sign(W[a][b]) [b = b*] + ||W||_1 sign(W[a][b]) [a = a*]. */
static void ns_backward(const head_state* s, const double* Gin, double* dW) {
    const int m = s->m, T = s->T;
    const size_t mm = (size_t)m * m;
    memset(dW, 0, mm * sizeof(double));
    if (s->c == 0.0) return;  /* R10: X does not depend on W there */
    double* G = (double*)malloc(mm * sizeof(double));
    double* Xt = (double*)malloc(mm * sizeof(double));
    double* Wt = (double*)malloc(mm * sizeof(double));
    double* t1 = (double*)malloc(mm * sizeof(double));
    double* t2 = (double*)malloc(mm * sizeof(double));
    double* Gn = (double*)malloc(mm * sizeof(double));
    memcpy(G, Gin, mm * sizeof(double));
    transpose(s->Wk, Wt, m, m);
    for (int t = T - 1; t >= 0; --t) {
        const double* X = s->Xs + (size_t)t * mm;
        transpose(X, Xt, m, m);
        /* dW -= X^T G X^T */
        matmul(Xt, G, t1, m, m, m);
        matmul(t1, Xt, t2, m, m, m);
        for (size_t e = 0; e < mm; ++e) dW[e] -= t2[e];
        /* G <- 2G - G X^T W^T - W^T X^T G */
        matmul(G, Xt, t1, m, m, m);
        matmul(t1, Wt, t2, m, m, m);
        for (size_t e = 0; e < mm; ++e) Gn[e] = 2.0 * G[e] - t2[e];
        matmul(Wt, Xt, t1, m, m, m);
        matmul(t1, G, t2, m, m, m);
        for (size_t e = 0; e < mm; ++e) Gn[e] -= t2[e];
        memcpy(G, Gn, mm * sizeof(double));
    }
    /* X0 = W^T / c */
    const double c = s->c;
    double n1, ninf; int bs, as;
    induced_norms(s->Wk, m, &n1, &bs, &ninf, &as);
    double gw = 0.0;   /* <G0, W^T> */
    for (int a = 0; a < m; ++a)
        for (int b = 0; b < m; ++b) gw += G[a * m + b] * s->Wk[b * m + a];
    const double dc = -gw / (c * c);
    for (int a = 0; a < m; ++a)
        for (int b = 0; b < m; ++b) dW[a * m + b] += G[b * m + a] / c;
    for (int a = 0; a < m; ++a) dW[a * m + bs] += dc * ninf * sgn(s->Wk[a * m + bs]);
    for (int b = 0; b < m; ++b) dW[as * m + b] += dc * n1 * sgn(s->Wk[as * m + b]);
    free(G); free(Xt); free(Wt); free(t1); free(t2); free(Gn);
}

static void head_backward(const double* q, const double* k, const double* v, const double* dO,
                          double* dq, double* dk, double* dvv,
                          double lambda, int norm, double eps, const double* wl, head_state* s) {
    const int n = s->n, d = s->d, m = s->m, T = s->T, dv = s->dv;
    double* outbuf = (double*)malloc((size_t)n * d * sizeof(double));
    head_forward(q, k, v, outbuf, lambda, norm, eps, wl, s);
    free(outbuf);

    double* dY = (double*)malloc((size_t)n * dv * sizeof(double));
    double* dvbar = (double*)calloc((size_t)d, sizeof(double));
    double* dM = (double*)malloc((size_t)m * dv * sizeof(double));
    double* dD = (double*)malloc((size_t)n * m * sizeof(double));
    double* dqt = (double*)calloc((size_t)m * d, sizeof(double));
    double* dkt = (double*)calloc((size_t)m * d, sizeof(double));
    double* dX = (double*)malloc((size_t)m * m * sizeof(double));
    double* dU = (double*)malloc((size_t)m * dv * sizeof(double));
    double* dW = (double*)malloc((size_t)m * m * sizeof(double));
    double* dDB = (double*)malloc((size_t)m * n * sizeof(double));

    /* Normalisation backward. */
    for (int i = 0; i < n; ++i) {
        const double* Yi = s->Y + (size_t)i * dv;
        const double* gi = dO + (size_t)i * d;
        double* dYi = dY + (size_t)i * dv;
        double si = Yi[d];
        if (norm == ORACLE_NORM_INLINE) {
            double t = 0.0;
            for (int c = 0; c < d; ++c) { dYi[c] = gi[c]; t += gi[c] * s->vbar[c]; }
            dYi[d] = -t;
        } else if (norm == ORACLE_NORM_ROWSUM) {
            double t = 0.0;
            for (int c = 0; c < d; ++c) { dYi[c] = gi[c] / si; t += gi[c] * Yi[c]; }
            dYi[d] = -t / (si * si);
        } else {
            for (int c = 0; c < d; ++c) dYi[c] = gi[c];
            dYi[d] = 0.0;
        }
    }
    if (norm == ORACLE_NORM_INLINE)
        for (int c = 0; c < d; ++c) {
            double t = 0.0;
            for (int i = 0; i < n; ++i) t += (1.0 - s->Y[(size_t)i * dv + d]) * dO[(size_t)i * d + c];
            dvbar[c] = t;
        }

    if (norm == ORACLE_NORM_MSPACE) {
        /* Out_i = sum_l z_il M_l[:d], z_il = w_l (a_il - abar_i) + 1/m:
         *   dz_il = dO_i . M_l[:d],   da_il = w_l dz_il - (1/m) sum_l' w_l' dz_il',
         *   dM_l[:d] = sum_i z_il dO_i,  dM_l[d] = 0 (the ones column does not enter). */
#pragma omp parallel for schedule(static)
        for (int i = 0; i < n; ++i) {
            double* dz = (double*)malloc((size_t)m * sizeof(double));
            double t = 0.0;
            for (int l = 0; l < m; ++l) {
                double a = 0.0;
                for (int c = 0; c < d; ++c) a += dO[(size_t)i * d + c] * s->M[l * dv + c];
                dz[l] = a;
                t += (wl ? wl[l] : 1.0) * a;
            }
            for (int l = 0; l < m; ++l) {
                const double da = (wl ? wl[l] : 1.0) * dz[l] - t / m;
                dD[(size_t)i * m + l] = -s->A[(size_t)i * m + l] * da / lambda;
            }
            free(dz);
        }
        double* abar = (double*)malloc((size_t)n * sizeof(double));
        for (int i = 0; i < n; ++i) {
            double a = 0.0;
            for (int l = 0; l < m; ++l) a += s->A[(size_t)i * m + l];
            abar[i] = a / m;
        }
#pragma omp parallel for schedule(static)
        for (int l = 0; l < m; ++l) {
            for (int c = 0; c < d; ++c) {
                double t = 0.0;
                for (int i = 0; i < n; ++i) {
                    const double z = (wl ? wl[l] : 1.0) * (s->A[(size_t)i * m + l] - abar[i]) + 1.0 / m;
                    t += z * dO[(size_t)i * d + c];
                }
                dM[l * dv + c] = t;
            }
            dM[l * dv + d] = 0.0;
        }
        free(abar);
    } else {
        /* Y = A M:  dA = dY M^T,  dM = A^T dY;  A = exp(-D/lambda): dD = -A dA / lambda. */
#pragma omp parallel for schedule(static)
        for (int i = 0; i < n; ++i)
            for (int l = 0; l < m; ++l) {
                double da = 0.0;
                for (int c = 0; c < dv; ++c) da += dY[(size_t)i * dv + c] * s->M[l * dv + c];
                dD[(size_t)i * m + l] = -s->A[(size_t)i * m + l] * da / lambda;
            }
#pragma omp parallel for schedule(static)
        for (int l = 0; l < m; ++l)
            for (int c = 0; c < dv; ++c) {
                double t = 0.0;
                for (int i = 0; i < n; ++i) t += s->A[(size_t)i * m + l] * dY[(size_t)i * dv + c];
                dM[l * dv + c] = t;
            }
    }
    /* D[i][l] = sum_c |q_ic - kt_lc|  ->  dq_ic += dD sign(.),  dkt_lc -= dD sign(.) */
#pragma omp parallel for schedule(static)
    for (int i = 0; i < n; ++i)
        for (int c = 0; c < d; ++c) {
            double t = 0.0;
            for (int l = 0; l < m; ++l)
                t += dD[(size_t)i * m + l] * sgn(q[(size_t)i * d + c] - lm32(s->kt[l * d + c]));
            dq[(size_t)i * d + c] = t;
        }
#pragma omp parallel for schedule(static)
    for (int l = 0; l < m; ++l)
        for (int c = 0; c < d; ++c) {
            double t = 0.0;
            for (int i = 0; i < n; ++i)
                t += dD[(size_t)i * m + l] * sgn(q[(size_t)i * d + c] - lm32(s->kt[l * d + c]));
            dkt[l * d + c] -= t;
        }

    /* M = X_T U:  dX = dM U^T,  dU = X_T^T dM. */
    const double* XT = s->Xs + (size_t)T * m * m;
    for (int a = 0; a < m; ++a)
        for (int b = 0; b < m; ++b) {
            double t = 0.0;
            for (int c = 0; c < dv; ++c) t += dM[a * dv + c] * s->U[b * dv + c];
            dX[a * m + b] = t;
        }
    for (int b = 0; b < m; ++b)
        for (int c = 0; c < dv; ++c) {
            double t = 0.0;
            for (int a = 0; a < m; ++a) t += XT[a * m + b] * dM[a * dv + c];
            dU[b * dv + c] = t;
        }

    /* Newton-Schulz backward. */
    ns_backward(s, dX, dW);

    /* U = B [V|1]:  dB[a][j] = dU_a . [v_j | 1],  dV_j += sum_a B[a][j] dU_a[:d];
     * B = exp(-D'/lambda):  dD' = -B dB / lambda. */
#pragma omp parallel for schedule(static)
    for (int a = 0; a < m; ++a)
        for (int j = 0; j < n; ++j) {
            double db = dU[a * dv + d];
            for (int c = 0; c < d; ++c) db += dU[a * dv + c] * v[(size_t)j * d + c];
            dDB[(size_t)a * n + j] = -s->Bm[(size_t)a * n + j] * db / lambda;
        }
#pragma omp parallel for schedule(static)
    for (int j = 0; j < n; ++j)
        for (int c = 0; c < d; ++c) {
            double tv = 0.0, tk = 0.0;
            for (int a = 0; a < m; ++a) {
                tv += s->Bm[(size_t)a * n + j] * dU[a * dv + c];
                tk += dDB[(size_t)a * n + j] * sgn(lm32(s->qt[a * d + c]) - k[(size_t)j * d + c]);
            }
            dvv[(size_t)j * d + c] = tv + dvbar[c] / n;   /* vbar = (1/n) sum_j v_j */
            dk[(size_t)j * d + c] = -tk;
        }
#pragma omp parallel for schedule(static)
    for (int a = 0; a < m; ++a)
        for (int c = 0; c < d; ++c) {
            double t = 0.0;
            for (int j = 0; j < n; ++j)
                t += dDB[(size_t)a * n + j] * sgn(lm32(s->qt[a * d + c]) - k[(size_t)j * d + c]);
            dqt[a * d + c] += t;
        }

    /* K_LL[a][b] = exp(-||qt_a - kt_b||_1 / lambda)  (the eps shift has unit derivative). */
    for (int a = 0; a < m; ++a)
        for (int b = 0; b < m; ++b) {
            double kab = s->Wk[a * m + b] - (a == b ? eps : 0.0);
            double g = -kab * dW[a * m + b] / lambda;
            for (int c = 0; c < d; ++c) {
                double sg = sgn(lm32(s->qt[a * d + c]) - lm32(s->kt[b * d + c]));
                dqt[a * d + c] += g * sg;
                dkt[b * d + c] -= g * sg;
            }
        }

    /* Landmark means: each token of segment (window) l receives d(mean)/|S_l|. */
    for (int l = 0; l < m; ++l) {
        int a0 = s->starts[l], a1 = s->starts[l + 1];
        double inv = 1.0 / (a1 - a0);
        for (int t = a0; t < a1; ++t)
            for (int c = 0; c < d; ++c) {
                const int i = s->members[t];
                dq[(size_t)i * d + c] += dqt[l * d + c] * inv;
                dk[(size_t)i * d + c] += dkt[l * d + c] * inv;
            }
    }

    free(dY); free(dvbar); free(dM); free(dD); free(dqt); free(dkt);
    free(dX); free(dU); free(dW); free(dDB);
}

int lapattn_oracle_backward(const double* Q, const double* K, const double* V,
                            const double* dOut, double* dQ, double* dK, double* dV,
                            int B, int H, int n, int d, int m, double lambda, int T,
                            int norm, double eps, int grid_w, int r, const double* whiten) {
    if (!Q || !K || !V || !dOut || !dQ || !dK || !dV) return 1;
    int rc = check_args(B, H, n, d, m, lambda, T, norm);
    if (rc) return rc;
    if ((rc = check_windows(n, m, grid_w, r))) return rc;
    const int BH = B * H;
    const size_t hs = (size_t)n * d;
    for (int h = 0; h < BH; ++h) {
        head_state s;
        head_alloc(&s, n, d, m, T, grid_w, r);
        const double* wl = whiten ? whiten + (size_t)(h % H) * m : NULL;
        head_backward(Q + h * hs, K + h * hs, V + h * hs, dOut + h * hs,
                      dQ + h * hs, dK + h * hs, dV + h * hs, lambda, norm, eps, wl, &s);
        head_free(&s);
    }
    return 0;
}

/* ---------------------------------------------------------------------------------------
 * Depth-wise convolution branch of Eq. (7) (R14): every channel of every head is
 * cross-correlated over the token map with its own k x k filter, zero padded to the map's
 * size.  Plain loops over output positions, channels and taps in index order. */
static int dwc_check(int B, int H, int n, int d, int grid_w, int k) {
    if (B < 1 || H < 1 || n < 1 || d < 1) return 4;
    if (grid_w < 1 || n % grid_w != 0) return 4;
    if (k < 1 || k % 2 == 0) return 4;
    return 0;
}

/* the token at map position (y, x) of an H' x W' map, or -1 outside it */
static int map_token(int y, int x, int gh, int gw) {
    if (y < 0 || y >= gh || x < 0 || x >= gw) return -1;
    return y * gw + x;
}

int lapattn_oracle_dwc(const double* V, const double* Wt, const double* bias, double* E,
                       int B, int H, int n, int d, int grid_w, int k) {
    if (dwc_check(B, H, n, d, grid_w, k)) return 4;
    const int gw = grid_w, gh = n / grid_w, p = (k - 1) / 2;
    for (int b = 0; b < B; ++b)
        for (int h = 0; h < H; ++h) {
            const double* v = V + ((size_t)b * H + h) * n * d;
            double* e = E + ((size_t)b * H + h) * n * d;
            for (int y = 0; y < gh; ++y)
                for (int x = 0; x < gw; ++x)
                    for (int c = 0; c < d; ++c) {
                        const double* w = Wt + ((size_t)h * d + c) * k * k;
                        double acc = bias ? bias[h * d + c] : 0.0;
                        for (int u = 0; u < k; ++u)
                            for (int t = 0; t < k; ++t) {
                                const int j = map_token(y + u - p, x + t - p, gh, gw);
                                if (j >= 0) acc += w[u * k + t] * v[(size_t)j * d + c];
                            }
                        e[((size_t)y * gw + x) * d + c] = acc;
                    }
        }
    return 0;
}

/* E_i depends on V_j through tap (u, t) exactly when j = i + (u - p, t - p); so
 * dV_j = sum over taps of w[u][t] dE_{j - (u - p, t - p)}, dW[u][t] = sum_i dE_i V_{i + (u - p, t - p)},
 * dbias = sum_i dE_i, per channel, the last two summed over the batch. */
int lapattn_oracle_dwc_backward(const double* V, const double* Wt, const double* dE,
                                double* dV, double* dWt, double* dbias,
                                int B, int H, int n, int d, int grid_w, int k) {
    if (dwc_check(B, H, n, d, grid_w, k)) return 4;
    const int gw = grid_w, gh = n / grid_w, p = (k - 1) / 2;
    for (size_t e = 0; e < (size_t)H * d * k * k; ++e) dWt[e] = 0.0;
    for (size_t e = 0; e < (size_t)H * d; ++e) dbias[e] = 0.0;
    for (int b = 0; b < B; ++b)
        for (int h = 0; h < H; ++h) {
            const double* v = V + ((size_t)b * H + h) * n * d;
            const double* g = dE + ((size_t)b * H + h) * n * d;
            double* dv = dV + ((size_t)b * H + h) * n * d;
            for (int y = 0; y < gh; ++y)
                for (int x = 0; x < gw; ++x)
                    for (int c = 0; c < d; ++c) {
                        const double* w = Wt + ((size_t)h * d + c) * k * k;
                        double acc = 0.0;
                        for (int u = 0; u < k; ++u)
                            for (int t = 0; t < k; ++t) {
                                const int i = map_token(y - (u - p), x - (t - p), gh, gw);
                                if (i >= 0) acc += w[u * k + t] * g[(size_t)i * d + c];
                            }
                        dv[((size_t)y * gw + x) * d + c] = acc;
                    }
            for (int y = 0; y < gh; ++y)
                for (int x = 0; x < gw; ++x)
                    for (int c = 0; c < d; ++c) {
                        const double gi = g[((size_t)y * gw + x) * d + c];
                        double* dw = dWt + ((size_t)h * d + c) * k * k;
                        for (int u = 0; u < k; ++u)
                            for (int t = 0; t < k; ++t) {
                                const int j = map_token(y + u - p, x + t - p, gh, gw);
                                if (j >= 0) dw[u * k + t] += gi * v[(size_t)j * d + c];
                            }
                        dbias[h * d + c] += gi;
                    }
        }
    return 0;
}
