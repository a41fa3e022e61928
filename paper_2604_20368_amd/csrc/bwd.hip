// bwd.hip -- backward kernels (fp32 inputs) of Nystrom-approximated Laplacian-kernel attention.
//
// Gradient of sum(Out * dOut) through, in reverse order: the normalisation (Eq. (4) / Eq. (3)),
// Y = K_QL M, M = X_T U, the Newton-Schulz updates of Algorithm 2 including the scale of X0,
// U = K_LK [V|1], K_LL, and the landmark means.  Kernel gradient (App. A):
//   d k(x,y) / dx_c = -(1/lambda) sign(x_c - y_c) k(x,y),  with sign(0) = 0.
//
//   bwd_query_kernel     query-major: dY, dA = dY M^T, dD = -A dA / lambda, direct dQ
//   bwd_query_lm_kernel  landmark-major over queries: dM = A^T dY, dkt from K_QL
//   bwd_ns_kernel        dX = dM U^T, dU = X_T^T dM, reverse Newton-Schulz, K_LL backward
//   bwd_key_kernel       key-major: dB = dU [v|1]^T, dV, dD' = -B dB / lambda, direct dK
//   bwd_key_lm_kernel    landmark-major over keys: dqt from K_LK
//   bwd_pool_kernel      landmark-mean backward into dQ, dK
#include "common.hpp"
#include "kernels.hpp"
#include "ns_mfma.hpp"

namespace lapattn {

static inline float kscale_of(float lambda) { return (float)(-1.4426950408889634 / (double)lambda); }

// ------------------------------------------------------------------------------------------
// Query-major pass.  grid (nqb, BH), one query per thread.
template <int D, int NORM>
__global__ __launch_bounds__(256) void bwd_query_kernel(const float* __restrict__ Q, const float* __restrict__ dO,
                                                        float* __restrict__ dQ, const float* __restrict__ kt,
                                                        const float* __restrict__ M, const float* __restrict__ vbar,
                                                        float* __restrict__ Aq, float* __restrict__ dDq,
                                                        float* __restrict__ rs, float* __restrict__ dYd,
                                                        float* __restrict__ dvbar_part, int n, int m,
                                                        float kscale, float inv_lambda, int nqb) {
    constexpr int D1 = D + 1;
    __shared__ float sK[64 * D];
    __shared__ float sM[64 * D1];
    __shared__ float sVb[D];
    __shared__ float sred[256];
    const int h = blockIdx.y, tid = threadIdx.x;
    for (int e = tid; e < m * D; e += 256) sK[e] = kt[(size_t)h * m * D + e];
    for (int e = tid; e < m * D1; e += 256) sM[e] = M[(size_t)h * m * D1 + e];
    if (tid < D) sVb[tid] = vbar[(size_t)h * D + tid];
    __syncthreads();
    const int i = blockIdx.x * 256 + tid;
    const bool live = i < n;
    const size_t row = ((size_t)h * n + (live ? i : 0)) * D;
    float q[D], g[D];
    float s = 0.f, rsc = 1.f, dyd = 0.f;
    if (live) {
#pragma unroll
        for (int c = 0; c < D; ++c) { q[c] = Q[row + c]; g[c] = dO[row + c]; }
        // forward recompute of y (only what the normalisation backward needs)
        float y[D1];
#pragma unroll
        for (int c = 0; c < D1; ++c) y[c] = 0.f;
        for (int l = 0; l < m; ++l) {
            float dist = 0.f;
#pragma unroll
            for (int c = 0; c < D; ++c) dist += fabsf(q[c] - sK[l * D + c]);
            const float a = exp2f(dist * kscale);
#pragma unroll
            for (int c = 0; c < D1; ++c) y[c] = fmaf(a, sM[l * D1 + c], y[c]);
        }
        s = y[D];
        if (NORM == NORM_INLINE) {
            float t = 0.f;
#pragma unroll
            for (int c = 0; c < D; ++c) t = fmaf(g[c], sVb[c], t);
            dyd = -t;
        } else if (NORM == NORM_ROWSUM) {
            float t = 0.f;
#pragma unroll
            for (int c = 0; c < D; ++c) t = fmaf(g[c], y[c], t);
            rsc = 1.f / s;
            dyd = -t / (s * s);
        }
        rs[(size_t)h * n + i] = rsc;
        dYd[(size_t)h * n + i] = dyd;
    }
    // dvbar partial (inline only): sum over this block's queries of (1 - s_i) dO_i, fixed order;
    // the other normalisations do not use vbar and their partials are zero.
    if (NORM != NORM_INLINE && tid < D) dvbar_part[((size_t)h * nqb + blockIdx.x) * D + tid] = 0.f;
    if (NORM == NORM_INLINE) {
        for (int c = 0; c < D; ++c) {
            sred[tid] = live ? (1.f - s) * g[c] : 0.f;
            __syncthreads();
            for (int w = 128; w > 0; w >>= 1) {
                if (tid < w) sred[tid] += sred[tid + w];
                __syncthreads();
            }
            if (tid == 0) dvbar_part[((size_t)h * nqb + blockIdx.x) * D + c] = sred[0];
            __syncthreads();
        }
    }
    if (!live) return;
    float dq[D];
#pragma unroll
    for (int c = 0; c < D; ++c) dq[c] = 0.f;
    for (int l = 0; l < m; ++l) {
        float dist = 0.f;
#pragma unroll
        for (int c = 0; c < D; ++c) dist += fabsf(q[c] - sK[l * D + c]);
        const float a = exp2f(dist * kscale);
        float da = dyd * sM[l * D1 + D];
#pragma unroll
        for (int c = 0; c < D; ++c) da = fmaf(g[c] * rsc, sM[l * D1 + c], da);
        const float dd = -a * da * inv_lambda;
        Aq[((size_t)h * n + i) * m + l] = a;
        dDq[((size_t)h * n + i) * m + l] = dd;
#pragma unroll
        for (int c = 0; c < D; ++c) dq[c] = fmaf(dd, sgnf(q[c] - sK[l * D + c]), dq[c]);
    }
#pragma unroll
    for (int c = 0; c < D; ++c) dQ[row + c] = dq[c];
}

// ------------------------------------------------------------------------------------------
// Landmark-major pass over queries.  grid (nlc, BH), 64 threads (lane = landmark l).
template <int D>
__global__ __launch_bounds__(64) void bwd_query_lm_kernel(const float* __restrict__ Q, const float* __restrict__ dO,
                                                          const float* __restrict__ kt, const float* __restrict__ Aq,
                                                          const float* __restrict__ dDq, const float* __restrict__ rs,
                                                          const float* __restrict__ dYd, float* __restrict__ dM_part,
                                                          float* __restrict__ dkt_part, int n, int m, int chunk,
                                                          int nlc) {
    constexpr int D1 = D + 1;
    const int ch = blockIdx.x, h = blockIdx.y, l = threadIdx.x;
    const bool live = l < m;
    float k[D], dm[D1], dk[D];
#pragma unroll
    for (int c = 0; c < D; ++c) { k[c] = live ? kt[((size_t)h * m + l) * D + c] : 0.f; dk[c] = 0.f; }
#pragma unroll
    for (int c = 0; c < D1; ++c) dm[c] = 0.f;
    const int i0 = ch * chunk, i1 = min(n, i0 + chunk);
    for (int i = i0; i < i1; ++i) {
        const size_t qrow = ((size_t)h * n + i) * D;
        const float a = live ? Aq[((size_t)h * n + i) * m + l] : 0.f;
        const float dd = live ? dDq[((size_t)h * n + i) * m + l] : 0.f;
        const float r = rs[(size_t)h * n + i];
#pragma unroll
        for (int c = 0; c < D; ++c) {
            dm[c] = fmaf(a, dO[qrow + c] * r, dm[c]);
            dk[c] = fmaf(-dd, sgnf(Q[qrow + c] - k[c]), dk[c]);
        }
        dm[D] = fmaf(a, dYd[(size_t)h * n + i], dm[D]);
    }
    if (!live) return;
    const size_t o = ((size_t)h * nlc + ch) * m + l;
#pragma unroll
    for (int c = 0; c < D1; ++c) dM_part[o * D1 + c] = dm[c];
#pragma unroll
    for (int c = 0; c < D; ++c) dkt_part[o * D + c] = dk[c];
}

// ------------------------------------------------------------------------------------------
// Newton-Schulz backward, one block of 256 threads per head, fp64, products on the fp64 matrix
// cores (ns_mfma.hpp).
//   dM = sum of partials;  dX_T = dM U^T;  dU = X_T^T dM.
//   For t = T-1..0, with G = dL/dX_{t+1} and X_{t+1} = 2 X_t - X_t W X_t:
//     dW -= X_t^T G X_t^T;   G <- 2G - G X_t^T W^T - W^T X_t^T G.
//   X0 = W^T / c:  dW += G^T / c + dc (||W||_inf [b = b*] + ||W||_1 [a = a*]) sign(W),
//     dc = -<G, W^T> / c^2.
//   K_LL: dDW = -k dW / lambda;  dqt_a += sum_b dDW_ab sign(qt_a - kt_b);  dkt_b -= same.
// W comes from the forward solve (stored after the iterates).  U and dM are held as value columns (MFMA operands) plus their ones columns.
template <int MP, int D>
__global__ __launch_bounds__(256) void bwd_ns_kernel(const float* __restrict__ qt, const float* __restrict__ kt,
                                                     const double* __restrict__ Xs, const double* __restrict__ cinfo,
                                                     const float* __restrict__ U, const float* __restrict__ dM_part,
                                                     const float* __restrict__ dvbar_part, float* __restrict__ dU,
                                                     float* __restrict__ dvbar, float* __restrict__ dqtW,
                                                     float* __restrict__ dktW, int n, int m, int T, double lambda,
                                                     double eps, int nlc, int nqb) {
    using SQ = ns_tiles<MP, MP>;
    using SU = ns_tiles<MP, D>;
    constexpr int D1 = D + 1;
    constexpr int P = ns_pitch(MP);
    constexpr int PU = ns_pitch(D);
    // W, X, G, T (MP x MP each, pitch P); before the reverse iteration the same space holds the
    // value columns of U and dM (MP x D each, pitch PU) and X_T (pitch P).
    constexpr int PRE = 2 * MP * PU + MP * P;
    constexpr int LDSN = (4 * MP * P > PRE) ? 4 * MP * P : PRE;
    __shared__ double lds[LDSN];
    __shared__ double su1[MP], sdm1[MP];
    __shared__ double svb[256];
    double* sW = lds;
    double* sX = lds + MP * P;
    double* sG = lds + 2 * MP * P;
    double* sT = lds + 3 * MP * P;
    const int h = blockIdx.x, tid = threadIdx.x;
    const float* q = qt + (size_t)h * m * D;
    const float* k = kt + (size_t)h * m * D;
    const size_t mm = (size_t)MP * MP;
    const double* Xh = Xs + (size_t)h * (T + 2) * mm;   // X_0 .. X_T, then W
    const double c = cinfo[h * 4 + 0], n1 = cinfo[h * 4 + 1], ninf = cinfo[h * 4 + 2];
    const int code = (int)cinfo[h * 4 + 3];

    // dvbar (inline normalisation; zeros otherwise because the partials are zero): 256 / D
    // partial sums per column over the query blocks, then in order
    {
        constexpr int G = 256 / D;
        const int g = tid / D, cc = tid % D;
        double s = 0.0;
#pragma unroll 4
        for (int b = g; b < nqb; b += G) s += dvbar_part[((size_t)h * nqb + b) * D + cc];
        svb[tid] = s;
        __syncthreads();
        if (tid < D) {
            double t = 0.0;
#pragma unroll
            for (int gg = 0; gg < G; ++gg) t += svb[gg * D + tid];
            dvbar[(size_t)h * D + tid] = (float)t;
        }
    }
    {
        double* sU = lds;
        double* sdM = lds + MP * PU;
        double* sXT = lds + 2 * MP * PU;
        // dM = sum of the landmark-chunk partials (in chunk order); each thread's entries are
        // loaded together, chunk by chunk
        constexpr int NE = (MP * D1 + 255) / 256;
        double dm[NE];
#pragma unroll
        for (int r = 0; r < NE; ++r) dm[r] = 0.0;
        const int lim = m * D1 - 1;
#pragma unroll 4
        for (int ch = 0; ch < nlc; ++ch) {
            const float* dp = dM_part + ((size_t)h * nlc + ch) * m * D1;
#pragma unroll
            for (int r = 0; r < NE; ++r) {
                const int e = tid + 256 * r;
                const float v = dp[min(e, lim)];
                dm[r] += (e <= lim) ? (double)v : 0.0;
            }
        }
        float uv[NE];
#pragma unroll
        for (int r = 0; r < NE; ++r) uv[r] = U[(size_t)h * m * D1 + min(tid + 256 * r, lim)];
#pragma unroll
        for (int r = 0; r < NE; ++r) {
            const int e = tid + 256 * r;
            if (e < MP * D1) {
                const int a = e / D1, cc = e % D1;
                const double u = (a < m) ? (double)uv[r] : 0.0;
                if (cc < D) {
                    sdM[a * PU + cc] = dm[r];
                    sU[a * PU + cc] = u;
                } else {
                    sdm1[a] = dm[r];
                    su1[a] = u;
                }
            }
        }
        ns_load<MP, P>(sXT, Xh + (size_t)T * mm);
        __syncthreads();
        // dX = dM U^T (registers, kept until G is stored) and dU = X_T^T dM (global)
        f64x4_t dX[SQ::NT];
        ns_mm<MP, MP, D, false, true, PU, PU>(sdM, sU, dX);
#pragma unroll
        for (int i = 0; i < SQ::NT; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) dX[i][j] += sdm1[SQ::row(i, j)] * su1[SQ::col(i)];
        {
            f64x4_t r[SU::NT];
            ns_mm<MP, D, MP, true, false, P, PU>(sXT, sdM, r);
#pragma unroll
            for (int i = 0; i < SU::NT; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int b = SU::row(i, j), cc = SU::col(i);
                    if (b < m) dU[((size_t)h * m + b) * D1 + cc] = (float)r[i][j];
                }
        }
        if (tid < m) {
            double s = 0.0;
            for (int a = 0; a < MP; ++a) s += sXT[a * P + tid] * sdm1[a];
            dU[((size_t)h * m + tid) * D1 + D] = (float)s;
        }
        __syncthreads();
        // W (kernel + eps I, as the forward solve stored it) and G = dX
        ns_load<MP, P>(sW, Xh + (size_t)(T + 1) * mm);
        ns_store<MP, MP, P>(sG, dX);
    }
    f64x4_t dW[SQ::NT];
#pragma unroll
    for (int i = 0; i < SQ::NT; ++i) dW[i] = f64x4_t{0.0, 0.0, 0.0, 0.0};
    if (c > 0.0) {
        // X_t comes through registers: the loads of X_{t-1} are issued before step t's products
        double xr[MP * MP / 256];
        if (T > 0) ns_fetch<MP>(xr, Xh + (size_t)(T - 1) * mm);
        __syncthreads();
        for (int t = T - 1; t >= 0; --t) {
            ns_put<MP, P>(sX, xr);
            __syncthreads();
            if (t > 0) ns_fetch<MP>(xr, Xh + (size_t)(t - 1) * mm);
            f64x4_t r[SQ::NT], r2[SQ::NT];
            // dW -= X^T G X^T
            ns_mm<MP, MP, MP, true, false, P, P>(sX, sG, r);       // X^T G
            ns_store<MP, MP, P>(sT, r);
            __syncthreads();
            ns_mm<MP, MP, MP, false, true, P, P>(sT, sX, r);       // (X^T G) X^T
#pragma unroll
            for (int i = 0; i < SQ::NT; ++i) dW[i] -= r[i];
            __syncthreads();
            // G X^T W^T
            ns_mm<MP, MP, MP, false, true, P, P>(sG, sX, r);       // G X^T
            ns_store<MP, MP, P>(sT, r);
            __syncthreads();
            ns_mm<MP, MP, MP, false, true, P, P>(sT, sW, r2);      // (G X^T) W^T
            __syncthreads();
            // W^T X^T G = (X W)^T G
            ns_mm<MP, MP, MP, true, true, P, P>(sW, sX, r);        // W^T X^T
            ns_store<MP, MP, P>(sT, r);
            __syncthreads();
            ns_mm<MP, MP, MP, false, false, P, P>(sT, sG, r);      // (W^T X^T) G
            __syncthreads();
#pragma unroll
            for (int i = 0; i < SQ::NT; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int a = SQ::row(i, j), b = SQ::col(i);
                    sG[a * P + b] = 2.0 * sG[a * P + b] - r2[i][j] - r[i][j];
                }
            __syncthreads();
        }
        // X0 = W^T / c
        const int as = code / 256, bs = code % 256;
        // <G, W^T>: block reduction in fixed order
        double part = 0.0;
#pragma unroll
        for (int i = 0; i < SQ::NT; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int a = SQ::row(i, j), b = SQ::col(i);
                part += sG[a * P + b] * sW[b * P + a];
            }
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) part += __shfl_xor(part, off, 64);
        if ((tid & 63) == 0) sT[tid >> 6] = part;
        __syncthreads();
        const double dc = -(((sT[0] + sT[1]) + sT[2]) + sT[3]) / (c * c);
#pragma unroll
        for (int i = 0; i < SQ::NT; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int a = SQ::row(i, j), b = SQ::col(i);
                double v = sG[b * P + a] / c;
                if (b == bs) v += dc * ninf * sgnd(sW[a * P + b]);
                if (a == as) v += dc * n1 * sgnd(sW[a * P + b]);
                dW[i][j] += v;
            }
        __syncthreads();
    } else {
        __syncthreads();
    }
    // dDW = -k dW / lambda (k = W - eps on the diagonal), fp32, into the T region; the landmark
    // rows (zero past m) into the X and G regions.  Entries past m are zero, so the sums below
    // run over all MP rows.
    float* sTf = reinterpret_cast<float*>(sT);
    float* sqf = reinterpret_cast<float*>(sX);
    float* skf = sqf + MP * D;
#pragma unroll
    for (int i = 0; i < SQ::NT; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int a = SQ::row(i, j), b = SQ::col(i);
            const double kab = sW[a * P + b] - (a == b && a < m ? eps : 0.0);
            sTf[a * MP + b] = (float)(-kab * dW[i][j] / lambda);
        }
    ns_stage_rows<MP, D>(sqf, q, m * D);
    ns_stage_rows<MP, D>(skf, k, m * D);
    __syncthreads();
    // dqt_a += sum_b dDW_ab sign(qt_a - kt_b);  dkt_b -= sum_a dDW_ab sign(qt_a - kt_b)
    for (int e = tid; e < m * D; e += 256) {
        const int a = e / D, cc = e % D;
        const float qa = sqf[e];
        float s = 0.f;
#pragma unroll 8
        for (int b = 0; b < MP; ++b) {
            const float kb = skf[b * D + cc], t = sTf[a * MP + b];
            s += (qa > kb) ? t : ((qa < kb) ? -t : 0.f);
        }
        dqtW[(size_t)h * m * D + e] = s;
    }
    for (int e = tid; e < m * D; e += 256) {
        const int b = e / D, cc = e % D;
        const float kb = skf[e];
        float s = 0.f;
#pragma unroll 8
        for (int a = 0; a < MP; ++a) {
            const float qa = sqf[a * D + cc], t = sTf[a * MP + b];
            s += (qa > kb) ? t : ((qa < kb) ? -t : 0.f);
        }
        dktW[(size_t)h * m * D + e] = -s;
    }
}

// ------------------------------------------------------------------------------------------
// Key-major pass.  grid (ceil(n/256), BH), one key per thread.
template <int D>
__global__ __launch_bounds__(256) void bwd_key_kernel(const float* __restrict__ K, const float* __restrict__ V,
                                                      float* __restrict__ dK, float* __restrict__ dV,
                                                      const float* __restrict__ qt, const float* __restrict__ dU,
                                                      const float* __restrict__ dvbar, float* __restrict__ dDk,
                                                      int n, int m, float kscale, float inv_lambda) {
    constexpr int D1 = D + 1;
    __shared__ float sQ[64 * D];
    __shared__ float sdU[64 * D1];
    __shared__ float sdv[D];
    const int h = blockIdx.y, tid = threadIdx.x;
    for (int e = tid; e < m * D; e += 256) sQ[e] = qt[(size_t)h * m * D + e];
    for (int e = tid; e < m * D1; e += 256) sdU[e] = dU[(size_t)h * m * D1 + e];
    if (tid < D) sdv[tid] = dvbar[(size_t)h * D + tid];
    __syncthreads();
    const int j = blockIdx.x * 256 + tid;
    if (j >= n) return;
    const size_t row = ((size_t)h * n + j) * D;
    float kk[D], v[D], dk[D], dv[D];
#pragma unroll
    for (int c = 0; c < D; ++c) { kk[c] = K[row + c]; v[c] = V[row + c]; dk[c] = 0.f; dv[c] = 0.f; }
    for (int a = 0; a < m; ++a) {
        float dist = 0.f;
#pragma unroll
        for (int c = 0; c < D; ++c) dist += fabsf(sQ[a * D + c] - kk[c]);
        const float b = exp2f(dist * kscale);
        float db = sdU[a * D1 + D];
#pragma unroll
        for (int c = 0; c < D; ++c) {
            db = fmaf(sdU[a * D1 + c], v[c], db);
            dv[c] = fmaf(b, sdU[a * D1 + c], dv[c]);
        }
        const float dd = -b * db * inv_lambda;
        dDk[((size_t)h * n + j) * m + a] = dd;
#pragma unroll
        for (int c = 0; c < D; ++c) dk[c] = fmaf(-dd, sgnf(sQ[a * D + c] - kk[c]), dk[c]);
    }
    const float invn = 1.f / (float)n;
#pragma unroll
    for (int c = 0; c < D; ++c) {
        dK[row + c] = dk[c];
        dV[row + c] = dv[c] + sdv[c] * invn;
    }
}

// ------------------------------------------------------------------------------------------
// Landmark-major pass over keys.  grid (nlc, BH), 64 threads (lane = landmark a).
template <int D>
__global__ __launch_bounds__(64) void bwd_key_lm_kernel(const float* __restrict__ K, const float* __restrict__ qt,
                                                        const float* __restrict__ dDk, float* __restrict__ dqt_part,
                                                        int n, int m, int chunk, int nlc) {
    const int ch = blockIdx.x, h = blockIdx.y, a = threadIdx.x;
    const bool live = a < m;
    float q[D], acc[D];
#pragma unroll
    for (int c = 0; c < D; ++c) { q[c] = live ? qt[((size_t)h * m + a) * D + c] : 0.f; acc[c] = 0.f; }
    const int j0 = ch * chunk, j1 = min(n, j0 + chunk);
    for (int j = j0; j < j1; ++j) {
        const size_t krow = ((size_t)h * n + j) * D;
        const float dd = live ? dDk[((size_t)h * n + j) * m + a] : 0.f;
#pragma unroll
        for (int c = 0; c < D; ++c) acc[c] = fmaf(dd, sgnf(q[c] - K[krow + c]), acc[c]);
    }
    if (!live) return;
    const size_t o = ((size_t)h * nlc + ch) * m + a;
#pragma unroll
    for (int c = 0; c < D; ++c) dqt_part[o * D + c] = acc[c];
}

// ------------------------------------------------------------------------------------------
// Landmark-mean backward.  grid (m, BH), 256 threads.
__global__ __launch_bounds__(256) void bwd_pool_kernel(float* __restrict__ dQ, float* __restrict__ dK,
                                                       const float* __restrict__ dqtW, const float* __restrict__ dktW,
                                                       const float* __restrict__ dqt_part,
                                                       const float* __restrict__ dkt_part, int n, int d, int m,
                                                       int nlc) {
    const int l = blockIdx.x, h = blockIdx.y, tid = threadIdx.x;
    __shared__ float sq[64], sk[64];
    const int s0 = seg_start(l, n, m), s1 = seg_start(l + 1, n, m);
    const float inv = 1.f / (float)(s1 - s0);
    if (tid < d) {
        const size_t o = ((size_t)h * m + l) * d + tid;
        double aq = dqtW[o], ak = dktW[o];
        for (int ch = 0; ch < nlc; ++ch) {
            const size_t p = (((size_t)h * nlc + ch) * m + l) * d + tid;
            aq += dqt_part[p];
            ak += dkt_part[p];
        }
        sq[tid] = (float)aq * inv;
        sk[tid] = (float)ak * inv;
    }
    __syncthreads();
    for (int e = tid; e < (s1 - s0) * d; e += 256) {
        const int i = s0 + e / d, c = e % d;
        const size_t idx = ((size_t)h * n + i) * d + c;
        dQ[idx] += sq[c];
        dK[idx] += sk[c];
    }
}

// ------------------------------------------------------------------------------------------
// Launch wrappers.

hipError_t launch_bwd_query(int norm, const float* Q, const float* dO, float* dQ, const float* kt, const float* M,
                            const float* vbar, float* Aq, float* dDq, float* rs, float* dYd, float* dvbar_part,
                            int BH, int n, int d, int m, float lambda, int nqb, hipStream_t st) {
    const float ks = kscale_of(lambda), il = 1.f / lambda;
    dim3 grid(nqb, BH);
#define LAPATTN_BQ(Dv, Nv)                                                                                  \
    hipLaunchKernelGGL((bwd_query_kernel<Dv, Nv>), grid, dim3(256), 0, st, Q, dO, dQ, kt, M, vbar, Aq, dDq, rs, \
                       dYd, dvbar_part, n, m, ks, il, nqb)
    if (d == 32) {
        if (norm == NORM_INLINE) LAPATTN_BQ(32, NORM_INLINE);
        else if (norm == NORM_ROWSUM) LAPATTN_BQ(32, NORM_ROWSUM);
        else LAPATTN_BQ(32, NORM_NONE);
    } else {
        if (norm == NORM_INLINE) LAPATTN_BQ(64, NORM_INLINE);
        else if (norm == NORM_ROWSUM) LAPATTN_BQ(64, NORM_ROWSUM);
        else LAPATTN_BQ(64, NORM_NONE);
    }
#undef LAPATTN_BQ
    return hipGetLastError();
}

hipError_t launch_bwd_query_lm(const float* Q, const float* dO, const float* kt, const float* Aq, const float* dDq,
                               const float* rs, const float* dYd, float* dM_part, float* dkt_part, int BH, int n,
                               int d, int m, int chunk, int nlc, hipStream_t st) {
    dim3 grid(nlc, BH);
    if (d == 32)
        hipLaunchKernelGGL((bwd_query_lm_kernel<32>), grid, dim3(64), 0, st, Q, dO, kt, Aq, dDq, rs, dYd, dM_part,
                           dkt_part, n, m, chunk, nlc);
    else
        hipLaunchKernelGGL((bwd_query_lm_kernel<64>), grid, dim3(64), 0, st, Q, dO, kt, Aq, dDq, rs, dYd, dM_part,
                           dkt_part, n, m, chunk, nlc);
    return hipGetLastError();
}

hipError_t launch_bwd_ns(const float* qt, const float* kt, const double* Xs, const double* cinfo, const float* U,
                         const float* dM_part, const float* dvbar_part, float* dU, float* dvbar, float* dqtW,
                         float* dktW, int BH, int n, int d, int m, int T, double lambda, double eps, int nlc,
                         int nqb, int MP, hipStream_t st) {
#define LAPATTN_BNS(MPv, Dv)                                                                                      \
    hipLaunchKernelGGL((bwd_ns_kernel<MPv, Dv>), dim3(BH), dim3(256), 0, st, qt, kt, Xs, cinfo, U, dM_part,       \
                       dvbar_part, dU, dvbar, dqtW, dktW, n, m, T, lambda, eps, nlc, nqb)
    if (MP == 32 && d == 32) LAPATTN_BNS(32, 32);
    else if (MP == 32) LAPATTN_BNS(32, 64);
    else if (d == 32) LAPATTN_BNS(64, 32);
    else LAPATTN_BNS(64, 64);
#undef LAPATTN_BNS
    return hipGetLastError();
}

hipError_t launch_bwd_key(const float* K, const float* V, float* dK, float* dV, const float* qt, const float* dU,
                          const float* dvbar, float* dDk, int BH, int n, int d, int m, float lambda, hipStream_t st) {
    const float ks = kscale_of(lambda), il = 1.f / lambda;
    dim3 grid((n + 255) / 256, BH);
    if (d == 32)
        hipLaunchKernelGGL((bwd_key_kernel<32>), grid, dim3(256), 0, st, K, V, dK, dV, qt, dU, dvbar, dDk, n, m, ks,
                           il);
    else
        hipLaunchKernelGGL((bwd_key_kernel<64>), grid, dim3(256), 0, st, K, V, dK, dV, qt, dU, dvbar, dDk, n, m, ks,
                           il);
    return hipGetLastError();
}

hipError_t launch_bwd_key_lm(const float* K, const float* qt, const float* dDk, float* dqt_part, int BH, int n, int d,
                             int m, int chunk, int nlc, hipStream_t st) {
    dim3 grid(nlc, BH);
    if (d == 32)
        hipLaunchKernelGGL((bwd_key_lm_kernel<32>), grid, dim3(64), 0, st, K, qt, dDk, dqt_part, n, m, chunk, nlc);
    else
        hipLaunchKernelGGL((bwd_key_lm_kernel<64>), grid, dim3(64), 0, st, K, qt, dDk, dqt_part, n, m, chunk, nlc);
    return hipGetLastError();
}

hipError_t launch_bwd_pool(float* dQ, float* dK, const float* dqtW, const float* dktW, const float* dqt_part,
                           const float* dkt_part, int BH, int n, int d, int m, int nlc, hipStream_t st) {
    hipLaunchKernelGGL(bwd_pool_kernel, dim3(m, BH), dim3(256), 0, st, dQ, dK, dqtW, dktW, dqt_part, dkt_part, n, d,
                       m, nlc);
    return hipGetLastError();
}

}  // namespace lapattn
