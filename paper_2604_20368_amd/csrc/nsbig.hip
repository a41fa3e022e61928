// nsbig.hip -- Algorithm 2 (Newton-Schulz) and the steps around it for 64 < m <= 128 landmarks
// (fp32 inputs, fp64 arithmetic).  A 128 x 128 fp64 matrix is 128 KB, so the solve no longer
// fits one workgroup's LDS as it does for m <= 64 (ns_solve_kernel); each matrix product of the
// iteration is instead one launch over 32 x 32 output tiles of every head, with the matrices in
// global memory (they stay in L2).
//
//   nsb_kll_kernel    W = K_LL + eps I of the landmark means (Eq. (9)), padded with zeros
//   nsb_norm_kernel   c = ||W||_1 ||W||_inf (first maximising column / row), X0 = W^T / c
//   nsb_mm_kernel     batched products Out = alpha op(A) op(B) + beta1 C1 + beta2 C2 + gamma I
//   nsb_usum_kernel   U = sum of the key-chunk partials (fp64; fp32 copy for the backward)
//   nsb_final_kernel  M = X_T U, Mc = M[:, :d] - M[:, d] vbar^T, vbar
// and the backward of the same steps (the Newton-Schulz backward of m <= 64, bwd_ns_kernel, split
// the same way):
//   nsb_bwd_vbar_kernel  dvbar and the landmark-space column sums from the query-block partials
//   nsb_bwd_dm_kernel    dM = sum of the landmark-chunk partials, U in fp64
//   (nsb_mm_kernel)      dX_T = dM U^T, dU = X_T^T dM, the reverse iteration
//   nsb_bwd_x0_kernel    the gradient through X0 = W^T / c, dDW = -k dW / lambda, dU to fp32
//   kll_bwd_kernel       the K_LL backward: dqt from the rows, the keys' pooling gradient (also
//                        for m <= 64, after bwd_ns_kernel)
//
// The iteration runs in product form: with E_0 = I - W X0, the updates X_{t+1} = X_t (2I - W X_t)
// satisfy I - W X_t = E_0^(2^t), so X_{t+1} = X_t + X_t E_t with E_{t+1} = E_t E_t -- the same
// iterates in exact arithmetic, and the two products of a step are independent (one launch).
// Matrices are 128 x 128, row-major (pitch 128); rows and columns at or past m are zero.
#include "common.hpp"
#include "kernels.hpp"

namespace lapattn {

constexpr int kBig = 128;

// ------------------------------------------------------------------------------------------
// W = K_LL + eps I in fp64 (L1 distance of the fp32 means in fp64, exp in fp64), zero outside
// m x m.  grid (kBig / 16, BH), 256 threads: block x covers rows 16 x .. 16 x + 15; thread
// (a-pair ag = tid / 128, column b = tid % 128) keeps key landmark row b in registers and forms
// rows 16 x + ag + 2 i.
template <int D>
__global__ __launch_bounds__(256) void nsb_kll_kernel(const float* __restrict__ qt, const float* __restrict__ kt,
                                                      double* __restrict__ W, long long wstride, int m,
                                                      double lambda, double eps) {
    __shared__ float sq[16 * D];
    const int h = blockIdx.y, a0 = 16 * blockIdx.x, tid = threadIdx.x;
    const int b = tid % kBig, ag = tid / kBig;
    for (int e = tid; e < 16 * D; e += 256) {
        const int a = a0 + e / D;
        sq[e] = a < m ? qt[((size_t)h * m + a) * D + e % D] : 0.f;
    }
    double kb[D];
#pragma unroll
    for (int c = 0; c < D; ++c) kb[c] = (b < m) ? (double)kt[((size_t)h * m + b) * D + c] : 0.0;
    __syncthreads();
    double* Wh = W + (size_t)h * wstride;
    for (int i = 0; i < 8; ++i) {
        const int ar = ag + 2 * i, a = a0 + ar;
        double w = 0.0;
        if (a < m && b < m) {
            double dist = 0.0;
#pragma unroll
            for (int c = 0; c < D; ++c) dist += fabs((double)sq[ar * D + c] - kb[c]);
            w = exp(-dist / lambda);
            if (a == b) w += eps;
        }
        Wh[a * kBig + b] = w;
    }
}

// ------------------------------------------------------------------------------------------
// Norms and X0.  grid (BH), 256 threads.  Threads 0..127 sum |W| down column t, threads
// 128..255 along row t - 128, each in index order; the first maximising column b* and row a*
// by a butterfly within each wave, then over the two waves of each kind (lower index on a tie).
// cinfo[h] = {c, ||W||_1, ||W||_inf, a* 256 + b*}; X0 = W^T / c (0 when c = 0).
__global__ __launch_bounds__(256) void nsb_norm_kernel(const double* __restrict__ W, long long wstride,
                                                       double* __restrict__ X0, long long xstride,
                                                       double* __restrict__ cinfo) {
    __shared__ double sv[4];
    __shared__ int si[4];
    __shared__ double sc;
    const int h = blockIdx.x, tid = threadIdx.x, w = tid >> 6;
    const double* Wh = W + (size_t)h * wstride;
    const int idx = tid % kBig;
    // 16 loads in flight per batch, summed in index order
    const int step = tid < kBig ? kBig : 1;
    const double* p = tid < kBig ? Wh + idx : Wh + (size_t)idx * kBig;
    double s = 0.0;
    for (int i0 = 0; i0 < kBig; i0 += 16) {
        double v[16];
#pragma unroll
        for (int i = 0; i < 16; ++i) v[i] = p[(size_t)(i0 + i) * step];
#pragma unroll
        for (int i = 0; i < 16; ++i) s += fabs(v[i]);
    }
    double v = isnan(s) ? -1.0 : s;
    int arg = idx;
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
        const double ov = __shfl_xor(v, off, 64);
        const int oi = __shfl_xor(arg, off, 64);
        if (ov > v || (ov == v && oi < arg)) {
            v = ov;
            arg = oi;
        }
    }
    if ((tid & 63) == 0) {
        sv[w] = v;
        si[w] = arg;
    }
    __syncthreads();
    if (tid == 0) {
        // waves 0, 1: columns 0..63, 64..127; waves 2, 3: rows
        const bool c1 = sv[1] > sv[0];
        const double n1 = c1 ? sv[1] : sv[0];
        const int bs = c1 ? si[1] : si[0];
        const bool r1 = sv[3] > sv[2];
        const double ninf = r1 ? sv[3] : sv[2];
        const int as = r1 ? si[3] : si[2];
        const double c = n1 * ninf;
        sc = c;
        cinfo[h * 4 + 0] = c;
        cinfo[h * 4 + 1] = n1;
        cinfo[h * 4 + 2] = ninf;
        cinfo[h * 4 + 3] = (double)(as * 256 + bs);
    }
    __syncthreads();
    const double c = sc;
    double* Xh = X0 + (size_t)h * xstride;
    for (int e0 = 0; e0 < kBig * kBig; e0 += 256 * 8) {
        double v[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int e = e0 + 256 * i + tid, a = e / kBig, b = e % kBig;
            v[i] = Wh[b * kBig + a];
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) Xh[e0 + 256 * i + tid] = (c > 0.0) ? v[i] / c : 0.0;
    }
}

// ------------------------------------------------------------------------------------------
// Batched fp64 products.  grid (tiles, BH, jobs), 256 threads; job z = blockIdx.z of `js`, head
// h = blockIdx.y, output tile blockIdx.x of 32 x 32 (row-major over the M x N output; blocks past
// the job's tiles return at once).  The tile's 32 rows of op(A) and 32 columns of op(B) are
// staged in LDS as [k][r] and [k][c] (zeros past K, M, N); thread (tr, tc) = (tid / 16, tid % 16)
// accumulates rows 2 tr, 2 tr + 1 and columns 2 tc, 2 tc + 1 over k in order.  Out may be C1 or C2
// (each element is read and written by one thread), never A or B.
__global__ __launch_bounds__(256) void nsb_mm_kernel(NsbJobs js) {
    const NsbJob& J = js.j[blockIdx.z];
    const int h = blockIdx.y, tid = threadIdx.x;
    const int tcn = (J.N + 31) / 32;
    if ((int)blockIdx.x >= ((J.M + 31) / 32) * tcn) return;   // the whole block: no barrier reached
    const int r0 = (blockIdx.x / tcn) * 32, c0 = (blockIdx.x % tcn) * 32;
    constexpr int SP = 34;   // even: a lane's two rows (columns) are one 16-byte read
    __shared__ __attribute__((aligned(16))) double sA[kBig * SP];
    __shared__ __attribute__((aligned(16))) double sB[kBig * SP];
    const double* A = J.A + (size_t)h * J.sA;
    const double* B = J.B + (size_t)h * J.sB;
    const int K = J.K;
    constexpr int NE = 32 * kBig / 256;   // staged elements per thread and operand
    double va[NE], vb[NE];   // every load issued before the first LDS write
#pragma unroll
    for (int i = 0; i < NE; ++i) {
        const int e = tid + 256 * i;
        const int kA = J.ta ? e / 32 : e % kBig, rA = J.ta ? e % 32 : e / kBig;
        const int kB = J.tb ? e % kBig : e / 32, cB = J.tb ? e / kBig : e % 32;
        const int rr = r0 + rA, cc = c0 + cB;
        va[i] = (kA < K && rr < J.M) ? (J.ta ? A[(size_t)kA * J.pa + rr] : A[(size_t)rr * J.pa + kA]) : 0.0;
        vb[i] = (kB < K && cc < J.N) ? (J.tb ? B[(size_t)cc * J.pb + kB] : B[(size_t)kB * J.pb + cc]) : 0.0;
    }
#pragma unroll
    for (int i = 0; i < NE; ++i) {
        const int e = tid + 256 * i;
        const int kA = J.ta ? e / 32 : e % kBig, rA = J.ta ? e % 32 : e / kBig;
        const int kB = J.tb ? e % kBig : e / 32, cB = J.tb ? e / kBig : e % 32;
        sA[kA * SP + rA] = va[i];
        sB[kB * SP + cB] = vb[i];
    }
    __syncthreads();
    const int tr = tid >> 4, tc = tid & 15;
    double a00 = 0.0, a01 = 0.0, a10 = 0.0, a11 = 0.0;
#pragma unroll 8
    for (int k = 0; k < K; ++k) {
        const double2 x = *reinterpret_cast<const double2*>(sA + k * SP + 2 * tr);
        const double2 y = *reinterpret_cast<const double2*>(sB + k * SP + 2 * tc);
        a00 = fma(x.x, y.x, a00);
        a01 = fma(x.x, y.y, a01);
        a10 = fma(x.y, y.x, a10);
        a11 = fma(x.y, y.y, a11);
    }
    const double acc[2][2] = {{a00, a01}, {a10, a11}};
    double* O = J.Out + (size_t)h * J.sOut;
    const double* C1 = J.C1 ? J.C1 + (size_t)h * J.sC1 : nullptr;
    const double* C2 = J.C2 ? J.C2 + (size_t)h * J.sC2 : nullptr;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int r = r0 + 2 * tr + i, c = c0 + 2 * tc + j;
            if (r < J.M && c < J.N) {
                double v = J.alpha * acc[i][j];
                if (C1) v += J.beta1 * C1[(size_t)r * J.pc1 + c];
                if (C2) v += J.beta2 * C2[(size_t)r * J.pc2 + c];
                if (r == c && r < J.idm) v += J.gamma;
                O[(size_t)r * J.pout + c] = v;
            }
        }
}

// ------------------------------------------------------------------------------------------
// U = sum over the key chunks (chunk order, fp64) of Upart[h][chunk][a][c]: Ud[h][a][c] (fp64,
// rows a < m) and U[h][a][c] (fp32, for the backward).  grid (ceil(m (d+1) / 256), BH).
__global__ __launch_bounds__(256) void nsb_usum_kernel(const float* __restrict__ Upart, double* __restrict__ Ud,
                                                       float* __restrict__ U, int m, int D1, int nkc) {
    const int h = blockIdx.y, e = blockIdx.x * 256 + threadIdx.x;
    if (e >= m * D1) return;
    double u = 0.0;
    const float* p = Upart + (size_t)h * nkc * m * D1 + e;
    int ch = 0;
    for (; ch + 8 <= nkc; ch += 8) {   // 8 loads in flight, added in chunk order
        float v[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = p[(size_t)(ch + i) * m * D1];
#pragma unroll
        for (int i = 0; i < 8; ++i) u += (double)v[i];
    }
    for (; ch < nkc; ++ch) u += (double)p[(size_t)ch * m * D1];
    Ud[(size_t)h * m * D1 + e] = u;
    U[(size_t)h * m * D1 + e] = (float)u;
}

// ------------------------------------------------------------------------------------------
// M = X_T U and Mc = M[:, :d] - M[:, d] vbar^T (fp64, then rounded), vbar = sum of the segment
// value sums / n.  grid (kBig / 32, BH), 256 threads: block x forms rows 32 x .. 32 x + 31 with
// U (all rows) and the block's rows of X_T in LDS.
template <int D>
__global__ __launch_bounds__(256) void nsb_final_kernel(const double* __restrict__ XT, long long xstride,
                                                        const double* __restrict__ Ud, const float* __restrict__ vpart,
                                                        float* __restrict__ M, float* __restrict__ Mc,
                                                        float* __restrict__ vbar, int n, int m, int nkc) {
    constexpr int D1 = D + 1;
    __shared__ double sU[kBig * D1];
    __shared__ double sX[32 * kBig];
    __shared__ double sM1[32];
    __shared__ double svb[D];
    const int h = blockIdx.y, r0 = 32 * blockIdx.x, tid = threadIdx.x;
    {
        constexpr int NU = (kBig * D1 + 255) / 256, NX = 32 * kBig / 256;
        double u[NU], x[NX];   // every load issued before the first LDS write
        const double* Xh = XT + (size_t)h * xstride + (size_t)r0 * kBig;
#pragma unroll
        for (int i = 0; i < NU; ++i) {
            const int e = tid + 256 * i;
            u[i] = e < m * D1 ? Ud[(size_t)h * m * D1 + e] : 0.0;
        }
#pragma unroll
        for (int i = 0; i < NX; ++i) x[i] = Xh[tid + 256 * i];
#pragma unroll
        for (int i = 0; i < NU; ++i)
            if (tid + 256 * i < kBig * D1) sU[tid + 256 * i] = u[i];
#pragma unroll
        for (int i = 0; i < NX; ++i) sX[tid + 256 * i] = x[i];
    }
    if (tid < D) {
        double t = 0.0;
        for (int k0 = 0; k0 < nkc; k0 += 16) {   // the key chunks' value sums: 16 loads in flight, in order
            float v[16];
#pragma unroll
            for (int i = 0; i < 16; ++i) v[i] = k0 + i < nkc ? vpart[((size_t)h * nkc + k0 + i) * D + tid] : 0.f;
#pragma unroll
            for (int i = 0; i < 16; ++i) t += (double)v[i];
        }
        svb[tid] = t / n;
        if (blockIdx.x == 0) vbar[(size_t)h * D + tid] = (float)(t / n);
    }
    __syncthreads();
    if (tid < 32) {
        double s = 0.0;
        for (int b = 0; b < kBig; ++b) s += sX[tid * kBig + b] * sU[b * D1 + D];
        sM1[tid] = s;
        if (r0 + tid < m) M[((size_t)h * m + r0 + tid) * D1 + D] = (float)s;
    }
    __syncthreads();
    for (int e = tid; e < 32 * D; e += 256) {
        const int t = e / D, cc = e % D, a = r0 + t;
        if (a >= m) continue;
        double r = 0.0;
        for (int b = 0; b < kBig; ++b) r += sX[t * kBig + b] * sU[b * D1 + cc];
        M[((size_t)h * m + a) * D1 + cc] = (float)r;
        Mc[((size_t)h * m + a) * D + cc] = (float)(r - sM1[t] * svb[cc]);
    }
}

// ------------------------------------------------------------------------------------------
// Backward.  dvbar (inline normalisation; the partials are zero otherwise) and, for the
// landmark-space form, the column sums of (1 - s_i) dO_i and of dO_i: spv[h] = {sp1, sp0}.
// grid (BH), 256 threads: 256 / D partial sums per column over the query blocks, then in order.
template <int D>
__global__ __launch_bounds__(256) void nsb_bwd_vbar_kernel(const float* __restrict__ dvbar_part,
                                                           const float* __restrict__ p0_part,
                                                           float* __restrict__ dvbar, double* __restrict__ spv,
                                                           int mspace, int nqb) {
    constexpr int G = 256 / D;
    __shared__ double svb[256];
    const int h = blockIdx.x, tid = threadIdx.x, g = tid / D, cc = tid % D;
    auto colsum = [&](const float* part) {   // blocks g, g + G, ... in order, 8 loads in flight
        double t = 0.0;
        int b = g;
        for (; b + 7 * G < nqb; b += 8 * G) {
            float v[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) v[i] = part[((size_t)h * nqb + b + i * G) * D + cc];
#pragma unroll
            for (int i = 0; i < 8; ++i) t += v[i];
        }
        for (; b < nqb; b += G) t += part[((size_t)h * nqb + b) * D + cc];
        return t;
    };
    svb[tid] = colsum(dvbar_part);
    __syncthreads();
    if (tid < D) {
        double t = 0.0;
#pragma unroll
        for (int gg = 0; gg < G; ++gg) t += svb[gg * D + tid];
        spv[(size_t)h * 2 * D + tid] = t;
        dvbar[(size_t)h * D + tid] = mspace ? 0.f : (float)t;
    }
    if (mspace) {
        __syncthreads();
        svb[tid] = colsum(p0_part);
        __syncthreads();
        if (tid < D) {
            double t = 0.0;
#pragma unroll
            for (int gg = 0; gg < G; ++gg) t += svb[gg * D + tid];
            spv[(size_t)h * 2 * D + D + tid] = t;
        }
    }
}

// dMd[h][a][c] = sum over the landmark chunks (chunk order, fp64) of dM_part; for the
// landmark-space form, whose partials hold the gradient of M~ = diag(w) M with the ones column
// 1/m: dM_l[:d] = w_l (dM~_l + sp1 - sp0) + sp0 / m and no gradient for the ones column.
// Ud = U in fp64.  Rows past m are zero.  grid (ceil(128 (d+1) / 256), BH).
__global__ __launch_bounds__(256) void nsb_bwd_dm_kernel(const float* __restrict__ dM_part, const float* __restrict__ U,
                                                         const double* __restrict__ spv,
                                                         const float* __restrict__ whiten, double* __restrict__ dMd,
                                                         double* __restrict__ Ud, int mspace, int H, int m, int D,
                                                         int nlc) {
    const int D1 = D + 1, h = blockIdx.y, e = blockIdx.x * 256 + threadIdx.x;
    if (e >= kBig * D1) return;
    const int a = e / D1, cc = e % D1;
    double dm = 0.0, u = 0.0;
    if (a < m) {
        const float* pp = dM_part + (size_t)h * nlc * m * D1 + e;
        int ch = 0;
        for (; ch + 8 <= nlc; ch += 8) {   // 8 loads in flight, added in chunk order
            float v[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) v[i] = pp[(size_t)(ch + i) * m * D1];
#pragma unroll
            for (int i = 0; i < 8; ++i) dm += (double)v[i];
        }
        for (; ch < nlc; ++ch) dm += (double)pp[(size_t)ch * m * D1];
        if (mspace) {
            const double wa = whiten ? (double)whiten[(size_t)(h % H) * m + a] : 1.0;
            const double* sp = spv + (size_t)h * 2 * D;
            dm = cc < D ? wa * (dm + sp[cc] - sp[D + cc]) + sp[D + cc] / m : 0.0;
        }
        u = (double)U[(size_t)h * m * D1 + e];
    }
    dMd[(size_t)h * kBig * D1 + e] = dm;
    Ud[(size_t)h * kBig * D1 + e] = u;
}

// The gradient through X0 = W^T / c, c = ||W||_1 ||W||_inf (when c > 0):
//   dW += G^T / c + dc (||W||_inf [b = b*] + ||W||_1 [a = a*]) sign(W),  dc = -<G, W^T> / c^2,
// then dDW = -k dW / lambda (k = W - eps on the diagonal) in fp32, and dU (fp64, pitch d+1) to
// fp32.  dW holds the reverse iteration's sum (have_dw = 0: none, T = 0).  grid (BH), 256 threads;
// <G, W^T> per thread, then over the lanes, then over the four waves in order.
__global__ __launch_bounds__(256) void nsb_bwd_x0_kernel(const double* __restrict__ G, const double* __restrict__ W,
                                                         long long wstride, const double* __restrict__ dW,
                                                         int have_dw, const double* __restrict__ cinfo,
                                                         float* __restrict__ dDW, const double* __restrict__ dUd,
                                                         float* __restrict__ dU, int m, int D1, double lambda,
                                                         double eps) {
    __shared__ double sp[4];
    const int h = blockIdx.x, tid = threadIdx.x;
    const size_t mm = (size_t)kBig * kBig;
    const double* Gh = G + (size_t)h * mm;
    const double* Wh = W + (size_t)h * wstride;
    const double c = cinfo[h * 4 + 0], n1 = cinfo[h * 4 + 1], ninf = cinfo[h * 4 + 2];
    const int code = (int)cinfo[h * 4 + 3], as = code / 256, bs = code % 256;
    double part = 0.0;
    for (int e0 = 0; e0 < kBig * kBig; e0 += 256 * 8) {   // 8 pairs of loads in flight
        double g[8], wt[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int e = e0 + 256 * i + tid;
            g[i] = Gh[e];
            wt[i] = Wh[(e % kBig) * kBig + e / kBig];
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) part += g[i] * wt[i];
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) part += __shfl_xor(part, off, 64);
    if ((tid & 63) == 0) sp[tid >> 6] = part;
    __syncthreads();
    const double dc = c > 0.0 ? -(((sp[0] + sp[1]) + sp[2]) + sp[3]) / (c * c) : 0.0;
    for (int e0 = 0; e0 < kBig * kBig; e0 += 256 * 8) {
        double wv[8], dv[8], gt[8];   // all loads of the batch in flight together
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int e = e0 + 256 * i + tid, a = e / kBig, b = e % kBig;
            wv[i] = Wh[e];
            dv[i] = have_dw ? dW[(size_t)h * mm + e] : 0.0;
            gt[i] = Gh[b * kBig + a];
        }
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int e = e0 + 256 * i + tid, a = e / kBig, b = e % kBig;
            const double wab = wv[i];
            double v = dv[i];
            if (c > 0.0) {
                v += gt[i] / c;
                if (b == bs) v += dc * ninf * sgnd(wab);
                if (a == as) v += dc * n1 * sgnd(wab);
            }
            const double kab = wab - (a == b && a < m ? eps : 0.0);
            dDW[(size_t)h * mm + e] = (float)(-kab * v / lambda);
        }
    }
    for (int e = tid; e < m * D1; e += 256) dU[(size_t)h * m * D1 + e] = (float)dUd[(size_t)h * kBig * D1 + e];
}

// K_LL backward: dqtW_a += sum_b dDW_ab sign(qt_a - kt_b) (blockIdx.z = 0, rows a) and
// dk~_b = -sum_a dDW_ab sign(qt_a - kt_b) plus the query-side partials (chunk order, fp64), over
// the landmark's token count (blockIdx.z = 1, columns b): the pooling gradient the key-major pass
// adds to its dK rows.  dDW is MPW x MPW per head (MPW = 32, 64 or 128, zero past m).  grid
// (ceil(m / R), BH, 2), R = 256 / D landmarks per block, thread (landmark x0 + tid / D,
// coordinate tid % D); the other side's landmark rows and the block's rows (columns) of dDW are
// staged in LDS.  Sums in index order.
template <int D, int MPW>
__global__ __launch_bounds__(256) void kll_bwd_kernel(const float* __restrict__ qt, const float* __restrict__ kt,
                                                      const float* __restrict__ dDW, float* __restrict__ dqtW,
                                                      float* __restrict__ dkpool,
                                                      const float* __restrict__ dkt_part, LmPool pl, int n,
                                                      int m, int nlc) {
    constexpr int R = 256 / D;
    __shared__ float so[MPW * D];
    __shared__ float st[R * MPW];
    const int h = blockIdx.y, z = blockIdx.z, tid = threadIdx.x;
    const int r = tid / D, cc = tid % D, x0 = blockIdx.x * R, x = x0 + r;
    const float* other = (z == 0 ? kt : qt) + (size_t)h * m * D;
    const float* Th = dDW + (size_t)h * MPW * MPW;
    {
        constexpr int NO = (MPW * D + 255) / 256, NT = (R * MPW + 255) / 256;
        float vo[NO], vt[NT];   // every load issued before the first LDS write
#pragma unroll
        for (int i = 0; i < NO; ++i) {
            const int e = tid + 256 * i;
            vo[i] = e < m * D ? other[e] : 0.f;
        }
#pragma unroll
        for (int i = 0; i < NT; ++i) {
            const int e = tid + 256 * i, xr = x0 + e / MPW, jj = e % MPW;
            vt[i] = (xr < m && e < R * MPW) ? (z == 0 ? Th[xr * MPW + jj] : Th[jj * MPW + xr]) : 0.f;
        }
#pragma unroll
        for (int i = 0; i < NO; ++i)
            if (tid + 256 * i < MPW * D) so[tid + 256 * i] = vo[i];
#pragma unroll
        for (int i = 0; i < NT; ++i)
            if (tid + 256 * i < R * MPW) st[tid + 256 * i] = vt[i];
    }
    __syncthreads();
    if (x >= m) return;
    const float* trow = st + r * MPW;
    float s = 0.f;
    if (z == 0) {
        const float qa = qt[((size_t)h * m + x) * D + cc];
        for (int b = 0; b < m; ++b) {
            const float kb = so[b * D + cc], t = trow[b];
            s += (qa > kb) ? t : ((qa < kb) ? -t : 0.f);
        }
        dqtW[((size_t)h * m + x) * D + cc] = s;
    } else {
        const float kb = kt[((size_t)h * m + x) * D + cc];
        for (int a = 0; a < m; ++a) {
            const float qa = so[a * D + cc], t = trow[a];
            s += (qa > kb) ? t : ((qa < kb) ? -t : 0.f);
        }
        double ak = -s;
        const float* pp = dkt_part + ((size_t)h * nlc * m + x) * D + cc;
        int ch = 0;
        for (; ch + 8 <= nlc; ch += 8) {   // 8 loads in flight, added in chunk order
            float v[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) v[i] = pp[(size_t)(ch + i) * m * D];
#pragma unroll
            for (int i = 0; i < 8; ++i) ak += v[i];
        }
        for (; ch < nlc; ++ch) ak += pp[(size_t)ch * m * D];
        dkpool[((size_t)h * m + x) * D + cc] = (float)ak * (1.f / (float)lm_tokens(pl, x, n, m).count);
    }
}

// ------------------------------------------------------------------------------------------
// Launch wrappers.

hipError_t launch_nsb_mm(const NsbJobs& js, int njobs, int BH, hipStream_t st) {
    int tiles = 1;
    for (int i = 0; i < njobs; ++i) {
        const int t = ((js.j[i].M + 31) / 32) * ((js.j[i].N + 31) / 32);
        tiles = t > tiles ? t : tiles;
    }
    hipLaunchKernelGGL(nsb_mm_kernel, dim3(tiles, BH, njobs), dim3(256), 0, st, js);
    return hipGetLastError();
}

NsbJob nsb_job(const double* A, long long sA, int pa, bool ta, const double* B, long long sB, int pb, bool tb,
               double* Out, long long sOut, int pout, int M, int N, int K, double alpha) {
    NsbJob j{};
    j.A = A; j.sA = sA; j.pa = pa; j.ta = ta ? 1 : 0;
    j.B = B; j.sB = sB; j.pb = pb; j.tb = tb ? 1 : 0;
    j.Out = Out; j.sOut = sOut; j.pout = pout;
    j.M = M; j.N = N; j.K = K;
    j.alpha = alpha;
    return j;
}

hipError_t launch_nsb_forward(const float* qt, const float* kt, const float* Upart, const float* vpart, double* Xs,
                              double* Ebuf, double* Ud, double* cinfo, float* U, float* M, float* Mc, float* vbar,
                              int BH, int n, int d, int m, int T, double lambda, double eps, int nkc, hipStream_t st) {
    const long long mm = (long long)kBig * kBig, xs = (long long)(T + 2) * mm, es = 2 * mm;
    double* W = Xs + (size_t)(T + 1) * mm;   // per head: X_0 .. X_T, then W
    if (d == 32)
        hipLaunchKernelGGL(nsb_kll_kernel<32>, dim3(kBig / 16, BH), dim3(256), 0, st, qt, kt, W, xs, m, lambda, eps);
    else
        hipLaunchKernelGGL(nsb_kll_kernel<64>, dim3(kBig / 16, BH), dim3(256), 0, st, qt, kt, W, xs, m, lambda, eps);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(nsb_norm_kernel, dim3(BH), dim3(256), 0, st, W, xs, Xs, xs, cinfo);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    if (T > 0) {
        // E_0 = I - W X0
        NsbJobs js{};
        js.j[0] = nsb_job(W, xs, kBig, false, Xs, xs, kBig, false, Ebuf, es, kBig, kBig, kBig, kBig, -1.0);
        js.j[0].gamma = 1.0;
        js.j[0].idm = m;
        if ((e = launch_nsb_mm(js, 1, BH, st)) != hipSuccess) return e;
    }
    for (int k = 0; k < T; ++k) {
        const double* Zk = Xs + (size_t)k * mm;
        const double* Ek = Ebuf + (size_t)(k & 1) * mm;
        NsbJobs js{};
        // X_{k+1} = X_k + X_k E_k
        js.j[0] = nsb_job(Zk, xs, kBig, false, Ek, es, kBig, false, Xs + (size_t)(k + 1) * mm, xs, kBig, kBig, kBig,
                          kBig, 1.0);
        js.j[0].C1 = Zk;
        js.j[0].sC1 = xs;
        js.j[0].pc1 = kBig;
        js.j[0].beta1 = 1.0;
        int nj = 1;
        if (k + 1 < T) {   // E_{k+1} = E_k E_k
            js.j[1] = nsb_job(Ek, es, kBig, false, Ek, es, kBig, false, Ebuf + (size_t)((k + 1) & 1) * mm, es, kBig,
                              kBig, kBig, kBig, 1.0);
            nj = 2;
        }
        if ((e = launch_nsb_mm(js, nj, BH, st)) != hipSuccess) return e;
    }
    const int D1 = d + 1;
    hipLaunchKernelGGL(nsb_usum_kernel, dim3((m * D1 + 255) / 256, BH), dim3(256), 0, st, Upart, Ud, U, m, D1, nkc);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const double* XT = Xs + (size_t)T * mm;
    if (d == 32)
        hipLaunchKernelGGL(nsb_final_kernel<32>, dim3(kBig / 32, BH), dim3(256), 0, st, XT, xs, Ud, vpart, M, Mc, vbar,
                           n, m, nkc);
    else
        hipLaunchKernelGGL(nsb_final_kernel<64>, dim3(kBig / 32, BH), dim3(256), 0, st, XT, xs, Ud, vpart, M, Mc, vbar,
                           n, m, nkc);
    return hipGetLastError();
}

// Backward of the steps above for 64 < m <= 128 (the role of bwd_ns_kernel):
//   dX_T = dM U^T, dU = X_T^T dM;  G = dX_T;  for t = T-1 .. 0, with X_{t+1} = 2 X_t - X_t W X_t:
//     dW -= X_t^T G X_t^T;   G <- 2G - G X_t^T W^T - W^T X_t^T G   (three launches a step);
//   then the X0 term and K_LL (nsb_bwd_x0_kernel, nsb_bwd_kll_kernel).
// scratch: per head 7 matrices of 128 x 128 (G twice, P1, P2, P3, R2, dW) and 3 of 128 x (d+1)
// (dM, U, dU) in fp64, spv (2 d fp64), dDW (128 x 128 fp32).
hipError_t launch_nsb_backward(const float* qt, const float* kt, const double* Xs, const double* cinfo,
                               const float* U, const float* dM_part, const float* dvbar_part,
                               const float* p0_part, const float* whiten, int mspace, float* dU, float* dvbar,
                               float* dqtW, float* dkpool, const float* dkt_part, LmPool pl, double* scratch,
                               float* dDW, int BH, int H, int n, int d, int m, int T, double lambda, double eps,
                               int nlc, int nqb, hipStream_t st) {
    const long long mm = (long long)kBig * kBig, xs = (long long)(T + 2) * mm;
    const int D1 = d + 1;
    const long long md = (long long)kBig * D1;
    double* Gb[2] = {scratch, scratch + (size_t)BH * mm};
    double* P1 = scratch + 2 * (size_t)BH * mm;
    double* P2 = scratch + 3 * (size_t)BH * mm;
    double* P3 = scratch + 4 * (size_t)BH * mm;
    double* R2 = scratch + 5 * (size_t)BH * mm;
    double* dW = scratch + 6 * (size_t)BH * mm;
    double* dMd = scratch + 7 * (size_t)BH * mm;
    double* Ud = dMd + (size_t)BH * md;
    double* dUd = Ud + (size_t)BH * md;
    double* spv = dUd + (size_t)BH * md;
    const double* W = Xs + (size_t)(T + 1) * mm;
    hipError_t e;
    if (d == 32)
        hipLaunchKernelGGL(nsb_bwd_vbar_kernel<32>, dim3(BH), dim3(256), 0, st, dvbar_part, p0_part, dvbar, spv, mspace,
                           nqb);
    else
        hipLaunchKernelGGL(nsb_bwd_vbar_kernel<64>, dim3(BH), dim3(256), 0, st, dvbar_part, p0_part, dvbar, spv, mspace,
                           nqb);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    hipLaunchKernelGGL(nsb_bwd_dm_kernel, dim3((kBig * D1 + 255) / 256, BH), dim3(256), 0, st, dM_part, U, spv, whiten,
                       dMd, Ud, mspace, H, m, d, nlc);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    {
        NsbJobs js{};
        // dX_T = dM U^T (the ones column included: k over d + 1)
        js.j[0] = nsb_job(dMd, md, D1, false, Ud, md, D1, true, Gb[0], mm, kBig, kBig, kBig, D1, 1.0);
        // dU = X_T^T dM
        js.j[1] = nsb_job(Xs + (size_t)T * mm, xs, kBig, true, dMd, md, D1, false, dUd, md, D1, kBig, D1, kBig, 1.0);
        if ((e = launch_nsb_mm(js, 2, BH, st)) != hipSuccess) return e;
    }
    for (int t = T - 1, i = 0; t >= 0; --t, ++i) {
        const double* X = Xs + (size_t)t * mm;
        double* Gc = Gb[i & 1];
        double* Gn = Gb[(i + 1) & 1];
        NsbJobs a{};
        a.j[0] = nsb_job(X, xs, kBig, true, Gc, mm, kBig, false, P1, mm, kBig, kBig, kBig, kBig, 1.0);   // X^T G
        a.j[1] = nsb_job(Gc, mm, kBig, false, X, xs, kBig, true, P2, mm, kBig, kBig, kBig, kBig, 1.0);   // G X^T
        a.j[2] = nsb_job(W, xs, kBig, true, X, xs, kBig, true, P3, mm, kBig, kBig, kBig, kBig, 1.0);    // W^T X^T
        if ((e = launch_nsb_mm(a, 3, BH, st)) != hipSuccess) return e;
        NsbJobs b{};
        b.j[0] = nsb_job(P1, mm, kBig, false, X, xs, kBig, true, dW, mm, kBig, kBig, kBig, kBig, -1.0);  // dW -= P1 X^T
        if (t < T - 1) {
            b.j[0].C1 = dW;
            b.j[0].sC1 = mm;
            b.j[0].pc1 = kBig;
            b.j[0].beta1 = 1.0;
        }
        b.j[1] = nsb_job(P2, mm, kBig, false, W, xs, kBig, true, R2, mm, kBig, kBig, kBig, kBig, 1.0);   // G X^T W^T
        if ((e = launch_nsb_mm(b, 2, BH, st)) != hipSuccess) return e;
        NsbJobs c{};
        c.j[0] = nsb_job(P3, mm, kBig, false, Gc, mm, kBig, false, Gn, mm, kBig, kBig, kBig, kBig, -1.0);
        c.j[0].C1 = Gc;   // G' = 2G - G X^T W^T - W^T X^T G
        c.j[0].sC1 = mm;
        c.j[0].pc1 = kBig;
        c.j[0].beta1 = 2.0;
        c.j[0].C2 = R2;
        c.j[0].sC2 = mm;
        c.j[0].pc2 = kBig;
        c.j[0].beta2 = -1.0;
        if ((e = launch_nsb_mm(c, 1, BH, st)) != hipSuccess) return e;
    }
    hipLaunchKernelGGL(nsb_bwd_x0_kernel, dim3(BH), dim3(256), 0, st, Gb[T & 1], W, xs, dW, T > 0 ? 1 : 0, cinfo, dDW,
                       dUd, dU, m, D1, lambda, eps);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    return launch_kll_backward(qt, kt, dDW, dqtW, dkpool, dkt_part, pl, BH, n, d, m, kBig, nlc, st);
}

hipError_t launch_kll_backward(const float* qt, const float* kt, const float* dDW, float* dqtW, float* dkpool,
                               const float* dkt_part, LmPool pl, int BH, int n, int d, int m, int MPW, int nlc,
                               hipStream_t st) {
    const int R = 256 / d;
    const dim3 grid((m + R - 1) / R, BH, 2);
#define LAPATTN_KB(Dv, Mv)                                                                                              hipLaunchKernelGGL((kll_bwd_kernel<Dv, Mv>), grid, dim3(256), 0, st, qt, kt, dDW, dqtW, dkpool, dkt_part, pl, n,                        m, nlc)
    if (MPW == 32) {
        if (d == 32) LAPATTN_KB(32, 32);
        else LAPATTN_KB(64, 32);
    } else if (MPW == 64) {
        if (d == 32) LAPATTN_KB(32, 64);
        else LAPATTN_KB(64, 64);
    } else {
        if (d == 32) LAPATTN_KB(32, 128);
        else LAPATTN_KB(64, 128);
    }
#undef LAPATTN_KB
    return hipGetLastError();
}

}  // namespace lapattn
