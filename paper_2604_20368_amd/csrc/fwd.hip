// fwd.hip -- forward kernels of Nystrom-approximated Laplacian-kernel attention.
//
//   pool_kernel         landmark means (Sec. 4.2, sampling; 1-D segments)
//   key_summary_kernel  U = K_LK [V | 1], split over key chunks (Sec. 3.2, Eq. (3) key summaries;
//                       K_LK of Algorithm 1 in the orientation K_QL X K_LK)
//   ns_solve_kernel     K_LL, Algorithm 2 in fp64 on the matrix cores, then M = X_T U
//   query_out_kernel    Y = K_QL M and the normalisation (Eq. (8), Eq. (4))
#include "common.hpp"
#include "kernels.hpp"
#include "ns_mfma.hpp"
#include "srows.hpp"

namespace lapattn {

// ------------------------------------------------------------------------------------------
// Landmark means.  grid (m, BH), 256 threads: thread (r, c) sums rows r, r+R, ... of the
// segment in column c; the R partial sums are added in a fixed order (deterministic).
template <int DT>
__global__ __launch_bounds__(256) void pool_kernel(const typename elem<DT>::type* __restrict__ Q,
                                                   const typename elem<DT>::type* __restrict__ K,
                                                   const typename elem<DT>::type* __restrict__ V,
                                                   float* __restrict__ qt, float* __restrict__ kt,
                                                   double* __restrict__ vseg, int n, int d, int m) {
    const int l = blockIdx.x, h = blockIdx.y;
    const int s0 = seg_start(l, n, m), s1 = seg_start(l + 1, n, m);
    const int c = threadIdx.x % d, r = threadIdx.x / d, R = blockDim.x / d;
    const size_t base = (size_t)h * n * d;
    double sq = 0.0, sk = 0.0, sv = 0.0;
    for (int i = s0 + r; i < s1; i += R) {
        const size_t idx = base + (size_t)i * d + c;
        sq += elem<DT>::load(Q, idx);
        sk += elem<DT>::load(K, idx);
        sv += elem<DT>::load(V, idx);
    }
    __shared__ double red[3][256];
    red[0][threadIdx.x] = sq;
    red[1][threadIdx.x] = sk;
    red[2][threadIdx.x] = sv;
    __syncthreads();
    if (r == 0) {
        double a = 0.0, b = 0.0, e = 0.0;
        for (int rr = 0; rr < R; ++rr) {
            a += red[0][rr * d + c];
            b += red[1][rr * d + c];
            e += red[2][rr * d + c];
        }
        const double cnt = (double)(s1 - s0);
        const size_t o = ((size_t)h * m + l) * d + c;
        qt[o] = (float)(a / cnt);
        kt[o] = (float)(b / cnt);
        vseg[o] = e;
    }
}

// ------------------------------------------------------------------------------------------
// Key-side summary (fp32 inputs).  grid (nkc, BH), 256 threads; block `chunk` covers keys
// [chunk * chunk_keys, ...) in tiles of 64, one tile per wave at a time (lane = key j).
//   Per tile: the key row in registers; for every landmark a, the L1 distance to qt_a -- the
//   landmark row is wave-uniform and comes through scalar registers, 32 coordinates at a time,
//   each unit's loads issued right after the first use of the previous one -- and
//   B_aj = exp2(dist * kscale) into the wave's LDS tile [a][j]; then U_part[a][c] +=
//   sum_j B_aj [V_j | 1]_c on fp32 MFMA 16x16x4 (A = B from LDS, B = value rows straight from
//   global memory, loaded before the landmark loop; the ones column is column 0 of the last
//   column tile).  At the end the four waves' partials are added in a fixed order.
// Writes Upart[h][chunk][a][c] for a < m, c <= d.
typedef float f32x4_t __attribute__((ext_vector_type(4)));

template <int D>
__global__ __launch_bounds__(256) void key_summary_kernel(const float* __restrict__ K, const float* __restrict__ V,
                                                          const float* __restrict__ qt, float* __restrict__ Upart,
                                                          int n, int m, float kscale, int chunk_keys, int nkc) {
    constexpr int D1 = D + 1;
    constexpr int NCH = D / 32;            // 32-coordinate units per landmark row
    constexpr int CT = D / 16 + 1;         // MFMA column tiles: the values, then the ones column
    constexpr int BP = 68;                 // LDS pitch of a wave's B tile (conflict-free reads)
    constexpr int RP = 16 * CT;            // pitch of the partial being reduced
    __shared__ __attribute__((aligned(16))) float lds[4 * 64 * BP];
    const int chunk = blockIdx.x, h = blockIdx.y;
    const int tid = threadIdx.x, w = tid >> 6, l = tid & 63, li = l & 15, lk = l >> 4;
    float* sB = lds + w * 64 * BP;
    const float* tab = qt + (size_t)h * m * D;
    const int units = m * NCH;
    for (int a = m; a < 64; ++a) sB[a * BP + l] = 0.f;
    f32x4_t acc[4][CT];
#pragma unroll
    for (int rt = 0; rt < 4; ++rt)
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) acc[rt][ct] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    const int j0 = chunk * chunk_keys, j1 = min(n, j0 + chunk_keys);
    for (int jt = j0 + 64 * w; jt < j1; jt += 256) {
        const int j = jt + l;
        const bool live = j < n;
        float x[D];
        {
            const float4* kr = reinterpret_cast<const float4*>(K + ((size_t)h * n + (live ? j : n - 1)) * D);
#pragma unroll
            for (int c4 = 0; c4 < D / 4; ++c4) {
                const float4 v = kr[c4];
                x[4 * c4 + 0] = v.x;
                x[4 * c4 + 1] = v.y;
                x[4 * c4 + 2] = v.z;
                x[4 * c4 + 3] = v.w;
            }
        }
        __builtin_amdgcn_sched_barrier(0);   // the key row's loads go first: waited for first
        // value operands of the tile's 16 k-steps (rows jt + 4s + lk, clamped to the last key)
        float bv[16][CT - 1];
#pragma unroll
        for (int s = 0; s < 16; ++s) {
            const int r = min(jt + 4 * s + lk, n - 1);
#pragma unroll
            for (int ct = 0; ct < CT - 1; ++ct)
                bv[s][ct] = V[((size_t)h * n + r) * D + 16 * ct + li];
        }
        // landmark loop: unit u = (a, 32-coordinate part) of the table, two units per pass in
        // alternating buffers; both units of a pass always run (a surplus unit past the table
        // repeats the last one and stores a zero row), so that each prefetch stays where it is
        // issued
        {
            float ta[32], tb[32];
            srow32(ta, tab);
            float dist = 0.f;
            for (int u = 0; u < units; u += 2) {
                dist = l1_unit(x + 32 * (u % NCH), ta, tb, tab + 32 * min(u + 1, units - 1), dist);
                if (NCH == 1) {
                    sB[u * BP + l] = live ? __builtin_amdgcn_exp2f(dist * kscale) : 0.f;
                    dist = 0.f;
                }
                dist = l1_unit(x + 32 * ((u + 1) % NCH), tb, ta, tab + 32 * min(u + 2, units - 1), dist);
                const int a = (u + 1) / NCH;   // < 64; a == m only past the table (zero row)
                sB[a * BP + l] = (live && a < m) ? __builtin_amdgcn_exp2f(dist * kscale) : 0.f;
                dist = 0.f;
            }
            // the last prefetch is consumed here, so that no prefetch is moved next to its use
            asm volatile("" ::"s"(ta[0]), "s"(ta[16]));
        }
        __builtin_amdgcn_wave_barrier();
        // U_part += B [V | 1] over the tile's 64 keys, one 16-row tile of landmarks at a time
#pragma unroll
        for (int rt = 0; rt < 4; ++rt) {
            if (16 * rt < m) {
#pragma unroll
                for (int s = 0; s < 16; ++s) {
                    const float av = sB[(16 * rt + li) * BP + 4 * s + lk];
#pragma unroll
                    for (int ct = 0; ct < CT - 1; ++ct)
                        acc[rt][ct] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv[s][ct], acc[rt][ct], 0, 0, 0);
                    acc[rt][CT - 1] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, li == 0 ? 1.f : 0.f, acc[rt][CT - 1],
                                                                             0, 0, 0);
                }
            }
        }
        __builtin_amdgcn_wave_barrier();
    }
    // partials of waves 3, 2, 1, 0 added in that order into one [64][RP] buffer; result register
    // r of a 16x16x4 tile at lane l is row 4 (l / 16) + r, column l % 16
    float* red = lds;
    for (int ww = 3; ww >= 0; --ww) {
        __syncthreads();
        if (w == ww) {
#pragma unroll
            for (int rt = 0; rt < 4; ++rt)
#pragma unroll
                for (int ct = 0; ct < CT; ++ct)
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        float* p = red + (16 * rt + 4 * lk + r) * RP + 16 * ct + li;
                        *p = (ww == 3) ? acc[rt][ct][r] : *p + acc[rt][ct][r];
                    }
        }
    }
    __syncthreads();
    for (int e = tid; e < m * D1; e += 256) {
        const int a = e / D1, c = e % D1;
        Upart[(((size_t)h * nkc + chunk) * m + a) * D1 + c] = red[a * RP + c];
    }
}

// ------------------------------------------------------------------------------------------
// Newton-Schulz solve, one block of 256 threads per head, fp64 in LDS, matrices padded to
// MP x MP with zeros (the padding stays zero under every update):
//   W = K_LL + eps I,  c = ||W||_1 ||W||_inf,  X0 = W^T / c (X := 0 if c = 0),
//   X_{t+1} = X_t (2I - W X_t);  then U = sum of the key-chunk partials, M = X_T U.
// With store_all, Xs[h] holds X_0 .. X_T and then W (T + 2 matrices, pitch MP) for the backward.
// Products on the fp64 matrix cores (ns_mfma.hpp); U's value columns and the ones column are
// kept apart so that the value part of M is one MFMA product and the ones column a matrix-vector
// product.
template <int MP, int D>
__global__ __launch_bounds__(256) void ns_solve_kernel(const float* __restrict__ qt, const float* __restrict__ kt,
                                                       const float* __restrict__ Upart,
                                                       const double* __restrict__ vseg,
                                                       double* __restrict__ Xs, double* __restrict__ cinfo,
                                                       float* __restrict__ U, float* __restrict__ M,
                                                       float* __restrict__ vbar, int n, int m, int T,
                                                       double lambda, double eps, int nkc, int store_all) {
    using SQ = ns_tiles<MP, MP>;
    using SU = ns_tiles<MP, D>;
    constexpr int D1 = D + 1;
    constexpr int P = ns_pitch(MP);
    constexpr int PU = ns_pitch(D);
    // X, W, T (MP x MP each, pitch P); after the iteration U's value columns (MP x D, pitch PU)
    // reuse the space from W on.
    constexpr int LDSN = (3 * MP * P > MP * P + MP * PU) ? 3 * MP * P : MP * P + MP * PU;
    __shared__ double lds[LDSN];
    __shared__ double sred[4];
    __shared__ double su1[MP];
    __shared__ double svb[256];
    __shared__ double sc;
    double* sX = lds;
    double* sW = lds + MP * P;
    double* sT = lds + 2 * MP * P;
    const int h = blockIdx.x, tid = threadIdx.x;
    const float* q = qt + (size_t)h * m * D;
    const float* k = kt + (size_t)h * m * D;

    const size_t mm = (size_t)MP * MP;
    double* Xh = Xs + (size_t)h * (store_all ? (T + 2) : 1) * mm;
    ns_kll<MP, D, P>(q, k, sW, reinterpret_cast<float*>(sT), m, lambda, eps);
    __syncthreads();
    if (store_all)
        for (int e = tid; e < MP * MP; e += 256) Xh[(size_t)(T + 1) * mm + e] = sW[(e / MP) * P + e % MP];
    // column sums (threads 0..MP-1) and row sums (MP..2MP-1) of |W|, each in index order, then
    // the first maximising column b* and row a* by a lane butterfly
    if (tid < 2 * MP) {
        const int idx = tid % MP;
        double s = 0.0;
        if (tid < MP) {
#pragma unroll 16
            for (int a = 0; a < MP; ++a) s += fabs(sW[a * P + idx]);
        } else {
#pragma unroll 16
            for (int b = 0; b < MP; ++b) s += fabs(sW[idx * P + b]);
        }
        double v = isnan(s) ? -1.0 : s;
        int arg = idx;
        ns_group_argmax<MP>(v, arg);
        if (idx == 0) {
            sred[tid < MP ? 0 : 2] = v;
            sred[tid < MP ? 1 : 3] = (double)arg;
        }
    }
    __syncthreads();
    if (tid == 0) {
        const double n1 = sred[0], ninf = sred[2];
        const int bs = (int)sred[1], as = (int)sred[3];
        const double c = n1 * ninf;
        sc = c;
        cinfo[h * 4 + 0] = c;
        cinfo[h * 4 + 1] = n1;
        cinfo[h * 4 + 2] = ninf;
        cinfo[h * 4 + 3] = (double)(as * 256 + bs);
    }
    __syncthreads();
    const double c = sc;
    for (int e = tid; e < MP * MP; e += 256) {
        const int a = e / MP, b = e % MP;
        const double x = (c > 0.0) ? sW[b * P + a] / c : 0.0;
        sX[a * P + b] = x;
        if (store_all) Xh[e] = x;
    }
    __syncthreads();
    for (int t = 0; t < T; ++t) {
        f64x4_t r[SQ::NT];
        ns_mm<MP, MP, MP, false, false, P, P>(sW, sX, r);      // W X
#pragma unroll
        for (int i = 0; i < SQ::NT; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int a = SQ::row(i, j), b = SQ::col(i);
                sT[a * P + b] = (a == b ? 2.0 : 0.0) - r[i][j];
            }
        __syncthreads();
        ns_mm<MP, MP, MP, false, false, P, P>(sX, sT, r);      // X (2I - W X)
        __syncthreads();
#pragma unroll
        for (int i = 0; i < SQ::NT; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int a = SQ::row(i, j), b = SQ::col(i);
                sX[a * P + b] = r[i][j];
                if (store_all) Xh[(size_t)(t + 1) * mm + a * MP + b] = r[i][j];
            }
        __syncthreads();
    }
    if (!store_all)
        for (int e = tid; e < MP * MP; e += 256) Xh[e] = sX[(e / MP) * P + e % MP];

    // U = sum over key chunks (in chunk order) in fp64: value columns from the W region on, the
    // ones column in su1.  Each thread's entries are loaded together, chunk by chunk.
    double* sU = sW;
    {
        constexpr int NE = (MP * D1 + 255) / 256;
        double u[NE];
#pragma unroll
        for (int r = 0; r < NE; ++r) u[r] = 0.0;
        const int lim = m * D1 - 1;
#pragma unroll 4
        for (int ch = 0; ch < nkc; ++ch) {
            const float* up = Upart + ((size_t)h * nkc + ch) * m * D1;
#pragma unroll
            for (int r = 0; r < NE; ++r) {
                const int e = tid + 256 * r;
                const float v = up[min(e, lim)];
                u[r] += (e <= lim) ? (double)v : 0.0;
            }
        }
#pragma unroll
        for (int r = 0; r < NE; ++r) {
            const int e = tid + 256 * r;
            if (e < MP * D1) {
                const int a = e / D1, cc = e % D1;
                if (cc < D) sU[a * PU + cc] = u[r];
                else su1[a] = u[r];
                if (a < m) U[(size_t)h * m * D1 + e] = (float)u[r];
            }
        }
    }
    __syncthreads();
    {
        f64x4_t r[SU::NT];
        ns_mm<MP, D, MP, false, false, P, PU>(sX, sU, r);     // X_T U (value columns)
#pragma unroll
        for (int i = 0; i < SU::NT; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int a = SU::row(i, j), cc = SU::col(i);
                if (a < m) M[((size_t)h * m + a) * D1 + cc] = (float)r[i][j];
            }
    }
    if (tid < m) {
        double s = 0.0;
#pragma unroll 16
        for (int b = 0; b < MP; ++b) s += sX[tid * P + b] * su1[b];
        M[((size_t)h * m + tid) * D1 + D] = (float)s;
    }
    // vbar = (sum of the segment value sums) / n: 256 / D partial sums per column, then in order
    {
        constexpr int G = 256 / D;
        const int g = tid / D, cc = tid % D;
        double s = 0.0;
#pragma unroll 4
        for (int l = g; l < m; l += G) s += vseg[((size_t)h * m + l) * D + cc];
        svb[tid] = s;
        __syncthreads();
        if (tid < D) {
            double t = 0.0;
#pragma unroll
            for (int gg = 0; gg < G; ++gg) t += svb[gg * D + tid];
            vbar[(size_t)h * D + tid] = (float)(t / n);
        }
    }
}

// ------------------------------------------------------------------------------------------
// Query side.  grid (ceil(n/256), BH), one query per thread:
//   y = sum_l k(q_i, kt_l) M_l  (d+1 columns),  s_i = y[d],  then the normalisation.
template <int DT, int D, int NORM>
__global__ __launch_bounds__(256) void query_out_kernel(const typename elem<DT>::type* __restrict__ Q,
                                                        typename elem<DT>::type* __restrict__ Out,
                                                        const float* __restrict__ kt,
                                                        const float* __restrict__ M,
                                                        const float* __restrict__ vbar, int n, int m,
                                                        float kscale) {
    constexpr int D1 = D + 1;
    __shared__ float sK[64 * D];
    __shared__ float sM[64 * D1];
    __shared__ float sVb[D];
    const int h = blockIdx.y, tid = threadIdx.x;
    for (int e = tid; e < m * D; e += 256) sK[e] = kt[(size_t)h * m * D + e];
    for (int e = tid; e < m * D1; e += 256) sM[e] = M[(size_t)h * m * D1 + e];
    if (tid < D) sVb[tid] = vbar[(size_t)h * D + tid];
    __syncthreads();
    const int i = blockIdx.x * 256 + tid;
    if (i >= n) return;
    const size_t row = ((size_t)h * n + i) * D;
    float q[D], y[D1];
#pragma unroll
    for (int c = 0; c < D; ++c) q[c] = elem<DT>::load(Q, row + c);
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
    const float s = y[D];
#pragma unroll
    for (int c = 0; c < D; ++c) {
        float o;
        if (NORM == NORM_INLINE) o = y[c] + (1.f - s) * sVb[c];
        else if (NORM == NORM_ROWSUM) o = y[c] / s;
        else o = y[c];
        elem<DT>::store(Out, row + c, o);
    }
}

// ------------------------------------------------------------------------------------------
// Launch wrappers.

static inline float kscale_of(float lambda) { return (float)(-1.4426950408889634 / (double)lambda); }

hipError_t launch_pool(int dt, const void* Q, const void* K, const void* V, float* qt, float* kt, double* vseg,
                       int BH, int n, int d, int m, hipStream_t st) {
    dim3 grid(m, BH);
    if (dt == DT_F32)
        hipLaunchKernelGGL(pool_kernel<DT_F32>, grid, dim3(256), 0, st, (const float*)Q, (const float*)K,
                           (const float*)V, qt, kt, vseg, n, d, m);
    else
        hipLaunchKernelGGL(pool_kernel<DT_BF16>, grid, dim3(256), 0, st, (const uint16_t*)Q, (const uint16_t*)K,
                           (const uint16_t*)V, qt, kt, vseg, n, d, m);
    return hipGetLastError();
}

hipError_t launch_key_summary(int dt, const void* K, const void* V, const float* qt, float* Upart, int BH, int n,
                              int d, int m, float lambda, int chunk_keys, int nkc, hipStream_t st) {
    if (dt != DT_F32) return hipErrorInvalidValue;   // bf16 inputs take the fast path
    const float ks = kscale_of(lambda);
    if (d == 32)
        hipLaunchKernelGGL((key_summary_kernel<32>), dim3(nkc, BH), dim3(256), 0, st, (const float*)K,
                           (const float*)V, qt, Upart, n, m, ks, chunk_keys, nkc);
    else
        hipLaunchKernelGGL((key_summary_kernel<64>), dim3(nkc, BH), dim3(256), 0, st, (const float*)K,
                           (const float*)V, qt, Upart, n, m, ks, chunk_keys, nkc);
    return hipGetLastError();
}

hipError_t launch_ns_solve(const float* qt, const float* kt, const float* Upart, const double* vseg, double* Xs,
                           double* cinfo, float* U, float* M, float* vbar, int BH, int n, int d, int m, int T,
                           double lambda, double eps, int nkc, int store_all, int MP, hipStream_t st) {
#define LAPATTN_NS(MPv, Dv)                                                                                  \
    hipLaunchKernelGGL((ns_solve_kernel<MPv, Dv>), dim3(BH), dim3(256), 0, st, qt, kt, Upart, vseg, Xs, cinfo, \
                       U, M, vbar, n, m, T, lambda, eps, nkc, store_all)
    if (MP == 32 && d == 32) LAPATTN_NS(32, 32);
    else if (MP == 32) LAPATTN_NS(32, 64);
    else if (d == 32) LAPATTN_NS(64, 32);
    else LAPATTN_NS(64, 64);
#undef LAPATTN_NS
    return hipGetLastError();
}

template <int DT, int D>
static void query_out_launch(int norm, const void* Q, void* Out, const float* kt, const float* M, const float* vbar,
                             int BH, int n, int m, float kscale, hipStream_t st) {
    using T = typename elem<DT>::type;
    dim3 grid((n + 255) / 256, BH);
    if (norm == NORM_INLINE)
        hipLaunchKernelGGL((query_out_kernel<DT, D, NORM_INLINE>), grid, dim3(256), 0, st, (const T*)Q, (T*)Out, kt,
                           M, vbar, n, m, kscale);
    else if (norm == NORM_ROWSUM)
        hipLaunchKernelGGL((query_out_kernel<DT, D, NORM_ROWSUM>), grid, dim3(256), 0, st, (const T*)Q, (T*)Out, kt,
                           M, vbar, n, m, kscale);
    else
        hipLaunchKernelGGL((query_out_kernel<DT, D, NORM_NONE>), grid, dim3(256), 0, st, (const T*)Q, (T*)Out, kt, M,
                           vbar, n, m, kscale);
}

hipError_t launch_query_out(int dt, int norm, const void* Q, void* Out, const float* kt, const float* M,
                            const float* vbar, int BH, int n, int d, int m, float lambda, hipStream_t st) {
    const float ks = kscale_of(lambda);
    if (dt == DT_F32 && d == 32) query_out_launch<DT_F32, 32>(norm, Q, Out, kt, M, vbar, BH, n, m, ks, st);
    else if (dt == DT_F32) query_out_launch<DT_F32, 64>(norm, Q, Out, kt, M, vbar, BH, n, m, ks, st);
    else if (d == 32) query_out_launch<DT_BF16, 32>(norm, Q, Out, kt, M, vbar, BH, n, m, ks, st);
    else query_out_launch<DT_BF16, 64>(norm, Q, Out, kt, M, vbar, BH, n, m, ks, st);
    return hipGetLastError();
}

}  // namespace lapattn
