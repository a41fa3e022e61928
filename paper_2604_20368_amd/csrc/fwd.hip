// fwd.hip -- forward kernels of Nystrom-approximated Laplacian-kernel attention.
//
//   pool_kernel         landmark means (Sec. 4.2, sampling; 1-D segments)
//   key_summary_kernel  U = K_LK [V | 1], split over key chunks (Sec. 3.2, Eq. (3) key summaries;
//                       K_LK of Algorithm 1 in the orientation K_QL X K_LK)
//   ns_solve_kernel     K_LL, Algorithm 2 in fp64 on the matrix cores, then M = X_T U
//   query_out_kernel    Y = K_QL M and the normalisation (Eq. (8), Eq. (4), or the landmark-space
//                       form of Appendix B)
//   mspace_vec_kernel   the two per-head vectors of the landmark-space normalisation
#include "common.hpp"
#include "kernels.hpp"
#include "ns_mfma.hpp"
#include "srows.hpp"

namespace lapattn {

// ------------------------------------------------------------------------------------------
// Landmark means of Q and K (the key side forms the value sums).  grid (m S, BH), 256 threads:
// block (l, s) = (x / S, x % S) sums part s of
// landmark l's tokens (segment or window, lm_tokens; S contiguous parts, S > 1 when m BH alone
// would leave most compute units idle); thread (r, c) sums the part's tokens r, r + R, ... in
// column c, four rows' loads in flight at a time, and the R partial sums are added in a fixed
// order (deterministic).  S = 1 writes the results; otherwise part[h][l][s][2][d] (fp64) for
// pool_combine_kernel, which adds the S parts in order.
template <int DT>
__global__ __launch_bounds__(256) void pool_kernel(const typename elem<DT>::type* __restrict__ Q,
                                                   const typename elem<DT>::type* __restrict__ K,
                                                   float* __restrict__ qt, float* __restrict__ kt,
                                                   double* __restrict__ part, int n, int d, int m, int S, LmPool pl) {
    const int l = blockIdx.x / S, sp = blockIdx.x % S, h = blockIdx.y;
    const LmTokens tok = lm_tokens(pl, l, n, m);
    const int cntl = tok.count;
    const int t0 = (int)((long long)cntl * sp / S), t1 = (int)((long long)cntl * (sp + 1) / S);
    const int c = threadIdx.x % d, r = threadIdx.x / d, R = blockDim.x / d;
    const size_t base = (size_t)h * n * d;
    double sq = 0.0, sk = 0.0;
    int t = t0 + r;
    for (; t + 3 * R < t1; t += 4 * R) {
        float a[4], b[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const size_t idx = base + (size_t)tok(t + u * R) * d + c;
            a[u] = elem<DT>::load(Q, idx);
            b[u] = elem<DT>::load(K, idx);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            sq += a[u];
            sk += b[u];
        }
    }
    for (; t < t1; t += R) {
        const size_t idx = base + (size_t)tok(t) * d + c;
        sq += elem<DT>::load(Q, idx);
        sk += elem<DT>::load(K, idx);
    }
    __shared__ double red[2][256];
    red[0][threadIdx.x] = sq;
    red[1][threadIdx.x] = sk;
    __syncthreads();
    if (r == 0) {
        double a = 0.0, b = 0.0;
        for (int rr = 0; rr < R; ++rr) {
            a += red[0][rr * d + c];
            b += red[1][rr * d + c];
        }
        if (S == 1) {
            const double cnt = (double)cntl;
            const size_t o = ((size_t)h * m + l) * d + c;
            qt[o] = (float)(a / cnt);
            kt[o] = (float)(b / cnt);
        } else {
            double* pp = part + (((size_t)h * m + l) * S + sp) * 2 * d + c;
            pp[0] = a;
            pp[d] = b;
        }
    }
}

// Landmark means when every landmark has few tokens (at most kPoolSmall): grid
// (ceil(m / (256 / d)), BH), 256 threads, thread (landmark x tid / d + blockIdx.x (256 / d),
// column tid % d) sums its landmark's tokens in its column (fp64, in token order), four tokens'
// loads in flight at a time.  The same outputs as pool_kernel with S = 1; at a handful of tokens
// per landmark one block per landmark would be mostly launch overhead.
constexpr int kPoolSmall = 16;

template <int DT>
__global__ __launch_bounds__(256) void pool_small_kernel(const typename elem<DT>::type* __restrict__ Q,
                                                         const typename elem<DT>::type* __restrict__ K,
                                                         float* __restrict__ qt, float* __restrict__ kt, int n, int d,
                                                         int m, LmPool pl) {
    const int lpb = 256 / d;
    const int l = blockIdx.x * lpb + threadIdx.x / d, c = threadIdx.x % d, h = blockIdx.y;
    if (l >= m) return;
    const LmTokens tok = lm_tokens(pl, l, n, m);
    const int cnt = tok.count;
    const size_t base = (size_t)h * n * d + c;
    double sq = 0.0, sk = 0.0;
    int t = 0;
    for (; t + 4 <= cnt; t += 4) {
        float a[4], b[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const size_t idx = base + (size_t)tok(t + u) * d;
            a[u] = elem<DT>::load(Q, idx);
            b[u] = elem<DT>::load(K, idx);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            sq += a[u];
            sk += b[u];
        }
    }
    for (; t < cnt; ++t) {
        const size_t idx = base + (size_t)tok(t) * d;
        sq += elem<DT>::load(Q, idx);
        sk += elem<DT>::load(K, idx);
    }
    const size_t o = ((size_t)h * m + l) * d + c;
    qt[o] = (float)(sq / cnt);
    kt[o] = (float)(sk / cnt);
}

// The S parts of each landmark's sums (S <= kPoolMaxSplit), added in order.  grid (m, BH),
// 2 d threads rounded up to a wave: thread c < d the query sums of column c, d <= c < 2 d the key
// sums of column c - d; the S loads are issued together.
constexpr int kPoolMaxSplit = 16;

__global__ void pool_combine_kernel(const double* __restrict__ part, float* __restrict__ qt, float* __restrict__ kt,
                                    int n, int d, int m, int S, LmPool pl) {
    const int l = blockIdx.x, h = blockIdx.y, c = threadIdx.x;
    if (c >= 2 * d) return;
    const double* pp = part + ((size_t)h * m + l) * S * 2 * d + c;
    double v[kPoolMaxSplit];
#pragma unroll
    for (int sp = 0; sp < kPoolMaxSplit; ++sp) v[sp] = sp < S ? pp[(size_t)sp * 2 * d] : 0.0;
    double a = 0.0;
#pragma unroll
    for (int sp = 0; sp < kPoolMaxSplit; ++sp)
        if (sp < S) a += v[sp];
    const double cnt = (double)lm_tokens(pl, l, n, m).count;
    const size_t o = ((size_t)h * m + l) * d + (c < d ? c : c - d);
    (c < d ? qt : kt)[o] = (float)(a / cnt);
}

// ------------------------------------------------------------------------------------------
// Key-side summary (fp32 inputs).  grid (nkc, BH), 256 threads; block `chunk` covers keys
// [chunk * chunk_keys, ...) (chunk_keys a multiple of 256) in tiles of 64, one tile per wave at a
// time (lane = key j).
//   Per tile: the key row in registers; for every landmark a, the L1 distance to qt_a -- the
//   landmark row is wave-uniform and comes through scalar registers, 32 coordinates at a time,
//   each unit's loads issued right after the first use of the previous one -- and
//   B_aj = exp2(dist * kscale) into the wave's LDS tile [a][j], 32 landmarks at a time (a
//   32 x 64 tile per wave: three blocks share a compute unit at d = 32); after each range,
//   U_part[a][c] += sum_j B_aj [V_j | 1]_c for its landmarks on fp32 MFMA 16x16x4 (A = B from
//   LDS, B = value rows straight from global memory, loaded before the landmark loop; the ones
//   column is column 0 of the last column tile).  At the end the four waves' partials are added
//   in a fixed order.
// Landmarks in groups of 64 (blockIdx.z = group g: landmarks 64 g .. 64 g + 63), so that m up to
// 128 takes two blocks per key chunk, each reading the chunk's keys.
// Writes Upart[h][chunk][a][c] for the group's landmarks a < m, c <= d, and (group 0) the chunk's value
// sums vpart[h][chunk][c] (c < d, for vbar); with Bsave, the keys' rows
// of B into Bsave[h][g][n][64] (group-major rows of 64 landmarks, zeros past m).
typedef float f32x4_t __attribute__((ext_vector_type(4)));

template <int D>
__global__ __launch_bounds__(256, D == 32 ? 3 : 2) void key_summary_kernel(const float* __restrict__ K, const float* __restrict__ V,
                                                          const float* __restrict__ qt, float* __restrict__ Upart,
                                                          float* __restrict__ vpart,
                                                          float* __restrict__ Bsave, int n, int m, float kscale,
                                                          int chunk_keys, int nkc) {
    constexpr int D1 = D + 1;
    constexpr int NCH = D / 32;            // 32-coordinate units per landmark row
    constexpr int CT = D / 16 + 1;         // MFMA column tiles: the values, then the ones column
    constexpr int BP = 68;                 // LDS pitch of a wave's B tile (conflict-free reads)
    constexpr int RP = 16 * CT;            // pitch of the partial being reduced
    __shared__ __attribute__((aligned(16))) float lds[4 * 32 * BP];
    static_assert(65 * RP <= 4 * 32 * BP, "the partial being reduced and the value sums fit the tiles");
    // blocks in XCD-contiguous order: the blocks that one XCD runs take consecutive (head, chunk)
    // pairs, so that a CU's scalar cache serves few landmark tables
    const int G = (int)(gridDim.x * gridDim.y), lin = xcd_order(blockIdx.y * gridDim.x + blockIdx.x, G);
    const int chunk = lin % (int)gridDim.x, h = lin / (int)gridDim.x;
    const int g = blockIdx.z, ng = gridDim.z, lm0 = 64 * g;
    const int mg = min(64, m - lm0);   // landmarks of the group
    const int tid = threadIdx.x, w = tid >> 6, l = tid & 63, li = l & 15, lk = l >> 4;
    float* sB = lds + w * 32 * BP;
    const float* tab = qt + __builtin_amdgcn_readfirstlane((h * m + lm0) * D);   // wave-uniform: scalar loads
    float* Bg = Bsave ? Bsave + (size_t)(h * ng + g) * n * 64 : nullptr;
    f32x4_t acc[4][CT];
#pragma unroll
    for (int rt = 0; rt < 4; ++rt)
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) acc[rt][ct] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    float vsa[CT - 1];   // group 0: this lane's sums of value column 16 ct + li over its keys
#pragma unroll
    for (int ct = 0; ct < CT - 1; ++ct) vsa[ct] = 0.f;
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
        if (g == 0) {
            // vbar's partial sums over the lane's live keys (rows past n repeat the last key)
#pragma unroll
            for (int s = 0; s < 16; ++s) {
                const bool kl = jt + 4 * s + lk < n;
#pragma unroll
                for (int ct = 0; ct < CT - 1; ++ct) vsa[ct] += kl ? bv[s][ct] : 0.f;
            }
        }
#pragma unroll
        for (int ri = 0; ri < 2; ++ri) {   // unrolled: acc is indexed by the range
            if (32 * ri >= mg) break;
            const int mh = min(32, mg - 32 * ri);   // landmarks lm0 + 32 ri .. + mh - 1: tile rows 0 .. mh - 1
            const float* tabr = tab + 32 * ri * D;
            const int units = mh * NCH;
            for (int a = mh; a < 32; ++a) sB[a * BP + l] = 0.f;   // rows past m (else the last range's)
            // landmark loop: unit u = (a, 32-coordinate part) of the range, two units per pass in
            // alternating buffers; both units of a pass always run (a surplus unit past the table
            // repeats the last one and stores a zero row), so that each prefetch stays where it is
            // issued
            {
                float ta[32], tb[32];
                srow32(ta, tabr);
                float dist = 0.f;
                for (int u = 0; u < units; u += 2) {
                    dist = l1_unit(x + 32 * (u % NCH), ta, tb, tabr + 32 * min(u + 1, units - 1), dist);
                    if (NCH == 1) {
                        sB[u * BP + l] = live ? __builtin_amdgcn_exp2f(dist * kscale) : 0.f;
                        dist = 0.f;
                    }
                    dist = l1_unit(x + 32 * ((u + 1) % NCH), tb, ta, tabr + 32 * min(u + 2, units - 1), dist);
                    const int a = (u + 1) / NCH;   // < 32; a == mh only past the table (zero row)
                    sB[a * BP + l] = (live && a < mh) ? __builtin_amdgcn_exp2f(dist * kscale) : 0.f;
                    dist = 0.f;
                }
                // the last prefetch is consumed here, so that no prefetch is moved next to its use
                asm volatile("" ::"s"(ta[0]), "s"(ta[16]));
            }
            __builtin_amdgcn_wave_barrier();
            // U_part += B [V | 1] over the tile's 64 keys, one 16-row tile of landmarks at a time
#pragma unroll
            for (int rl = 0; rl < 2; ++rl) {
                const int rt = 2 * ri + rl;
                if (16 * rt < mg) {
#pragma unroll
                    for (int s = 0; s < 16; ++s) {
                        const float av = sB[(16 * rl + li) * BP + 4 * s + lk];
#pragma unroll
                        for (int ct = 0; ct < CT - 1; ++ct)
                            acc[rt][ct] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv[s][ct], acc[rt][ct], 0, 0, 0);
                        acc[rt][CT - 1] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, li == 0 ? 1.f : 0.f,
                                                                                 acc[rt][CT - 1], 0, 0, 0);
                    }
                }
            }
            if (Bg && live) {   // the key's row of B for the backward (zeros past m)
                float4* dst = reinterpret_cast<float4*>(Bg + (size_t)j * 64 + 32 * ri);
#pragma unroll 4
                for (int a4 = 0; a4 < 8; ++a4)
                    dst[a4] = make_float4(sB[(4 * a4) * BP + l], sB[(4 * a4 + 1) * BP + l],
                                          sB[(4 * a4 + 2) * BP + l], sB[(4 * a4 + 3) * BP + l]);
            }
            __builtin_amdgcn_wave_barrier();   // the next range overwrites the tile
        }
        if (Bg && live && mg <= 32) {   // no second range: its columns are zeros
            float4* dst = reinterpret_cast<float4*>(Bg + (size_t)j * 64 + 32);
#pragma unroll
            for (int a4 = 0; a4 < 8; ++a4) dst[a4] = make_float4(0.f, 0.f, 0.f, 0.f);
        }
        __builtin_amdgcn_wave_barrier();
    }
    // the value sums over the wave's four key groups (lanes li + 16 lk), the same order in every lane
    if (g == 0) {
#pragma unroll
        for (int ct = 0; ct < CT - 1; ++ct) {
            vsa[ct] += __shfl_xor(vsa[ct], 16, 64);
            vsa[ct] += __shfl_xor(vsa[ct], 32, 64);
        }
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
            if (g == 0 && l < 16) {   // the value sums: row 64 of the buffer
#pragma unroll
                for (int ct = 0; ct < CT - 1; ++ct) {
                    float* p = red + 64 * RP + 16 * ct + li;
                    *p = (ww == 3) ? vsa[ct] : *p + vsa[ct];
                }
            }
        }
    }
    __syncthreads();
    for (int e = tid; e < mg * D1; e += 256) {
        const int a = e / D1, c = e % D1;
        Upart[(((size_t)h * nkc + chunk) * m + lm0 + a) * D1 + c] = red[a * RP + c];
    }
    if (g == 0 && tid < D) vpart[((size_t)h * nkc + chunk) * D + tid] = red[64 * RP + tid];
}

// ------------------------------------------------------------------------------------------
// Newton-Schulz solve, one block of 256 threads per head, matrices padded to MP x MP with zeros
// (the padding stays zero under every update):
//   W = K_LL + eps I,  c = ||W||_1 ||W||_inf,  X0 = W^T / c (X := 0 if c = 0),
//   X_{t+1} = X_t (2I - W X_t);  then U = sum of the key-chunk partials, M = X_T U, and
//   Mc = M[:, :d] - M[:, d] vbar^T (fp64, then rounded), the value part the inline form reads:
//   sum_l a_il Mc_l = Y_i[:d] - s_i vbar without the difference of the two rounded terms.
// Precision: K_LL in fp32 as the key side forms K_LK (exp2 of the code distance times
// -log2(e)/lambda, the distance summed in four fp32 chains); the norms in fp64 (sums of the fp32
// entries, exact up to the spread of their exponents, so the first maximising column and row
// do not depend on the order); the iteration on the fp32 matrix cores; U, M and Mc in fp64.
// With store_all, Xs[h] holds X_0 .. X_T and then W (T + 2 matrices, pitch MP, fp64 copies of the
// fp32 iterates) for the backward.
// Products on the fp32 matrix cores (ns32_mm, ns_mfma.hpp).  X is kept both ways (row-major as A
// of X T, transposed as B of W X) in two alternating buffers, and 2I - W X is written transposed
// (as B of X T): two block barriers per step.
// ---- Pieces of the Newton-Schulz solve shared by ns_solve_kernel and small_forward_kernel, for
// one workgroup of 256 threads and W (MP x MP, zero outside m x m) in LDS with pitch
// ns32_tiles<MP>::P.
//
// Norms: column sums (s < MP) and row sums (s >= MP) of |W| in fp64, each over 256 / (2 MP) parts
// of the index range, then the first maximising column b* and row a* by a lane butterfly; c =
// ||W||_1 ||W||_inf into *sc (LDS) and, when cinfo is given, {c, ||W||_1, ||W||_inf, a* 256 + b*}.
// spart is 256 doubles of LDS, sred 4.  Begins after a barrier that completes W; ends with one.
template <int MP>
__device__ __forceinline__ void ns_norms(const float* sW, double* spart, double* sred, double* sc, double* cinfo) {
    constexpr int P = ns32_tiles<MP>::P;
    const int tid = threadIdx.x;
    {
        constexpr int NPART = 256 / (2 * MP), LEN = MP / NPART;
        const int s = tid % (2 * MP), part = tid / (2 * MP), idx = s % MP;
        double acc[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
        for (int i = 0; i < LEN; ++i) {
            const int ii = part * LEN + i;
            acc[i & 3] += fabs((double)(s < MP ? sW[ii * P + idx] : sW[idx * P + ii]));
        }
        spart[tid] = (acc[0] + acc[1]) + (acc[2] + acc[3]);
    }
    __syncthreads();
    if (tid < 2 * MP) {
        constexpr int NPART = 256 / (2 * MP);
        const int idx = tid % MP;
        double s = 0.0;
#pragma unroll
        for (int p = 0; p < NPART; ++p) s += spart[p * 2 * MP + tid];
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
        *sc = c;
        if (cinfo) {
            cinfo[0] = c;
            cinfo[1] = n1;
            cinfo[2] = ninf;
            cinfo[3] = (double)(as * 256 + bs);
        }
    }
    __syncthreads();
}

// X0 = W^T / c (X := 0 if c = 0) and T updates X <- X (2I - W X) on the fp32 matrix cores: X is
// kept both ways (row-major as A of X T, transposed as B of W X) in two alternating buffers each
// (sX0 + i MSZ, sXT0 + i MSZ), and 2I - W X is written transposed (as B of X T) into sTT: two
// block barriers per step.  With Xh, X_0 .. X_T and then W go there (fp64 copies, pitch MP).
// Returns the buffer holding X_T; ends with a barrier.
template <int MP>
__device__ __forceinline__ const float* ns_direct_steps(const float* sW, float* sX0, float* sXT0, float* sTT, double c,
                                                        int T, double* Xh) {
    using L = ns32_tiles<MP>;
    constexpr int P = L::P;
    constexpr int MSZ = MP * P;
    const size_t mm = (size_t)MP * MP;
    const int tid = threadIdx.x, l = tid & 63, li = l & 15, g = l >> 4;
    // ---- X0 = W^T / c: row-major into X buffer 0, and X0^T = W / c into its transposed buffer
    {
        const double ic = c > 0.0 ? 1.0 / c : 0.0;
        for (int e = tid; e < MP * MP; e += 256) {
            const int a = e / MP, b = e % MP;
            const float wab = sW[a * P + b];
            const float x = (float)((double)wab * ic);   // X0[b][a]
            sX0[b * P + a] = x;
            sXT0[a * P + b] = x;
            if (Xh) {
                Xh[(size_t)b * MP + a] = (double)x;
                Xh[(size_t)(T + 1) * mm + e] = (double)wab;
            }
        }
    }
    __syncthreads();
    // ---- T steps of X <- X (2I - W X)
    for (int t = 0; t < T; ++t) {
        const int cur = t & 1;
        f32x4_t r[L::NT];
        ns32_mm<MP>(sW, sXT0 + cur * MSZ, r);   // W X
#pragma unroll
        for (int i = 0; i < L::NT; ++i) {
            const int row0 = 16 * L::tr(i) + 4 * g, col = 16 * L::tc() + li;
            float4 tv;
            tv.x = (row0 + 0 == col ? 2.f : 0.f) - r[i][0];
            tv.y = (row0 + 1 == col ? 2.f : 0.f) - r[i][1];
            tv.z = (row0 + 2 == col ? 2.f : 0.f) - r[i][2];
            tv.w = (row0 + 3 == col ? 2.f : 0.f) - r[i][3];
            *reinterpret_cast<float4*>(sTT + col * P + row0) = tv;   // (2I - W X)^T
        }
        __syncthreads();
        ns32_mm<MP>(sX0 + cur * MSZ, sTT, r);   // X (2I - W X)
        float* nX = sX0 + (cur ^ 1) * MSZ;
        float* nXT = sXT0 + (cur ^ 1) * MSZ;
#pragma unroll
        for (int i = 0; i < L::NT; ++i) {
            const int row0 = 16 * L::tr(i) + 4 * g, col = 16 * L::tc() + li;
#pragma unroll
            for (int j = 0; j < 4; ++j) nX[(row0 + j) * P + col] = r[i][j];
            *reinterpret_cast<float4*>(nXT + col * P + row0) = make_float4(r[i][0], r[i][1], r[i][2], r[i][3]);
            if (Xh)
#pragma unroll
                for (int j = 0; j < 4; ++j) Xh[(size_t)(t + 1) * mm + (row0 + j) * MP + col] = (double)r[i][j];
        }
        __syncthreads();
    }
    return sX0 + (T & 1) * MSZ;
}

template <int MP, int D>
__global__ __launch_bounds__(256) void ns_solve_kernel(const float* __restrict__ qt, const float* __restrict__ kt,
                                                       const float* __restrict__ Upart,
                                                       const float* __restrict__ vpart,
                                                       double* __restrict__ Xs, double* __restrict__ cinfo,
                                                       float* __restrict__ U, float* __restrict__ M,
                                                       float* __restrict__ Mc, float* __restrict__ vbar, int n,
                                                       int m, int T, double lambda, double eps, int nkc,
                                                       int store_all) {
    using L = ns32_tiles<MP>;
    using SU = ns_tiles<MP, D>;
    constexpr int D1 = D + 1;
    constexpr int P = L::P;
    constexpr int MSZ = MP * P;                  // floats per LDS matrix
    constexpr int P64 = ns_pitch(MP);
    constexpr int PU = ns_pitch(D);
    // fp32 phase: W, X (two buffers), X^T (two buffers), (2I - W X)^T; the query landmark rows
    // are staged after W while W is formed.  fp64 phase (after the iteration): X_T
    // and U's value columns from the start of the same space.
    constexpr int F32 = 6 * MSZ * 4;
    constexpr int F64 = (MP * P64 + MP * PU) * 8;
    __shared__ __attribute__((aligned(16))) char lds[F32 > F64 ? F32 : F64];
    __shared__ double sred[4];
    __shared__ double spart[256];
    __shared__ double su1[MP];
    __shared__ double svb[256];
    __shared__ double sM1[MP];
    __shared__ double svbar[D];
    __shared__ double sc;
    float* const sW = reinterpret_cast<float*>(lds);
    float* const sX0 = sW + MSZ;    // X buffers i = 0, 1 at sX0 + i MSZ
    float* const sXT0 = sW + 3 * MSZ;   // X^T buffers at sXT0 + i MSZ
    float* const sTT = sW + 5 * MSZ;
    const int h = blockIdx.x, tid = threadIdx.x;
    const float* q = qt + (size_t)h * m * D;
    const float* k = kt + (size_t)h * m * D;
    const size_t mm = (size_t)MP * MP;
    double* Xh = Xs + (size_t)h * (store_all ? (T + 2) : 1) * mm;

    // The first CB key chunks of U's partial sums and the key chunks' value sums behind vbar are
    // loaded here and added after the iteration: their latency hides behind it.
    constexpr int NE = (MP * D1 + 255) / 256;
    // (MP = 64 runs one block per CU, so registers are plentiful; MP = 32 keeps them few)
    constexpr int CB = MP == 64 ? (NE > 9 ? 4 : 8) : 2;
    const int ulim = m * D1 - 1;
    float ub[CB][NE];
#pragma unroll
    for (int cc = 0; cc < CB; ++cc) {
        const float* up = Upart + ((size_t)h * nkc + min(cc, nkc - 1)) * m * D1;
#pragma unroll
        for (int r = 0; r < NE; ++r) ub[cc][r] = up[min(tid + 256 * r, ulim)];
    }
    // vbar's 256 / D partial sums per column over the key chunks' value sums (chunks gq, gq + G,
    // ... in order, eight loads in flight), formed here beside the landmark rows' loads and kept
    // in LDS until the end
    constexpr int G = 256 / D;
    {
        const int gq = tid / D, cc = tid % D;
        double vs = 0.0;
        for (int k0 = gq; k0 < nkc; k0 += 8 * G) {
            float v[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) v[i] = k0 + G * i < nkc ? vpart[((size_t)h * nkc + k0 + G * i) * D + cc] : 0.f;
#pragma unroll
            for (int i = 0; i < 8; ++i) vs += (double)v[i];
        }
        svb[tid] = vs;
    }

    // ---- W = K_LL + eps I: thread (a-group, b = tid % MP) keeps the key landmark row b in
    // registers; both landmark tables are staged in LDS first (coalesced loads; the key rows
    // with a pitch of D + 4 floats, so that each lane's 16-byte reads of its own row are free of
    // bank conflicts), the query rows a are read by one or two rows per wave.
    {
        constexpr int KP = D + 4;
        float* sQ = sX0;            // MP x D floats (in the five matrices after W), zero rows past m
        float* sK = sX0 + MP * D;   // MP x KP
        static_assert(MP * (2 * D + 4) <= 5 * MSZ, "the landmark rows fit");
        ns_stage_rows<MP, D>(sQ, q, m * D);
        {
            constexpr int NK = (MP * D / 4 + 255) / 256;
            const int cnt4 = m * D / 4;
            float4 kv[NK];
#pragma unroll
            for (int r = 0; r < NK; ++r)
                kv[r] = reinterpret_cast<const float4*>(k)[min((int)tid + 256 * r, cnt4 - 1)];
#pragma unroll
            for (int r = 0; r < NK; ++r) {
                const int e = tid + 256 * r;
                if (e < MP * D / 4)
                    *reinterpret_cast<float4*>(sK + (e / (D / 4)) * KP + 4 * (e % (D / 4))) =
                        e < cnt4 ? kv[r] : make_float4(0.f, 0.f, 0.f, 0.f);
            }
        }
        const float ks = (float)(-1.4426950408889634 / lambda);
        __syncthreads();
        const int b = tid % MP;
        float kb[D];
#pragma unroll
        for (int c4 = 0; c4 < D / 4; ++c4) {
            const float4 v = *reinterpret_cast<const float4*>(sK + b * KP + 4 * c4);
            kb[4 * c4] = v.x; kb[4 * c4 + 1] = v.y; kb[4 * c4 + 2] = v.z; kb[4 * c4 + 3] = v.w;
        }
#pragma unroll 2
        for (int a = tid / MP; a < MP; a += 256 / MP) {   // two rows per pass: the next row's reads overlap
            const float4* qa = reinterpret_cast<const float4*>(sQ + a * D);
            float d4[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int c4 = 0; c4 < D / 4; ++c4) {
                const float4 v = qa[c4];
                d4[0] += fabsf(v.x - kb[4 * c4]);
                d4[1] += fabsf(v.y - kb[4 * c4 + 1]);
                d4[2] += fabsf(v.z - kb[4 * c4 + 2]);
                d4[3] += fabsf(v.w - kb[4 * c4 + 3]);
            }
            float wv = 0.f;
            if (a < m && b < m) {
                wv = __builtin_amdgcn_exp2f(((d4[0] + d4[1]) + (d4[2] + d4[3])) * ks);
                if (a == b) wv = (float)((double)wv + eps);
            }
            sW[a * P + b] = wv;
        }
    }
    __syncthreads();
    ns_norms<MP>(sW, spart, sred, &sc, cinfo + h * 4);
    const float* sXf = ns_direct_steps<MP>(sW, sX0, sXT0, sTT, sc, T, store_all ? Xh : nullptr);   // X_T
    // ---- U = sum over key chunks (in chunk order) in fp64: the first CB chunks from the early
    // loads, then 2 CB chunks' loads in flight at a time
    double u[NE];
#pragma unroll
    for (int r = 0; r < NE; ++r) u[r] = 0.0;
#pragma unroll
    for (int cc = 0; cc < CB; ++cc)
#pragma unroll
        for (int r = 0; r < NE; ++r)
            if (cc < nkc && tid + 256 * r <= ulim) u[r] += (double)ub[cc][r];
    // the remaining chunks CB2 at a time (registers are free again after the iteration)
    constexpr int CB2 = 2 * CB;
    for (int c0 = CB; c0 < nkc; c0 += CB2) {
        float ub2[CB2][NE];
#pragma unroll
        for (int cc = 0; cc < CB2; ++cc) {
            const float* up = Upart + ((size_t)h * nkc + min(c0 + cc, nkc - 1)) * m * D1;
#pragma unroll
            for (int r = 0; r < NE; ++r) ub2[cc][r] = up[min(tid + 256 * r, ulim)];
        }
#pragma unroll
        for (int cc = 0; cc < CB2; ++cc)
#pragma unroll
            for (int r = 0; r < NE; ++r)
                if (c0 + cc < nkc && tid + 256 * r <= ulim) u[r] += (double)ub2[cc][r];
    }
    // X_T to fp64 (registers first: the fp64 copy overwrites the fp32 buffers)
    constexpr int NX = MP * MP / 256;
    double xv[NX];
#pragma unroll
    for (int r = 0; r < NX; ++r) {
        const int e = tid + 256 * r;
        xv[r] = (double)sXf[(e / MP) * P + e % MP];
        if (!store_all) Xh[e] = xv[r];
    }
    __syncthreads();   // every read of the fp32 buffers is done
    double* sX = reinterpret_cast<double*>(lds);
    double* sU = sX + MP * P64;
#pragma unroll
    for (int r = 0; r < NX; ++r) {
        const int e = tid + 256 * r;
        sX[(e / MP) * P64 + e % MP] = xv[r];
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
    __syncthreads();   // sX, sU, su1 (svb since the start)
    if (tid < m) {
        double s = 0.0;
#pragma unroll 16
        for (int b = 0; b < MP; ++b) s += sX[tid * P64 + b] * su1[b];
        M[((size_t)h * m + tid) * D1 + D] = (float)s;
        sM1[tid] = s;
    }
    if (tid < D) {
        double t = 0.0;
#pragma unroll
        for (int gg = 0; gg < G; ++gg) t += svb[gg * D + tid];
        vbar[(size_t)h * D + tid] = (float)(t / n);
        svbar[tid] = t / n;
    }
    __syncthreads();
    {
        // X_T U (value columns); Mc = M[:, :d] - M[:, d] vbar^T in fp64 for the inline form
        f64x4_t r[SU::NT];
        ns_mm<MP, D, MP, false, false, P64, PU>(sX, sU, r);
#pragma unroll
        for (int i = 0; i < SU::NT; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int a = SU::row(i, j), cc = SU::col(i);
                if (a < m) {
                    M[((size_t)h * m + a) * D1 + cc] = (float)r[i][j];
                    Mc[((size_t)h * m + a) * D + cc] = (float)(r[i][j] - sM1[a] * svbar[cc]);
                }
            }
    }
}

// ------------------------------------------------------------------------------------------
// Query side (fp32 inputs).  grid (ceil(n/256), BH), 256 threads, lane = query (wave w of block
// b covers queries 256 b + 64 w ..).
//   Landmark pass: a_il = k(q_i, kt_l) into the wave's [query][landmark] LDS tile (the landmark
//   rows of kt through scalar registers), 32 landmarks at a time: the tile is 64 x 33 floats per
//   wave, so that three blocks share a compute unit.  s_i = sum_l a_il M[l][d] in fp32 is formed
//   with the contraction, which reads the tile anyway, where the normalisation needs it; the
//   inline form contracts with Mc = M[:, :d] - M[:, d] vbar^T instead: out_i = (A Mc)_i + vbar.
//   Contraction: for each 32-query half, Y^T = M^T A^T on fp32 MFMA 32x32x2 (k = a pair of
//   landmarks).  The B operands of a pair for both halves come from one permlane32 swap of the
//   pair's two tile columns (queries 0..31 keep theirs and receive the other landmark of 32..63
//   and vice versa).  The result holds, per lane, 16 output columns of one query: normalised
//   (Eq. (4) / Eq. (3)) and stored four columns at a time.
// Any m up to 128 (up to four ranges); with Asave, A's rows go to Asave[h][g][n][64] for the
// landmark groups g of 64.
typedef float f32x16_t __attribute__((ext_vector_type(16)));

template <int D, int NORM>
__global__ __launch_bounds__(256) void query_out_kernel(const float* __restrict__ Q, float* __restrict__ Out,
                                                        const float* __restrict__ kt, const float* __restrict__ M,
                                                        const float* __restrict__ Mc,
                                                        const float* __restrict__ vbar,
                                                        const float* __restrict__ extra,
                                                        const float* __restrict__ whiten,
                                                        const float* __restrict__ mvec, float* __restrict__ Asave,
                                                        int H, int n, int m, float kscale) {
    constexpr int D1 = D + 1;
    constexpr int NCH = D / 32;
    constexpr int CB = D / 32;             // 32-column blocks of the output
    constexpr int TP = 33;   // one half (32 landmarks) of the tile and a zero column
    // MFMA A operand of pair s of the current 32-landmark range (staged per range, 4 KB at d = 32,
    // so that four blocks share a compute unit), column block cb: lane j + 32 k holds
    // M[32 hh + 2s + k][32 cb + j]
    __shared__ __attribute__((aligned(16))) float sMT[16 * CB * 64];
    __shared__ float sMo[128];
    __shared__ float sVb[D];
    __shared__ float sMb[NORM == NORM_MSPACE ? D : 1];
    __shared__ float sT[4 * 64 * TP];
    const int h = blockIdx.y, tid = threadIdx.x, w = tid >> 6, l = tid & 63;
    const int ng = (m + 63) / 64;   // landmark groups of the saved rows
    // landmark-space normalisation: the rows of M scaled by the whitening w, the ones column
    // replaced by 1/m (so that s_i becomes the landmark mean of a_i), and the vectors
    // sum_l w_l M_l and (1/m) sum_l M_l from mvec
    const float* wl = (NORM == NORM_MSPACE && whiten) ? whiten + (size_t)(h % H) * m : nullptr;
    auto stage = [&](int hh) {
        for (int e = tid; e < 16 * CB * 64; e += 256) {
            const int s = 16 * hh + e / (CB * 64), cb = (e / 64) % CB, ln = e % 64;
            const int lm = 2 * s + ln / 32;
            const float wv = wl && lm < m ? wl[lm] : 1.f;
            const float* src = NORM == NORM_INLINE ? Mc + ((size_t)h * m + lm) * D : M + ((size_t)h * m + lm) * D1;
            sMT[e] = (lm < m) ? wv * src[32 * cb + ln % 32] : 0.f;
        }
    };
    if (tid < 128) {
        if (NORM == NORM_MSPACE) sMo[tid] = (tid < m) ? 1.f / (float)m : 0.f;
        else sMo[tid] = (tid < m) ? M[((size_t)h * m + tid) * D1 + D] : 0.f;
    }
    if (NORM == NORM_MSPACE) {
        if (tid < D) {
            sVb[tid] = mvec[(size_t)h * 2 * D + tid];
            sMb[tid] = mvec[(size_t)h * 2 * D + D + tid];
        }
    } else if (tid < D) {
        sVb[tid] = vbar[(size_t)h * D + tid];
    }
    float* tile = sT + w * 64 * TP;
    const int i0 = blockIdx.x * 256 + w * 64;
    const int i = i0 + l;
    const bool live = i < n;
    float q[D];
    {
        const float4* qr = reinterpret_cast<const float4*>(Q + ((size_t)h * n + (live ? i : n - 1)) * D);
#pragma unroll
        for (int c4 = 0; c4 < D / 4; ++c4) {
            const float4 v = qr[c4];
            q[4 * c4 + 0] = v.x; q[4 * c4 + 1] = v.y; q[4 * c4 + 2] = v.z; q[4 * c4 + 3] = v.w;
        }
    }
    __syncthreads();   // sMT, sMo, sVb
    f32x16_t acc[2][CB];
#pragma unroll
    for (int qb = 0; qb < 2; ++qb)
#pragma unroll
        for (int cb = 0; cb < CB; ++cb)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[qb][cb][r] = 0.f;
    float s = 0.f;   // s_i = sum_l a_il M[l][d], in landmark order
    for (int hh = 0; 32 * hh < m; ++hh) {
        const int mh = min(32, m - 32 * hh);   // landmarks 32 hh .. 32 hh + mh - 1
        const float* tab = kt + __builtin_amdgcn_readfirstlane((h * m + 32 * hh) * D);   // wave-uniform: scalar loads
        const int units = mh * NCH;
        // no LDS reads in this loop: a wait for one would also wait for the row prefetch
        auto emit = [&](int a, float dist) {   // a == mh only past the table: a zero column
            tile[l * TP + a] = (live && a < mh) ? __builtin_amdgcn_exp2f(dist * kscale) : 0.f;
        };
        {
            float ta[32], tb[32];
            srow32(ta, tab);
            float dist = 0.f;
            for (int u = 0; u < units; u += 2) {
                dist = l1_unit(q + 32 * (u % NCH), ta, tb, tab + 32 * min(u + 1, units - 1), dist);
                if (NCH == 1) {
                    emit(u, dist);
                    dist = 0.f;
                }
                dist = l1_unit(q + 32 * ((u + 1) % NCH), tb, ta, tab + 32 * min(u + 2, units - 1), dist);
                emit((u + 1) / NCH, dist);
                dist = 0.f;
            }
            asm volatile("" ::"s"(ta[0]), "s"(ta[16]));
        }
        if (mh & 1) tile[l * TP + mh] = 0.f;   // the pair loop reads column mh (unwritten when d = 64)
        __builtin_amdgcn_wave_barrier();
        if (Asave)   // A's rows for the backward, group-major: Asave[h][g][n][64], g = landmark / 64
            store_half_rows(Asave + (size_t)(h * ng + (hh >> 1)) * n * 64, tile, i0, n, 32 * (hh & 1), mh);
        const int npair = (mh + 1) / 2;
        __syncthreads();   // the last range's operands are read by every wave
        stage(hh);
        __syncthreads();
#pragma unroll 2
        for (int pl = 0; pl < npair; ++pl) {
            const int p = 16 * hh + pl;   // landmark pair of the whole tile
            const float x0 = tile[l * TP + 2 * pl], x1 = tile[l * TP + 2 * pl + 1];
            if (NORM == NORM_ROWSUM || NORM == NORM_MSPACE) s = fmaf(x1, sMo[2 * p + 1], fmaf(x0, sMo[2 * p], s));
            const auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x0), __float_as_uint(x1), false, false);
#pragma unroll
            for (int cb = 0; cb < CB; ++cb) {
                const float av = sMT[(pl * CB + cb) * 64 + l];
#pragma unroll
                for (int qb = 0; qb < 2; ++qb)
                    acc[qb][cb] =
                        __builtin_amdgcn_mfma_f32_32x32x2f32(av, __uint_as_float(b[qb]), acc[qb][cb], 0, 0, 0);
            }
        }
        __builtin_amdgcn_wave_barrier();   // the next half overwrites the tile
    }
    // result register r at lane l: column 8 (r / 4) + 4 (l / 32) + r % 4 of the block, query l % 32
    // of the half; s_i of that query from the same swap
    const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(s), __float_as_uint(s), false, false);
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
        const int iq = i0 + 32 * qb + (l & 31);
        const float si = __uint_as_float(sw[qb]);
        if (iq < n) {
            float* orow = Out + ((size_t)h * n + iq) * D;
#pragma unroll
            for (int cb = 0; cb < CB; ++cb)
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const int c0 = 32 * cb + 8 * g + 4 * (l >> 5);
                    float o[4];
#pragma unroll
                    for (int t = 0; t < 4; ++t) {
                        const float y = acc[qb][cb][4 * g + t];
                        if (NORM == NORM_INLINE) o[t] = y + sVb[c0 + t];   // y = Y[:d] - s vbar (Mc)
                        else if (NORM == NORM_ROWSUM) o[t] = y / si;
                        else if (NORM == NORM_MSPACE) o[t] = fmaf(-si, sVb[c0 + t], y) + sMb[c0 + t];
                        else o[t] = y;
                    }
                    if (extra) {   // the convolution branch of Eq. (7)
                        const float4 ex = *reinterpret_cast<const float4*>(extra + ((size_t)h * n + iq) * D + c0);
                        o[0] += ex.x;
                        o[1] += ex.y;
                        o[2] += ex.z;
                        o[3] += ex.w;
                    }
                    *reinterpret_cast<float4*>(orow + c0) = make_float4(o[0], o[1], o[2], o[3]);
                }
        }
    }
}

// ------------------------------------------------------------------------------------------
// Launch wrappers.

static inline float kscale_of(float lambda) { return (float)(-1.4426950408889634 / (double)lambda); }

int pool_split(int BH, int n, int m) {
    const int per = n / m;   // tokens per landmark (segments: this or one more; windows: exactly)
    int S = 1;
    while (S < kPoolMaxSplit && (long long)m * BH * S < 512 && per / (2 * S) >= 64) S *= 2;
    return S;
}

hipError_t launch_pool(int dt, const void* Q, const void* K, float* qt, float* kt, double* part, int BH, int n, int d,
                       int m, LmPool pl, hipStream_t st) {
    const int most = pl.r > 0 ? pl.r * pl.r : (n + m - 1) / m;   // tokens of the largest landmark
    if (most <= kPoolSmall) {
        const dim3 grid((m + 256 / d - 1) / (256 / d), BH);
        if (dt == DT_F32)
            hipLaunchKernelGGL(pool_small_kernel<DT_F32>, grid, dim3(256), 0, st, (const float*)Q, (const float*)K,
                               qt, kt, n, d, m, pl);
        else
            hipLaunchKernelGGL(pool_small_kernel<DT_BF16>, grid, dim3(256), 0, st, (const uint16_t*)Q,
                               (const uint16_t*)K, qt, kt, n, d, m, pl);
        return hipGetLastError();
    }
    const int S = pool_split(BH, n, m);
    dim3 grid(m * S, BH);
    if (dt == DT_F32)
        hipLaunchKernelGGL(pool_kernel<DT_F32>, grid, dim3(256), 0, st, (const float*)Q, (const float*)K, qt, kt,
                           part, n, d, m, S, pl);
    else
        hipLaunchKernelGGL(pool_kernel<DT_BF16>, grid, dim3(256), 0, st, (const uint16_t*)Q, (const uint16_t*)K, qt, kt,
                           part, n, d, m, S, pl);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || S == 1) return e;
    hipLaunchKernelGGL(pool_combine_kernel, dim3(m, BH), dim3((2 * d + 63) / 64 * 64), 0, st, part, qt, kt, n, d, m,
                       S, pl);
    return hipGetLastError();
}

hipError_t launch_key_summary(int dt, const void* K, const void* V, const float* qt, float* Upart, float* vpart,
                              float* Bsave, int BH, int n, int d, int m, float lambda, int chunk_keys, int nkc,
                              hipStream_t st) {
    if (dt != DT_F32) return hipErrorInvalidValue;   // bf16 inputs take the fast path
    const float ks = kscale_of(lambda);
    if (d == 32)
        hipLaunchKernelGGL((key_summary_kernel<32>), dim3(nkc, BH, (m + 63) / 64), dim3(256), 0, st, (const float*)K,
                           (const float*)V, qt, Upart, vpart, Bsave, n, m, ks, chunk_keys, nkc);
    else
        hipLaunchKernelGGL((key_summary_kernel<64>), dim3(nkc, BH, (m + 63) / 64), dim3(256), 0, st, (const float*)K,
                           (const float*)V, qt, Upart, vpart, Bsave, n, m, ks, chunk_keys, nkc);
    return hipGetLastError();
}

hipError_t launch_ns_solve(const float* qt, const float* kt, const float* Upart, const float* vpart, double* Xs,
                           double* cinfo, float* U, float* M, float* Mc, float* vbar, int BH, int n, int d, int m, int T,
                           double lambda, double eps, int nkc, int store_all, int MP, hipStream_t st) {
#define LAPATTN_NS(MPv, Dv)                                                                                  \
    hipLaunchKernelGGL((ns_solve_kernel<MPv, Dv>), dim3(BH), dim3(256), 0, st, qt, kt, Upart, vpart, Xs, cinfo, \
                       U, M, Mc, vbar, n, m, T, lambda, eps, nkc, store_all)
    if (MP == 32 && d == 32) LAPATTN_NS(32, 32);
    else if (MP == 32) LAPATTN_NS(32, 64);
    else if (d == 32) LAPATTN_NS(64, 32);
    else LAPATTN_NS(64, 64);
#undef LAPATTN_NS
    return hipGetLastError();
}

template <int D>
static void query_out_launch(int norm, const void* Q, void* Out, const float* kt, const float* M, const float* Mc,
                             const float* vbar,
                             const float* extra, const float* whiten, const float* mvec, float* Asave, int BH, int H,
                             int n, int m, float kscale, hipStream_t st) {
    dim3 grid((n + 255) / 256, BH);
    const float* q = (const float*)Q;
    float* o = (float*)Out;
#define LAPATTN_QO(Nv)                                                                                             \
    hipLaunchKernelGGL((query_out_kernel<D, Nv>), grid, dim3(256), 0, st, q, o, kt, M, Mc, vbar, extra, whiten, mvec, \
                       Asave, H, n, m, kscale)
    if (norm == NORM_INLINE) LAPATTN_QO(NORM_INLINE);
    else if (norm == NORM_ROWSUM) LAPATTN_QO(NORM_ROWSUM);
    else if (norm == NORM_MSPACE) LAPATTN_QO(NORM_MSPACE);
    else LAPATTN_QO(NORM_NONE);
#undef LAPATTN_QO
}

hipError_t launch_query_out(int dt, int norm, const void* Q, void* Out, const float* kt, const float* M,
                            const float* Mc, const float* vbar, const float* extra, const float* whiten, const float* mvec,
                            float* Asave, int BH, int H, int n, int d, int m, float lambda, hipStream_t st) {
    if (dt != DT_F32) return hipErrorInvalidValue;   // bf16 inputs take the fast path
    const float ks = kscale_of(lambda);
    if (d == 32) query_out_launch<32>(norm, Q, Out, kt, M, Mc, vbar, extra, whiten, mvec, Asave, BH, H, n, m, ks, st);
    else query_out_launch<64>(norm, Q, Out, kt, M, Mc, vbar, extra, whiten, mvec, Asave, BH, H, n, m, ks, st);
    return hipGetLastError();
}

// ------------------------------------------------------------------------------------------
// Small heads (fp32 inputs, n <= 256 tokens, m <= 32 landmarks): the whole forward of one head in
// one workgroup of 256 threads, every intermediate in LDS -- one launch instead of four, where
// each of those would run a few waves per head and wait on its own latency chains (the
// DeiT-small shape: 197 tokens, 32 landmarks).
//
// L1 distances in fixed point (fcode, common.hpp): K_LL (Eq. (9)), B and A (Eq. (8)) are all
// formed from the head's codes with one v_sad_u32 per coordinate and the same exponential, so a
// query equal to a landmark mean gives exactly that row of K_LL (m = n reproduces dense attention
// through X = W^-1).  A non-finite value in Q or K makes every output of the head NaN.
//
// Steps:
//   pool     thread (landmark a = t / 8, columns (t % 8) D/8 ..): the landmark means in fp64,
//            rounded once; R by a block maximum; the means coded into LDS;
//   K_LL     thread (a = t / 8, b = 4 (t % 8) ..): four sad chains;
//   solve    ns_norms, ns_direct_steps (MP = 32), X_T copied aside;
//   key side thread t: keys t % 128 and t % 128 + 128 against the 16 landmarks of half t / 128
//            (each LDS broadcast of a landmark word serves two keys), B[a][j] into a [32][256]
//            tile; then wave w contracts keys 64 w .. 64 w + 63 with [V | 1] on fp32 MFMA 16x16x4
//            (the V rows loaded together, their fp64 column sums giving vbar) and the four
//            waves' partials are added in a fixed order;
//   M        M = X_T U in fp64 (ns_mm), Mc = M[:, :d] - M[:, d] vbar^T for the inline form;
//   query    thread t: queries t % 128, t % 128 + 128 against half t / 128 of the landmarks, A
//            into a [256][33] tile (and the two halves of s_i for the row sums); then
//            Y = A M on fp32 MFMA, normalised (Eq. (4) / Eq. (3)) and stored.

// Coded L1 distances of two tokens (codes x0, x1) to rows 0 .. na - 1 of an LDS code table
// (pitch LP words); emit(aa, dist0, dist1) per row.  The rows are read as half rows of D / 8
// 16-byte words into two buffers: the reads of the next half row are issued before the sads of
// the current one, so that D / 8 reads are always in flight (one or two waves per SIMD leave
// the LDS latency to the wave itself).  Each word serves both tokens.  na is wave-uniform.
template <int D, int LP, class Emit>
__device__ __forceinline__ void sf_dist2(const uint32_t* __restrict__ tab, int na, const uint32_t (&x0)[D],
                                         const uint32_t (&x1)[D], Emit&& emit) {
    constexpr int H = D / 8;
    if (na <= 0) return;
    uint4 cur[H], nxt[H];
#pragma unroll
    for (int q = 0; q < H; ++q) cur[q] = reinterpret_cast<const uint4*>(tab)[q];
    for (int aa = 0; aa < na; ++aa) {
        const uint4* r = reinterpret_cast<const uint4*>(tab + aa * LP);
#pragma unroll
        for (int q = 0; q < H; ++q) nxt[q] = r[H + q];
        __builtin_amdgcn_sched_barrier(0);
        uint32_t u0 = 0u, w0 = 0u, u1 = 0u, w1 = 0u;
#pragma unroll
        for (int q = 0; q < H; ++q) {
            const uint4 v = cur[q];
            u0 = sad32(x0[4 * q], v.x, u0); w0 = sad32(x0[4 * q + 1], v.y, w0);
            u1 = sad32(x1[4 * q], v.x, u1); w1 = sad32(x1[4 * q + 1], v.y, w1);
            u0 = sad32(x0[4 * q + 2], v.z, u0); w0 = sad32(x0[4 * q + 3], v.w, w0);
            u1 = sad32(x1[4 * q + 2], v.z, u1); w1 = sad32(x1[4 * q + 3], v.w, w1);
        }
        __builtin_amdgcn_sched_barrier(0);
        const uint4* rn = reinterpret_cast<const uint4*>(tab + min(aa + 1, na - 1) * LP);
#pragma unroll
        for (int q = 0; q < H; ++q) cur[q] = rn[q];
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int q = 0; q < H; ++q) {
            const uint4 v = nxt[q];
            const int c = 4 * (H + q);
            u0 = sad32(x0[c], v.x, u0); w0 = sad32(x0[c + 1], v.y, w0);
            u1 = sad32(x1[c], v.x, u1); w1 = sad32(x1[c + 1], v.y, w1);
            u0 = sad32(x0[c + 2], v.z, u0); w0 = sad32(x0[c + 3], v.w, w0);
            u1 = sad32(x1[c + 2], v.z, u1); w1 = sad32(x1[c + 3], v.w, w1);
        }
        __builtin_amdgcn_sched_barrier(0);
        emit(aa, u0 + w0, u1 + w1);
    }
}

template <int D, int NORM>
__global__ __launch_bounds__(256, 2) void small_forward_kernel(const float* __restrict__ Q, const float* __restrict__ K,
                                                               const float* __restrict__ V, float* __restrict__ Out,
                                                               int n, int m, double lambda, int T, double eps,
                                                               LmPool pl) {
    constexpr int MP = 32;
    using L = ns32_tiles<MP>;
    using SU = ns_tiles<MP, D>;
    constexpr int P = L::P;               // pitch of the solve's fp32 matrices
    constexpr int MSZ = MP * P;
    constexpr int LP = D + 4;             // pitch of the landmark code rows and of M
    constexpr int BP = 256 + 4;           // pitch of the key tile [a][j]
    constexpr int AP = 33;                // pitch of the query tile [i][l]
    constexpr int P64 = ns_pitch(MP);
    constexpr int PU = ns_pitch(D);
    constexpr int CT = D / 16 + 1;        // key-side column tiles: the values, then the ones column
    constexpr int RP = 16 * CT;           // pitch of the key-side partial being reduced
    constexpr int R1 = 6 * MSZ * 4, R2 = MP * BP * 4, R3 = 256 * AP * 4, R4 = (MP * P64 + MP * PU) * 8;
    constexpr int R5 = MP * RP * 4;
    constexpr int RB = R1 > R2 ? (R1 > R3 ? (R1 > R4 ? R1 : R4) : (R3 > R4 ? R3 : R4))
                               : (R2 > R3 ? (R2 > R4 ? R2 : R4) : (R3 > R4 ? R3 : R4));
    static_assert(R5 <= RB, "the key-side partial fits the shared region");
    __shared__ __attribute__((aligned(16))) uint32_t sQc[MP * LP];   // coded landmark means
    __shared__ __attribute__((aligned(16))) uint32_t sKc[MP * LP];
    __shared__ __attribute__((aligned(16))) char reg[RB];   // solve / key tile / partial / M / query tile
    __shared__ __attribute__((aligned(16))) float sXT[MSZ];
    __shared__ __attribute__((aligned(16))) float sMv[MP * LP];
    __shared__ float sM1[MP];
    __shared__ float sS[2][256];
    __shared__ float smx[4];
    __shared__ double spart[256];
    __shared__ double sred[4];
    __shared__ double sc;
    __shared__ double svp[4][D];
    __shared__ double svb[D];
    __shared__ double su1[MP];
    __shared__ double sM1d[MP];
    const int h = blockIdx.x, tid = threadIdx.x, w = tid >> 6, l = tid & 63, li = l & 15, lk = l >> 4;
    const int hf = tid >> 7, t0 = tid & 127;   // key / query sides: landmark half, first token
    const float* Qh = Q + (size_t)h * n * D;
    const float* Kh = K + (size_t)h * n * D;
    const float* Vh = V + (size_t)h * n * D;

    // ---- landmark means, R = max |x| (infinite when a mean is not finite), the codes
    constexpr int CPT = D / 8;   // columns per thread
    float qm[CPT], km[CPT];
    {
        const int a = tid >> 3, c0 = (tid & 7) * CPT;
        double sq[CPT], sk[CPT];
#pragma unroll
        for (int c = 0; c < CPT; ++c) sq[c] = sk[c] = 0.0;
        float mx = 0.f;
        int cnt = 1;
        if (a < m) {
            const LmTokens tok = lm_tokens(pl, a, n, m);
            cnt = tok.count;
#pragma unroll 4
            for (int t = 0; t < tok.count; ++t) {
                const size_t o = (size_t)tok(t) * D + c0;
#pragma unroll
                for (int c4 = 0; c4 < CPT / 4; ++c4) {
                    const float4 qv = *reinterpret_cast<const float4*>(Qh + o + 4 * c4);
                    const float4 kv = *reinterpret_cast<const float4*>(Kh + o + 4 * c4);
                    sq[4 * c4] += qv.x; sq[4 * c4 + 1] += qv.y; sq[4 * c4 + 2] += qv.z; sq[4 * c4 + 3] += qv.w;
                    sk[4 * c4] += kv.x; sk[4 * c4 + 1] += kv.y; sk[4 * c4 + 2] += kv.z; sk[4 * c4 + 3] += kv.w;
                    mx = fmaxf(mx, fmaxf(fmaxf(fabsf(qv.x), fabsf(qv.y)), fmaxf(fabsf(qv.z), fabsf(qv.w))));
                    mx = fmaxf(mx, fmaxf(fmaxf(fabsf(kv.x), fabsf(kv.y)), fmaxf(fabsf(kv.z), fabsf(kv.w))));
                }
            }
        }
        bool fin = true;
#pragma unroll
        for (int c = 0; c < CPT; ++c) {
            qm[c] = a < m ? (float)(sq[c] / (double)cnt) : 0.f;
            km[c] = a < m ? (float)(sk[c] / (double)cnt) : 0.f;
            fin = fin && isfinite(qm[c]) && isfinite(km[c]);
        }
        // a NaN or infinite input leaves its landmark mean non-finite (fmaxf alone would skip a NaN)
        if (!fin) mx = __builtin_inff();
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off, 64));
        if (l == 0) smx[w] = mx;
    }
    __syncthreads();
    const float R = fmaxf(fmaxf(smx[0], smx[1]), fmaxf(smx[2], smx[3]));
    const bool nan_head = !(R <= 3.4028234663852886e38f);
    float s, kss;
    fgrid(nan_head ? 1.f : R, (float)(-1.4426950408889634 / lambda), s, kss);
    {
        const int a = tid >> 3, c0 = (tid & 7) * CPT;
#pragma unroll
        for (int c = 0; c < CPT; ++c) {
            sQc[a * LP + c0 + c] = fcode(qm[c], s);
            sKc[a * LP + c0 + c] = fcode(km[c], s);
        }
    }
    __syncthreads();
    // ---- W = K_LL + eps I (zero outside m x m)
    float* const sW = reinterpret_cast<float*>(reg);
    float* const sX0 = sW + MSZ;
    float* const sXT0 = sW + 3 * MSZ;
    float* const sTT = sW + 5 * MSZ;
    {
        const int a = tid >> 3, b0 = 4 * (tid & 7);
        uint32_t u[4] = {0u, 0u, 0u, 0u};
#pragma unroll 4
        for (int c4 = 0; c4 < D / 4; ++c4) {
            const uint4 v = *reinterpret_cast<const uint4*>(sQc + a * LP + 4 * c4);
#pragma unroll
            for (int bb = 0; bb < 4; ++bb) {
                const uint4 kb = *reinterpret_cast<const uint4*>(sKc + (b0 + bb) * LP + 4 * c4);
                u[bb] = sad32(v.x, kb.x, u[bb]);
                u[bb] = sad32(v.y, kb.y, u[bb]);
                u[bb] = sad32(v.z, kb.z, u[bb]);
                u[bb] = sad32(v.w, kb.w, u[bb]);
            }
        }
#pragma unroll
        for (int bb = 0; bb < 4; ++bb) {
            const int b = b0 + bb;
            float wv = 0.f;
            if (a < m && b < m) {
                wv = fkval(u[bb], kss);
                if (a == b) wv = (float)((double)wv + eps);
            }
            sW[a * P + b] = wv;
        }
    }
    __syncthreads();
    // ---- Algorithm 2
    ns_norms<MP>(sW, spart, sred, &sc, nullptr);
    {
        const float* sXf = ns_direct_steps<MP>(sW, sX0, sXT0, sTT, sc, T, nullptr);
        for (int e = tid; e < MSZ; e += 256) sXT[e] = sXf[e];
    }
    __syncthreads();   // the solve's buffers are free
    // ---- key side: B[a][j] = k(qt_a, k_j), then U = B [V | 1]
    float* const sB = reinterpret_cast<float*>(reg);
    {
        uint32_t x0[D], x1[D];
        {
            const float4* r0 = reinterpret_cast<const float4*>(Kh + (size_t)min(t0, n - 1) * D);
            const float4* r1 = reinterpret_cast<const float4*>(Kh + (size_t)min(t0 + 128, n - 1) * D);
#pragma unroll
            for (int c4 = 0; c4 < D / 4; ++c4) {
                const float4 v0 = r0[c4], v1 = r1[c4];
                x0[4 * c4] = fcode(v0.x, s); x0[4 * c4 + 1] = fcode(v0.y, s);
                x0[4 * c4 + 2] = fcode(v0.z, s); x0[4 * c4 + 3] = fcode(v0.w, s);
                x1[4 * c4] = fcode(v1.x, s); x1[4 * c4 + 1] = fcode(v1.y, s);
                x1[4 * c4 + 2] = fcode(v1.z, s); x1[4 * c4 + 3] = fcode(v1.w, s);
            }
        }
        const bool live0 = t0 < n, live1 = t0 + 128 < n;
        const int na = __builtin_amdgcn_readfirstlane(min(max(m - 16 * hf, 0), 16));
        sf_dist2<D, LP>(sQc + 16 * hf * LP, na, x0, x1, [&](int aa, uint32_t d0, uint32_t d1) {
            const int a = 16 * hf + aa;
            sB[a * BP + t0] = live0 ? fkval(d0, kss) : 0.f;
            sB[a * BP + t0 + 128] = live1 ? fkval(d1, kss) : 0.f;
        });
        for (int a = 16 * hf + na; a < 16 * hf + 16; ++a) {   // landmarks past m
            sB[a * BP + t0] = 0.f;
            sB[a * BP + t0 + 128] = 0.f;
        }
    }
    // wave w's operands: V rows of keys 64 w + 4 s + lk (clamped past n: their B columns are 0)
    float vv[16][CT - 1];
#pragma unroll
    for (int s4 = 0; s4 < 16; ++s4) {
        const float* vr = Vh + (size_t)min(64 * w + 4 * s4 + lk, n - 1) * D;
#pragma unroll
        for (int ct = 0; ct < CT - 1; ++ct) vv[s4][ct] = vr[16 * ct + li];
    }
    // vbar: this lane's live keys in fp64, then the four key groups of the wave (a butterfly);
    // the waves' sums are added in order 0..3 after the next barrier
    {
        double vs[CT - 1];
#pragma unroll
        for (int ct = 0; ct < CT - 1; ++ct) vs[ct] = 0.0;
#pragma unroll
        for (int s4 = 0; s4 < 16; ++s4)
            if (64 * w + 4 * s4 + lk < n)
#pragma unroll
                for (int ct = 0; ct < CT - 1; ++ct) vs[ct] += (double)vv[s4][ct];
#pragma unroll
        for (int ct = 0; ct < CT - 1; ++ct) {
            vs[ct] += __shfl_xor(vs[ct], 16, 64);
            vs[ct] += __shfl_xor(vs[ct], 32, 64);
            if (lk == 0) svp[w][16 * ct + li] = vs[ct];
        }
    }
    __syncthreads();   // B complete (a wave's keys were formed by two waves)
    f32x4_t acc[2][CT];
#pragma unroll
    for (int rt = 0; rt < 2; ++rt)
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) acc[rt][ct] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s4 = 0; s4 < 16; ++s4) {
        const int jr = 64 * w + 4 * s4 + lk;
#pragma unroll
        for (int rt = 0; rt < 2; ++rt) {
            const float av = sB[(16 * rt + li) * BP + jr];
#pragma unroll
            for (int ct = 0; ct < CT - 1; ++ct) acc[rt][ct] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, vv[s4][ct], acc[rt][ct], 0, 0, 0);
            acc[rt][CT - 1] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, li == 0 ? 1.f : 0.f, acc[rt][CT - 1], 0, 0, 0);
        }
    }
    if (tid < D) svb[tid] = (((svp[0][tid] + svp[1][tid]) + svp[2][tid]) + svp[3][tid]) / n;
    // the four waves' partials added in the order 3, 2, 1, 0 (register r of a 16x16x4 tile at
    // lane l: row 4 (l / 16) + r, column l % 16)
    float* const red = reinterpret_cast<float*>(reg);
    for (int ww = 3; ww >= 0; --ww) {
        __syncthreads();   // (first pass: every wave is done with the key tile)
        if (w == ww) {
#pragma unroll
            for (int rt = 0; rt < 2; ++rt)
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
    // ---- M = X_T U in fp64 (the partial and X_T through registers: fp64 copies replace them)
    constexpr int NU = (MP * (D + 1) + 255) / 256;
    double uv[NU];
#pragma unroll
    for (int r = 0; r < NU; ++r) {
        const int e = tid + 256 * r;
        uv[r] = e < MP * (D + 1) ? (double)red[(e / (D + 1)) * RP + e % (D + 1)] : 0.0;
    }
    __syncthreads();
    double* const sX64 = reinterpret_cast<double*>(reg);
    double* const sU64 = sX64 + MP * P64;
#pragma unroll
    for (int r = 0; r < NU; ++r) {
        const int e = tid + 256 * r;
        if (e < MP * (D + 1)) {
            const int a = e / (D + 1), c = e % (D + 1);
            if (c < D) sU64[a * PU + c] = uv[r];
            else su1[a] = uv[r];
        }
    }
    for (int e = tid; e < MP * MP; e += 256) sX64[(e / MP) * P64 + e % MP] = (double)sXT[(e / MP) * P + e % MP];
    __syncthreads();
    if (tid < MP) {
        double sacc = 0.0;
#pragma unroll 8
        for (int b = 0; b < MP; ++b) sacc += sX64[tid * P64 + b] * su1[b];
        sM1d[tid] = sacc;
        sM1[tid] = (float)sacc;
    }
    __syncthreads();
    {
        f64x4_t r[SU::NT];
        ns_mm<MP, D, MP, false, false, P64, PU>(sX64, sU64, r);
#pragma unroll
        for (int i = 0; i < SU::NT; ++i)
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) {
                const int a = SU::row(i, jj), cc = SU::col(i);
                sMv[a * LP + cc] = NORM == NORM_INLINE ? (float)(r[i][jj] - sM1d[a] * svb[cc]) : (float)r[i][jj];
            }
    }
    __syncthreads();   // sMv, sM1; the shared region is free
    // ---- query side: A[i][l] = k(q_i, kt_l) and the halves of s_i, then Y = A M
    float* const sA = reinterpret_cast<float*>(reg);
    {
        uint32_t x0[D], x1[D];
        {
            const float4* r0 = reinterpret_cast<const float4*>(Qh + (size_t)min(t0, n - 1) * D);
            const float4* r1 = reinterpret_cast<const float4*>(Qh + (size_t)min(t0 + 128, n - 1) * D);
#pragma unroll
            for (int c4 = 0; c4 < D / 4; ++c4) {
                const float4 v0 = r0[c4], v1 = r1[c4];
                x0[4 * c4] = fcode(v0.x, s); x0[4 * c4 + 1] = fcode(v0.y, s);
                x0[4 * c4 + 2] = fcode(v0.z, s); x0[4 * c4 + 3] = fcode(v0.w, s);
                x1[4 * c4] = fcode(v1.x, s); x1[4 * c4 + 1] = fcode(v1.y, s);
                x1[4 * c4 + 2] = fcode(v1.z, s); x1[4 * c4 + 3] = fcode(v1.w, s);
            }
        }
        const bool live0 = t0 < n, live1 = t0 + 128 < n;
        float sr0 = 0.f, sr1 = 0.f;
        const int na = __builtin_amdgcn_readfirstlane(min(max(m - 16 * hf, 0), 16));
        sf_dist2<D, LP>(sKc + 16 * hf * LP, na, x0, x1, [&](int aa, uint32_t d0, uint32_t d1) {
            const int a = 16 * hf + aa;
            const float a0 = live0 ? fkval(d0, kss) : 0.f;
            const float a1 = live1 ? fkval(d1, kss) : 0.f;
            if (NORM == NORM_ROWSUM) {
                sr0 = fmaf(a0, sM1[a], sr0);
                sr1 = fmaf(a1, sM1[a], sr1);
            }
            sA[t0 * AP + a] = a0;
            sA[(t0 + 128) * AP + a] = a1;
        });
        for (int a = 16 * hf + na; a < 16 * hf + 16; ++a) {   // landmarks past m
            sA[t0 * AP + a] = 0.f;
            sA[(t0 + 128) * AP + a] = 0.f;
        }
        if (NORM == NORM_ROWSUM) {
            sS[hf][t0] = sr0;
            sS[hf][t0 + 128] = sr1;
        }
    }
    __syncthreads();   // A complete (a query's landmarks were formed by two waves)
    {
        constexpr int NCT = D / 16;
        f32x4_t y[4][NCT];
#pragma unroll
        for (int rt = 0; rt < 4; ++rt)
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) y[rt][ct] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s4 = 0; s4 < MP / 4; ++s4) {
            const int kl = 4 * s4 + lk;   // landmark
            float bv[NCT];
#pragma unroll
            for (int ct = 0; ct < NCT; ++ct) bv[ct] = sMv[kl * LP + 16 * ct + li];
#pragma unroll
            for (int rt = 0; rt < 4; ++rt) {
                const float av = sA[(64 * w + 16 * rt + li) * AP + kl];
#pragma unroll
                for (int ct = 0; ct < NCT; ++ct) y[rt][ct] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv[ct], y[rt][ct], 0, 0, 0);
            }
        }
        const float nanv = nan_head ? __builtin_nanf("") : 0.f;   // added: NaN for the whole head
#pragma unroll
        for (int rt = 0; rt < 4; ++rt)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int i = 64 * w + 16 * rt + 4 * lk + r;
                if (i < n) {
                    const float inv_s = NORM == NORM_ROWSUM ? 1.f / (sS[0][i] + sS[1][i]) : 1.f;
#pragma unroll
                    for (int ct = 0; ct < NCT; ++ct) {
                        const int c = 16 * ct + li;
                        float o = y[rt][ct][r];
                        if (NORM == NORM_INLINE) o += (float)svb[c];
                        else if (NORM == NORM_ROWSUM) o *= inv_s;
                        Out[((size_t)h * n + i) * D + c] = o + nanv;
                    }
                }
            }
    }
}

hipError_t launch_small_forward(int norm, const float* Q, const float* K, const float* V, float* Out, int BH, int n,
                                int d, int m, float lambda, int T, float eps, LmPool pl, hipStream_t st) {
#define LAPATTN_SF(Dv, Nv)                                                                                  \
    hipLaunchKernelGGL((small_forward_kernel<Dv, Nv>), dim3(BH), dim3(256), 0, st, Q, K, V, Out, n, m,       \
                       (double)lambda, T, (double)eps, pl)
    if (d == 32) {
        if (norm == NORM_INLINE) LAPATTN_SF(32, NORM_INLINE);
        else if (norm == NORM_ROWSUM) LAPATTN_SF(32, NORM_ROWSUM);
        else LAPATTN_SF(32, NORM_NONE);
    } else {
        if (norm == NORM_INLINE) LAPATTN_SF(64, NORM_INLINE);
        else if (norm == NORM_ROWSUM) LAPATTN_SF(64, NORM_ROWSUM);
        else LAPATTN_SF(64, NORM_NONE);
    }
#undef LAPATTN_SF
    return hipGetLastError();
}

// Landmark-space normalisation vectors: mvec[h] = {sum_l w_l M_l[:d], (1/m) sum_l M_l[:d]}
// (w = ones when whiten is NULL), summed in landmark order.  grid (BH), D threads.
__global__ void mspace_vec_kernel(const float* __restrict__ M, const float* __restrict__ whiten,
                                  float* __restrict__ mvec, int H, int m, int D) {
    const int h = blockIdx.x, c = threadIdx.x;
    if (c >= D) return;
    const float* wl = whiten ? whiten + (size_t)(h % H) * m : nullptr;
    float sw = 0.f, sb = 0.f;
    for (int l = 0; l < m; ++l) {
        const float v = M[((size_t)h * m + l) * (D + 1) + c];
        sw = fmaf(wl ? wl[l] : 1.f, v, sw);
        sb += v;
    }
    mvec[(size_t)h * 2 * D + c] = sw;
    mvec[(size_t)h * 2 * D + D + c] = sb / (float)m;
}

hipError_t launch_mspace_vec(const float* M, const float* whiten, float* mvec, int BH, int H, int d, int m,
                             hipStream_t st) {
    hipLaunchKernelGGL(mspace_vec_kernel, dim3(BH), dim3(64), 0, st, M, whiten, mvec, H, m, d);
    return hipGetLastError();
}

}  // namespace lapattn
