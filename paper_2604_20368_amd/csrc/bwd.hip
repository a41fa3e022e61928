// bwd.hip -- backward kernels (fp32 inputs) of Nystrom-approximated Laplacian-kernel attention.
//
// Gradient of sum(Out * dOut) through, in reverse order: the normalisation (Eq. (4) / Eq. (3)),
// Y = K_QL M, M = X_T U, the Newton-Schulz updates of Algorithm 2 including the scale of X0,
// U = K_LK [V|1], K_LL, and the landmark means.  Kernel gradient (App. A):
//   d k(x,y) / dx_c = -(1/lambda) sign(x_c - y_c) k(x,y),  with sign(0) = 0.
//
//   bwd_query_kernel     query-major: dY, dA = dY M^T, dD = -A dA / lambda, direct dQ
//   bwd_query_lm_kernel  landmark-major over queries: dM = A^T dY, dkt from K_QL
//   bwd_ns_kernel        dX = dM U^T, dU = X_T^T dM, reverse Newton-Schulz, dDW (the K_LL
//                        backward itself runs in kll_bwd_kernel, nsbig.hip)
//   bwd_key_kernel       key-major: dB = dU [v|1]^T, dV, dD' = -B dB / lambda, dK
//   bwd_key_lm_kernel    landmark-major over keys: dqt from K_LK
//   bwd_pool_kernel      landmark-mean backward into dQ
#include "common.hpp"
#include "kernels.hpp"
#include "ns_mfma.hpp"
#include "srows.hpp"

namespace lapattn {

static inline float kscale_of(float lambda) { return (float)(-1.4426950408889634 / (double)lambda); }

typedef float f32x16_t __attribute__((ext_vector_type(16)));

// ------------------------------------------------------------------------------------------
// Direct global -> LDS copies (global_load_lds_dwordx4): each instruction moves 64 lanes x 16
// bytes to consecutive LDS addresses.  Their completion is tracked by vmcnt alone -- the
// compiler does not order later LDS reads after them -- so a reader waits with lds_dma_wait().
typedef __attribute__((address_space(3))) void lds_void_t;

__device__ __forceinline__ void lds_dma16(float* lds_dst, const float* src_lane) {
    __builtin_amdgcn_global_load_lds(reinterpret_cast<const void*>(src_lane), (lds_void_t*)(lds_dst),
                                     16, 0, 0);
}
__device__ __forceinline__ void lds_dma4(float* lds_dst, const float* src_lane) {
    __builtin_amdgcn_global_load_lds(reinterpret_cast<const void*>(src_lane), (lds_void_t*)(lds_dst),
                                     4, 0, 0);
}
__device__ __forceinline__ void lds_dma_wait() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// Rows r0 .. r0+63 of a [n][64] array into a wave's [row][column] tile of pitch 65 by direct
// copies (one row per instruction, all 64 in flight, no data registers); rows past n are zero.
// The row addresses are formed in the loop (partly unrolled): fully unrolled, a caller's loop
// would hoist all 64 of them and keep them in registers.
// Columns at or past m hold whatever the array holds there: the callers never read them.
__device__ __forceinline__ void load_rows64_dma(float* tile, const float* __restrict__ src, int r0, int n) {
    const int l = (int)(threadIdx.x & 63);
    const float* col = src + l;
#pragma unroll 8
    for (int r = 0; r < 64; ++r) lds_dma4(tile + r * 65, col + (size_t)min(r0 + r, n - 1) * 64);
    lds_dma_wait();
    for (int r = max(0, n - r0); r < 64; ++r) tile[r * 65 + l] = 0.f;
    __builtin_amdgcn_wave_barrier();
}

// Columns c0 .. c0 + 31 of the same rows into a 64 x 32 tile of pitch 33: one row per copy, on
// lanes 0..31 (a copy writes consecutive LDS words, and consecutive rows are 33 words apart).
__device__ __forceinline__ void load_half_rows_dma(float* tile, const float* __restrict__ src, int r0, int n, int c0) {
    const int l = (int)(threadIdx.x & 63);
    if (l < 32) {
        const float* col = src + c0 + l;
#pragma unroll 8
        for (int r = 0; r < 64; ++r) lds_dma4(tile + r * 33, col + (size_t)min(r0 + r, n - 1) * 64);
    }
    lds_dma_wait();
    if (l < 32)
        for (int r = max(0, n - r0); r < 64; ++r) tile[r * 33 + l] = 0.f;
    __builtin_amdgcn_wave_barrier();
}

// ------------------------------------------------------------------------------------------
// Query-major pass.  grid (nqb, BH), 256 threads, lane = query (wave w of block b covers
// queries 256 b + 64 w ..).  Landmark rows of kt come through scalar registers (srows.hpp),
// the rows of M are LDS broadcasts; loops that stream rows read no LDS (see pass 1).
//   Pass 1: a_il = k(q_i, kt_l) into the wave's [query][landmark] LDS tile.
//   Then, from the tile: s_i (and y_i for the row-sum normalisation), rs, dYd; whole rows of
//   Aq; dA_il = rs_i dO_i . M_l[:d] + dYd_i M_l[d] and dD_il = -a_il dA_il / lambda back into
//   the tile; whole rows of dDq.
//   Pass 2: dq_i += dD_il sign(q_i - kt_l).
//   dvbar partial (inline normalisation): sum over the block's queries of (1 - s_i) dO_i,
//   per wave through the tile, then over the waves in order.
//   Landmark-space normalisation (Appendix B): the same as inline with M's rows scaled by the
//   whitening, its ones column replaced by 1/m and vbar by sum_l w_l M_l (mvec); the partial
//   sums of (1 - s_i) dO_i and of dO_i (into p0_part) give the gradient of the two vectors.
// MPK = 64 for m <= 64, 128 for m up to 128.  The rows of A and dD (Aq, dDq) are group-major:
// [h][g][n][64] for the landmark groups g of 64 (one group when m <= 64).
template <int D, int NORM, int MPK>
__global__ __launch_bounds__(256, D == 32 ? 3 : 2) void bwd_query_kernel(const float* __restrict__ Q, const float* __restrict__ dO,
                                                        float* __restrict__ dQ, const float* __restrict__ kt,
                                                        const float* __restrict__ M, const float* __restrict__ vbar,
                                                        float* __restrict__ Aq, float* __restrict__ dDq,
                                                        float* __restrict__ rs, float* __restrict__ dYd,
                                                        float* __restrict__ dvbar_part, float* __restrict__ p0_part,
                                                        const float* __restrict__ whiten,
                                                        const float* __restrict__ mvec, int saved, int H, int n,
                                                        int m, float kscale, float inv_lambda, int nqb) {
    constexpr bool CENTRED = NORM == NORM_INLINE || NORM == NORM_MSPACE;
    constexpr int D1 = D + 1;
    constexpr int NCH = D / 32;
    // Landmarks in ranges of LW: 32 (a 64 x 33 tile per wave, which lets three blocks share a
    // compute unit), except for the row-sum normalisation, which needs s_i and y_i over all
    // landmarks before dA and takes them in one range of 64 when m <= 64; for m > 64 it takes
    // them in a first walk over the ranges (PRE) and forms the kernel values again for dA.
    // Every sum keeps landmark order.
    constexpr int LW = (NORM == NORM_ROWSUM && MPK == 64) ? 64 : 32;
    constexpr bool PRE = NORM == NORM_ROWSUM && MPK == 128;
    constexpr int TP = LW + 1;             // tile pitch: lane-strided accesses are conflict-free
    __shared__ __attribute__((aligned(16))) float sM[MPK * D1];
    __shared__ float sVb[D];
    __shared__ float sT[4 * 64 * TP];
    __shared__ float sred[4 * D];
    const int h = blockIdx.y, tid = threadIdx.x, w = tid >> 6, l = tid & 63;
    if (NORM == NORM_MSPACE) {
        const float* wl = whiten ? whiten + (size_t)(h % H) * m : nullptr;
        for (int e = tid; e < MPK * D1; e += 256) {
            const int a = e / D1, cc = e % D1;
            float v = 0.f;
            if (a < m) v = cc < D ? (wl ? wl[a] : 1.f) * M[(size_t)h * m * D1 + e] : 1.f / (float)m;
            sM[e] = v;
        }
        if (tid < D) sVb[tid] = mvec[(size_t)h * 2 * D + tid];
    } else {
        for (int e = tid; e < MPK * D1; e += 256) sM[e] = (e < m * D1) ? M[(size_t)h * m * D1 + e] : 0.f;
        if (tid < D) sVb[tid] = vbar[(size_t)h * D + tid];
    }
    float* tile = sT + w * 64 * TP;
    const int i0 = blockIdx.x * 256 + w * 64;
    const int i = i0 + l;
    const bool live = i < n;
    const size_t row = ((size_t)h * n + (live ? i : n - 1)) * D;
    float q[D], g[D];
#pragma unroll
    for (int c4 = 0; c4 < D / 4; ++c4) {
        const float4 a = reinterpret_cast<const float4*>(Q + row)[c4];
        const float4 b = reinterpret_cast<const float4*>(dO + row)[c4];
        q[4 * c4 + 0] = a.x; q[4 * c4 + 1] = a.y; q[4 * c4 + 2] = a.z; q[4 * c4 + 3] = a.w;
        g[4 * c4 + 0] = b.x; g[4 * c4 + 1] = b.y; g[4 * c4 + 2] = b.z; g[4 * c4 + 3] = b.w;
    }
    __syncthreads();   // sM, sVb
    float rsc = 1.f, dyd = 0.f;
    if (CENTRED) {
        float t = 0.f;
#pragma unroll
        for (int c = 0; c < D; ++c) t = fmaf(g[c], sVb[c], t);
        dyd = -t;
    }
    float s = 0.f;   // s_i (and y_i for the row-sum normalisation), in landmark order
    float y[NORM == NORM_ROWSUM ? D : 1];
#pragma unroll
    for (int c = 0; c < (NORM == NORM_ROWSUM ? D : 1); ++c) y[c] = 0.f;
    float dq[D];
#pragma unroll
    for (int c = 0; c < D; ++c) dq[c] = 0.f;
    const int ng = (m + 63) / 64;   // landmark groups of the row arrays
    const int nrange = LW == 64 ? 1 : (m + LW - 1) / LW;
    // pass 1 over the range of landmarks lo .. lo + mh - 1 (tile columns 0 .. mh - 1): a_il into
    // the tile (a column mh, reached only past the table, holds zeros).  The streaming loops read
    // no LDS: a wait for an LDS read would also wait for the row prefetch.
    auto pass1 = [&](int lo, int mh, const float* tab) {
        const float* Ag = Aq + (size_t)(h * ng + lo / 64) * n * 64;
        const int units = mh * NCH;
        auto emit = [&](int a, float dist) {
            tile[l * TP + a] = (live && a < mh) ? __builtin_amdgcn_exp2f(dist * kscale) : 0.f;
        };
        if (saved) {   // the forward left the rows of A in Aq: copy them into the tile
            if (LW == 64) load_rows64_dma(tile, Ag, i0, n);
            else load_half_rows_dma(tile, Ag, i0, n, lo % 64);
        } else {
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
        if (mh & 1) tile[l * TP + mh] = 0.f;   // the pair loops read column mh (unwritten when d = 64)
        __builtin_amdgcn_wave_barrier();
    };
    // s_i (and y_i for the row-sum normalisation) over the range, then the range's rows of A
    auto sums_and_rows = [&](int lo, int mh) {
        for (int a = 0; a < mh; ++a) {
            const float av = tile[l * TP + a];
            const float* mr = sM + (lo + a) * D1;
            s = fmaf(av, mr[D], s);
            if (NORM == NORM_ROWSUM) {
#pragma unroll
                for (int c = 0; c < D; ++c) y[c] = fmaf(av, mr[c], y[c]);
            }
        }
        if (!saved) {
            float* Ag = Aq + (size_t)(h * ng + lo / 64) * n * 64;
            if (LW == 64) store_rows64(Ag, tile, i0, n, mh);
            else store_half_rows(Ag, tile, i0, n, lo % 64, mh);
        }
    };
    auto rowsum_scales = [&]() {   // s and y complete
        float t = 0.f;
#pragma unroll
        for (int c = 0; c < D; ++c) t = fmaf(g[c], y[c], t);
        rsc = 1.f / s;
        dyd = -t / (s * s);
    };
    if (PRE) {
        for (int ri = 0; ri < nrange; ++ri) {
            const int lo = LW * ri, mh = min(LW, m - lo);
            pass1(lo, mh, kt + __builtin_amdgcn_readfirstlane((h * m + lo) * D));
            sums_and_rows(lo, mh);
            __builtin_amdgcn_wave_barrier();   // the next range overwrites the tile
        }
        rowsum_scales();
    }
    for (int ri = 0; ri < nrange; ++ri) {
        const int lo = LW * ri, mh = min(LW, m - lo);   // landmarks lo .. lo + mh - 1: tile columns 0 .. mh - 1
        const float* tab = kt + __builtin_amdgcn_readfirstlane((h * m + lo) * D);   // wave-uniform: scalar loads
        const int units = mh * NCH;
        pass1(lo, mh, tab);
        if (!PRE) {
            sums_and_rows(lo, mh);
            if (NORM == NORM_ROWSUM) rowsum_scales();   // one range: s and y are complete
        }
        __builtin_amdgcn_wave_barrier();

        // dA_il = sum_c M[l][c] dY_i[c] (dY_i = [rs_i dO_i | dYd_i]) on fp32 MFMA 32x32x2 as
        // dA^T = M dY^T, per 32-landmark block lb of the range and 32-query half qb, k = a
        // coordinate pair (the ones column is coordinate D, coordinate D + 1 is zero).  A operand:
        // lane l holds M[32 lb + l % 32][2 s + l / 32]; B operand: one permlane32 swap of the
        // lane's own pair of coordinates gives both halves (queries 0..31 keep theirs and receive
        // coordinate 2s+1 of 32..63, and vice versa).  Result register r at lane l: landmark
        // 32 lb + 8 (r / 4) + 4 (l / 32) + r % 4, query 32 qb + l % 32; dD = -a dA / lambda
        // replaces a in the tile.
        {
            constexpr int KS = D / 2 + 1;   // coordinate pairs, the last one (dYd, 0)
            const int nlb = (mh + 31) / 32, lb0 = lo / 32;
            const int hk = l >> 5, lr = l & 31;
            // one 32 x 32 block at a time (16 accumulator registers); the swaps are redone per block
            for (int blk = 0; blk < 2 * nlb; ++blk) {
                const int lb = blk >> 1, qb = blk & 1;
                f32x16_t acc;
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[r] = 0.f;
#pragma unroll
                for (int ks = 0; ks < KS; ++ks) {
                    const float x0 = (2 * ks < D) ? g[2 * ks] * rsc : dyd;
                    const float x1 = (2 * ks + 1 < D) ? g[2 * ks + 1] * rsc : 0.f;
                    const auto bsw =
                        __builtin_amdgcn_permlane32_swap(__float_as_uint(x0), __float_as_uint(x1), false, false);
                    const int c = 2 * ks + hk;
                    const float av = c <= D ? sM[(32 * (lb0 + lb) + lr) * D1 + c] : 0.f;
                    acc = __builtin_amdgcn_mfma_f32_32x32x2f32(av, __uint_as_float(qb ? bsw[1] : bsw[0]), acc, 0, 0,
                                                               0);
                }
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int a = 32 * lb + 8 * (r >> 2) + 4 * hk + (r & 3);
                    float* t = tile + (32 * qb + lr) * TP + a;
                    *t = -*t * acc[r] * inv_lambda;
                }
            }
        }
        __builtin_amdgcn_wave_barrier();
        {
            float* Dg = dDq + (size_t)(h * ng + lo / 64) * n * 64;
            if (LW == 64) store_rows64(Dg, tile, i0, n, mh);
            else store_half_rows(Dg, tile, i0, n, lo % 64, mh);
        }

        // pass 2: dq_i += dD_il sign(q_i - kt_l); each unit's dD is read before the unit's
        // first wait (which covers it); landmarks past m have dD = 0 (a zero column when mh is odd)
        {
            float ta[32], tb[32];
            srow32(ta, tab);
            for (int u = 0; u < units; u += 2) {
                if (NCH == 1) {
                    const float d0 = tile[l * TP + u], d1 = tile[l * TP + u + 1];
                    __builtin_amdgcn_sched_barrier(0);
                    sgn_unit(dq, q, ta, tb, tab + 32 * min(u + 1, units - 1), d0);
                    sgn_unit(dq, q, tb, ta, tab + 32 * min(u + 2, units - 1), d1);
                } else {
                    const float d0 = tile[l * TP + u / NCH];
                    __builtin_amdgcn_sched_barrier(0);
                    sgn_unit(dq, q, ta, tb, tab + 32 * min(u + 1, units - 1), d0);
                    sgn_unit(dq + 32, q + 32, tb, ta, tab + 32 * min(u + 2, units - 1), d0);
                }
            }
            asm volatile("" ::"s"(ta[0]), "s"(ta[16]));
        }
        __builtin_amdgcn_wave_barrier();   // the next range overwrites the tile
    }
    if (live) {
        rs[(size_t)h * n + i] = rsc;
        dYd[(size_t)h * n + i] = dyd;
#pragma unroll
        for (int c4 = 0; c4 < D / 4; ++c4)
            reinterpret_cast<float4*>(dQ + row)[c4] = make_float4(dq[4 * c4], dq[4 * c4 + 1], dq[4 * c4 + 2], dq[4 * c4 + 3]);
    }
    // dvbar partial (and for the landmark-space form the plain sum of dO): per wave through the
    // tile, 32 columns at a time (rows in order), then over the waves in order
    if (CENTRED) {
        auto block_sum = [&](float wt, float* part) {
#pragma unroll
            for (int c0 = 0; c0 < D; c0 += 32) {
                __builtin_amdgcn_wave_barrier();
#pragma unroll
                for (int c = 0; c < 32; ++c) tile[l * TP + c] = wt * g[c0 + c];
                __builtin_amdgcn_wave_barrier();
                if (l < 32) {
                    float t = 0.f;
                    for (int r = 0; r < 64; ++r) t += tile[r * TP + l];
                    sred[w * D + c0 + l] = t;
                }
            }
            __syncthreads();
            if (tid < D)
                part[((size_t)h * nqb + blockIdx.x) * D + tid] =
                    ((sred[tid] + sred[D + tid]) + sred[2 * D + tid]) + sred[3 * D + tid];
        };
        block_sum(live ? 1.f - s : 0.f, dvbar_part);
        if (NORM == NORM_MSPACE) {
            __syncthreads();   // sred is reused
            block_sum(live ? 1.f : 0.f, p0_part);
        }
    } else if (tid < D) {
        dvbar_part[((size_t)h * nqb + blockIdx.x) * D + tid] = 0.f;
    }
}

// The rows of a [token][W] array (W floats per row, W a multiple of 4) for tokens t0 .. t0 + R - 1
// (clamped to the last token) into dst[R][W]; R W must be a multiple of 256.
template <int R, int W>
__device__ __forceinline__ void stage_rows(float* dst, const float* base, int t0, int n) {
    static_assert((R * W) % 256 == 0, "whole 1 KB copies");
    const int l = threadIdx.x & 63;
#pragma unroll
    for (int k = 0; k < R * W / 256; ++k) {
        const int e = 256 * k + 4 * l;
        lds_dma16(dst + 256 * k, base + (size_t)min(t0 + e / W, n - 1) * W + e % W);
    }
}

// ------------------------------------------------------------------------------------------
// Landmark-major pass over queries.  grid (nlc, BH), 64 threads (lane = landmark l); block ch
// covers queries [ch * chunk, ...) in sub-tiles of 8 whose data -- rows of Q and dO, rows of Aq
// and dDq (pitch 64), rs and dYd -- is copied to LDS one sub-tile ahead (two buffers).  Per
// query i:
//   dM_l[:d] += a_il rs_i dO_i on fp32 MFMA 32x32x1 (A = a_il, lane = landmark = MFMA row; B =
//   rs_i dO_i[32 hh + l % 32], one 32-column half per instruction), dM_l[d] += a_il dYd_i;
//   dkt_l -= dD_il sign(q_i - kt_l).
// Queries past the chunk contribute zeros.  Landmarks in groups of 64: blockIdx.z = group g, lane l
// = landmark 64 g + l, reading the group's rows of Aq and dDq ([h][g][n][64]).
typedef float f32x32_t __attribute__((ext_vector_type(32)));

template <int D>
__global__ __launch_bounds__(64) void bwd_query_lm_kernel(const float* __restrict__ Q, const float* __restrict__ dO,
                                                          const float* __restrict__ kt, const float* __restrict__ Aq,
                                                          const float* __restrict__ dDq, const float* __restrict__ rs,
                                                          const float* __restrict__ dYd, float* __restrict__ dM_part,
                                                          float* __restrict__ dkt_part, int n, int m, int chunk,
                                                          int nlc) {
    constexpr int D1 = D + 1;
    constexpr int NH = D / 32;
    constexpr int ST = 8;                                            // queries per sub-tile
    constexpr int BUF = ST * D + ST * 64 + ST * 64 + ST * D + 64;   // Q, Aq, dDq, dO, rs | dYd
    __shared__ __attribute__((aligned(16))) float sbuf[2 * BUF];
    const int ch = blockIdx.x, h = blockIdx.y, l = threadIdx.x, g = blockIdx.z, ng = gridDim.z;
    const int lm0 = 64 * g;
    const bool live = lm0 + l < m;
    const int lc = live ? lm0 + l : m - 1;   // landmark
    const int lcol = lc - lm0;               // its column in the group's rows
    const float* Qh = Q + (size_t)h * n * D;
    const float* dOh = dO + (size_t)h * n * D;
    const float* Ah = Aq + (size_t)(h * ng + g) * n * 64;
    const float* DDh = dDq + (size_t)(h * ng + g) * n * 64;
    const int i0 = ch * chunk, i1 = min(n, i0 + chunk);
    auto stage = [&](int b, int t0) {
        float* sb = sbuf + b * BUF;
        stage_rows<ST, D>(sb, Qh, t0, n);
        stage_rows<ST, 64>(sb + ST * D, Ah, t0, n);
        stage_rows<ST, 64>(sb + ST * D + ST * 64, DDh, t0, n);
        stage_rows<ST, D>(sb + ST * D + 2 * ST * 64, dOh, t0, n);
        const int r = min(t0 + (l & (ST - 1)), n - 1);
        lds_dma4(sb + 2 * ST * D + 2 * ST * 64, (l < ST ? rs : dYd) + (size_t)h * n + r);
    };
    float k[D], dk[D];
#pragma unroll
    for (int c = 0; c < D; ++c) {
        k[c] = kt[((size_t)h * m + lc) * D + c];
        dk[c] = 0.f;
    }
    float dml = 0.f;
    f32x32_t acc[NH];
#pragma unroll
    for (int hh = 0; hh < NH; ++hh)
#pragma unroll
        for (int r = 0; r < 32; ++r) acc[hh][r] = 0.f;
    if (i0 < i1) stage(0, i0);
    int buf = 0;
    for (int t0 = i0; t0 < i1; t0 += ST, buf ^= 1) {
        lds_dma_wait();
        __builtin_amdgcn_wave_barrier();
        if (t0 + ST < i1) stage(buf ^ 1, t0 + ST);
        const float* sb = sbuf + buf * BUF;
        const float* sQ = sb;
        const float* sA = sb + ST * D;
        const float* sDD = sA + ST * 64;
        const float* sdO = sDD + ST * 64;
        const float* sRY = sdO + ST * D;
#pragma unroll 4
        for (int r = 0; r < ST; ++r) {
            const bool in = live && t0 + r < i1;
            const float av = sA[r * 64 + lcol], ddv = sDD[r * 64 + lcol];   // unconditional reads
            const float a = in ? av : 0.f;
            const float dd = in ? ddv : 0.f;
            const float rsi = sRY[r], ydi = sRY[ST + r];
#pragma unroll
            for (int hh = 0; hh < NH; ++hh)
                acc[hh] = __builtin_amdgcn_mfma_f32_32x32x1f32(a, sdO[r * D + 32 * hh + (l & 31)] * rsi, acc[hh], 0, 0, 0);
            dml = fmaf(a, ydi, dml);
            const float* qr = sQ + r * D;
            const float dds = -dd * 0x1p64f;
#pragma unroll
            for (int c = 0; c < D; ++c) dk[c] = fmaf(dds, sgn_term(qr[c], k[c]), dk[c]);
        }
        __builtin_amdgcn_wave_barrier();
    }
    // result register r of the 32x32x1 product: landmark 32 (r / 16) + 8 ((r % 16) / 4) + 4 (l / 32)
    // + r % 4, column 32 hh + l % 32
    const size_t o = ((size_t)h * nlc + ch) * m;
#pragma unroll
    for (int hh = 0; hh < NH; ++hh)
#pragma unroll
        for (int r = 0; r < 32; ++r) {
            const int lm = lm0 + 32 * (r / 16) + 8 * ((r % 16) / 4) + 4 * (l / 32) + r % 4;
            if (lm < m) dM_part[(o + lm) * D1 + 32 * hh + (l & 31)] = acc[hh][r];
        }
    if (!live) return;
    dM_part[(o + lc) * D1 + D] = dml;
#pragma unroll
    for (int c = 0; c < D; ++c) dkt_part[(o + lc) * D + c] = dk[c];
}

// ------------------------------------------------------------------------------------------
// Newton-Schulz backward, one block of 256 threads per head (ns_mfma.hpp).
//   dM = sum of partials;  dX_T = dM U^T;  dU = X_T^T dM  (fp64, fp64 matrix cores).
//   For t = T-1..0, with G = dL/dX_{t+1} and X_{t+1} = 2 X_t - X_t W X_t:
//     dW -= X_t^T G X_t^T;   G <- 2G - G X_t^T W^T - W^T X_t^T G,
//   five fp32 products per step (fp32 matrix cores, ns32_mm): P = X^T G, P X^T, W^T P (the
//   last term, reusing P), G X^T and (G X^T) W^T; G, X, W and P are held both ways in LDS
//   (row-major as left factors, transposed as right ones), X_{t-1} is loaded while step t runs.
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
                                                     float* __restrict__ dkpool, const float* __restrict__ dkt_part,
                                                     LmPool pl, const float* __restrict__ p0_part,
                                                     const float* __restrict__ whiten, int mspace,
                                                     float* __restrict__ dDW, int H, int n,
                                                     int m, int T, double lambda, double eps, int nlc, int nqb) {
    using SQ = ns_tiles<MP, MP>;
    using SU = ns_tiles<MP, D>;
    constexpr int D1 = D + 1;
    constexpr int P = ns_pitch(MP);
    constexpr int PU = ns_pitch(D);
    using L = ns32_tiles<MP>;
    constexpr int PF = L::P;              // pitch (floats) of the fp32 matrices
    constexpr int MSZ = MP * PF;
    // fp32 reverse iteration: W, W^T, X, X^T, G, G^T, P (later G X^T), P^T.  Before it the same
    // space holds the fp64 value columns of U and dM (MP x D each, pitch PU) and X_T (pitch P).
    constexpr int PRE = (2 * MP * PU + MP * P) * 8;
    constexpr int F32 = 8 * MSZ * 4;
    __shared__ __attribute__((aligned(16))) char lds[F32 > PRE ? F32 : PRE];
    __shared__ double su1[MP], sdm1[MP];
    __shared__ double svb[256];
    __shared__ double sred4[4];
    __shared__ double sp1[D], sp0[D];   // landmark-space form: sums of (1 - s_i) dO_i and of dO_i
    float* const fW = reinterpret_cast<float*>(lds);
    float* const fWT = fW + MSZ;
    float* const fX = fW + 2 * MSZ;
    float* const fXT = fW + 3 * MSZ;
    float* const fG = fW + 4 * MSZ;
    float* const fGT = fW + 5 * MSZ;
    float* const fP = fW + 6 * MSZ;
    float* const fPT = fW + 7 * MSZ;
    const int h = blockIdx.x, tid = threadIdx.x;
    const size_t mm = (size_t)MP * MP;
    const double* Xh = Xs + (size_t)h * (T + 2) * mm;   // X_0 .. X_T, then W
    // W's loads go first: they are waited for only when the reverse iteration begins
    double wr[MP * MP / 256];
    ns_fetch<MP>(wr, Xh + (size_t)(T + 1) * mm);
    const double c = cinfo[h * 4 + 0], n1 = cinfo[h * 4 + 1], ninf = cinfo[h * 4 + 2];
    const int code = (int)cinfo[h * 4 + 3];

    // dvbar (inline normalisation; zeros otherwise because the partials are zero): 256 / D
    // partial sums per column over the query blocks, then in order.  The landmark-space form
    // keeps that sum (sp1) and the sum of dO (sp0) for the gradient of M, and has no dvbar.
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
            sp1[tid] = t;
            dvbar[(size_t)h * D + tid] = mspace ? 0.f : (float)t;
        }
        if (mspace) {
            __syncthreads();
            double s0 = 0.0;
            for (int b = g; b < nqb; b += G) s0 += p0_part[((size_t)h * nqb + b) * D + cc];
            svb[tid] = s0;
            __syncthreads();
            if (tid < D) {
                double t = 0.0;
#pragma unroll
                for (int gg = 0; gg < G; ++gg) t += svb[gg * D + tid];
                sp0[tid] = t;
            }
        }
        __syncthreads();
    }
    f64x4_t dX[SQ::NT];
    {
        double* sU = reinterpret_cast<double*>(lds);
        double* sdM = sU + MP * PU;
        double* sXT = sU + 2 * MP * PU;
        // dM = sum of the landmark-chunk partials (in chunk order); each thread's entries are
        // loaded together, chunk by chunk
        constexpr int NE = (MP * D1 + 255) / 256;
        double dm[NE];
#pragma unroll
        for (int r = 0; r < NE; ++r) dm[r] = 0.0;
        const int lim = m * D1 - 1;
        // CB chunks' loads in flight at a time, added in chunk order
        constexpr int CB = NE > 9 ? 4 : 8;
        for (int c0 = 0; c0 < nlc; c0 += CB) {
            float v[CB][NE];
#pragma unroll
            for (int cc = 0; cc < CB; ++cc) {
                const float* dp = dM_part + ((size_t)h * nlc + min(c0 + cc, nlc - 1)) * m * D1;
#pragma unroll
                for (int r = 0; r < NE; ++r) v[cc][r] = dp[min(tid + 256 * r, lim)];
            }
#pragma unroll
            for (int cc = 0; cc < CB; ++cc)
#pragma unroll
                for (int r = 0; r < NE; ++r)
                    if (c0 + cc < nlc && tid + 256 * r <= lim) dm[r] += (double)v[cc][r];
        }
        if (mspace) {
            // the partials hold the gradient of M~ = diag(w) M with the ones column 1/m; with
            // mw = sum_l w_l M_l and mb = (1/m) sum_l M_l entering as - s_i mw + mb:
            // dM_l[:d] = w_l (dM~_l + sp1 - sp0) + sp0 / m, and no gradient for the ones column
            const float* wl = whiten ? whiten + (size_t)(h % H) * m : nullptr;
#pragma unroll
            for (int r = 0; r < NE; ++r) {
                const int e = tid + 256 * r;
                const int a = e / D1, cc = e % D1;
                if (e <= lim) {
                    const double wa = wl ? (double)wl[a] : 1.0;
                    dm[r] = cc < D ? wa * (dm[r] + sp1[cc] - sp0[cc]) + sp0[cc] / m : 0.0;
                }
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
        __syncthreads();   // the fp64 operands are dead: the fp32 matrices take the space
    }
    // W (kernel + eps I as the forward solve stored it: fp64 copies of fp32 values) both ways,
    // and G = dX both ways
    {
#pragma unroll
        for (int r = 0; r < MP * MP / 256; ++r) {
            const int e = tid + 256 * r, a = e / MP, b = e % MP;
            const float wv = (float)wr[r];
            fW[a * PF + b] = wv;
            fWT[b * PF + a] = wv;
        }
#pragma unroll
        for (int i = 0; i < SQ::NT; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int a = SQ::row(i, j), b = SQ::col(i);
                const float gv = (float)dX[i][j];
                fG[a * PF + b] = gv;
                fGT[b * PF + a] = gv;
            }
    }
    const int row0 = 4 * ((tid & 63) >> 4), col = ns32_col<MP>();   // this lane's tile rows: 16 tr + row0 + j
    f32x4_t dW[L::NT];
#pragma unroll
    for (int i = 0; i < L::NT; ++i) dW[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    if (c > 0.0) {
        // X_t comes through registers: the loads of X_{t-1} are issued while step t runs
        double xr[MP * MP / 256];
        if (T > 0) ns_fetch<MP>(xr, Xh + (size_t)(T - 1) * mm);
        for (int t = T - 1; t >= 0; --t) {
#pragma unroll
            for (int r = 0; r < MP * MP / 256; ++r) {
                const int e = tid + 256 * r, a = e / MP, b = e % MP;
                const float xv = (float)xr[r];
                fX[a * PF + b] = xv;
                fXT[b * PF + a] = xv;
            }
            __syncthreads();   // X_t, and G from the previous step
            if (t > 0) ns_fetch<MP>(xr, Xh + (size_t)(t - 1) * mm);
            f32x4_t r1[L::NT], r3[L::NT], r4[L::NT];
            ns32_mm<MP>(fXT, fGT, r1);   // P = X^T G
#pragma unroll
            for (int i = 0; i < L::NT; ++i) {
                const int ra = 16 * L::tr(i) + row0;
#pragma unroll
                for (int j = 0; j < 4; ++j) fP[(ra + j) * PF + col] = r1[i][j];
                *reinterpret_cast<float4*>(fPT + col * PF + ra) = make_float4(r1[i][0], r1[i][1], r1[i][2], r1[i][3]);
            }
            __syncthreads();
            ns32_mm<MP>(fP, fX, r1);     // P X^T
#pragma unroll
            for (int i = 0; i < L::NT; ++i) dW[i] -= r1[i];
            ns32_mm<MP>(fWT, fPT, r3);   // W^T P = W^T X^T G
            ns32_mm<MP>(fG, fX, r4);     // G X^T
            __syncthreads();   // P, X and X^T are read: G X^T takes P's buffer
#pragma unroll
            for (int i = 0; i < L::NT; ++i) {
                const int ra = 16 * L::tr(i) + row0;
#pragma unroll
                for (int j = 0; j < 4; ++j) fP[(ra + j) * PF + col] = r4[i][j];
            }
            __syncthreads();
            ns32_mm<MP>(fP, fW, r1);     // (G X^T) W^T
            // G <- 2G - G X^T W^T - W^T X^T G (each lane rewrites its own entries; G is not
            // read again in this step)
#pragma unroll
            for (int i = 0; i < L::NT; ++i) {
                const int ra = 16 * L::tr(i) + row0;
                float gn[4];
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    gn[j] = 2.f * fG[(ra + j) * PF + col] - r1[i][j] - r3[i][j];
                    fG[(ra + j) * PF + col] = gn[j];
                }
                *reinterpret_cast<float4*>(fGT + col * PF + ra) = make_float4(gn[0], gn[1], gn[2], gn[3]);
            }
        }
        __syncthreads();   // G = dL/dX_0
        // X0 = W^T / c
        const int as = code / 256, bs = code % 256;
        // <G, W^T>: block reduction in fixed order
        double part = 0.0;
#pragma unroll
        for (int i = 0; i < L::NT; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int a = 16 * L::tr(i) + row0 + j;
                part += (double)fG[a * PF + col] * (double)fW[col * PF + a];
            }
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) part += __shfl_xor(part, off, 64);
        if ((tid & 63) == 0) sred4[tid >> 6] = part;
        __syncthreads();
        const double dc = -(((sred4[0] + sred4[1]) + sred4[2]) + sred4[3]) / (c * c);
#pragma unroll
        for (int i = 0; i < L::NT; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int a = 16 * L::tr(i) + row0 + j, b = col;
                const double wab = (double)fW[a * PF + b];
                double v = (double)fG[b * PF + a] / c;
                if (b == bs) v += dc * ninf * sgnd(wab);
                if (a == as) v += dc * n1 * sgnd(wab);
                dW[i][j] += (float)v;
            }
        __syncthreads();
    } else {
        __syncthreads();
    }
    // dDW = -k dW / lambda (k = W - eps on the diagonal), fp32, [MP][MP] (zero past m: W and the
    // gradient vanish there); launch_kll_backward maps it to the landmarks over the whole chip
    float* Dh = dDW + (size_t)h * MP * MP;
#pragma unroll
    for (int i = 0; i < L::NT; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int a = 16 * L::tr(i) + row0 + j, b = col;
            const double kab = (double)fW[a * PF + b] - (a == b && a < m ? eps : 0.0);
            Dh[a * MP + b] = (float)(-kab * (double)dW[i][j] / lambda);
        }
}

// ------------------------------------------------------------------------------------------
// Key-major pass.  grid (ceil(n/256), BH), 256 threads, lane = key (wave w of block b covers
// keys 256 b + 64 w ..).  Landmark rows of qt come through scalar registers (srows.hpp), the
// rows of dU are LDS broadcasts.  Three phases over the landmarks a:
//   distance pass: B_aj = k(qt_a, k_j) into the wave's [key][landmark] LDS tile;
//   from the tile (LDS only): dB_aj = dU_a[:d] . v_j + dU_a[d], dV_j += B_aj dU_a[:d],
//   dD_aj = -B_aj dB_aj / lambda back into the tile (then whole rows of dDk);
//   sign pass: dK_j -= dD_aj sign(qt_a - k_j).
// The landmark rows are streamed twice (the table is small and stays in cache).  dV_j gets
// dvbar / n at the end.  MPK = 64 for m <= 64, 128 for m up to 128; the rows of B and dD (dDk)
// are group-major, [h][g][n][64] for the landmark groups g of 64.
template <int D, int MPK>
__global__ __launch_bounds__(256, D == 32 ? 3 : 2) void bwd_key_kernel(const float* __restrict__ K, const float* __restrict__ V,
                                                      float* __restrict__ dK, float* __restrict__ dV,
                                                      const float* __restrict__ qt, const float* __restrict__ dU,
                                                      const float* __restrict__ dvbar, float* __restrict__ dDk,
                                                      const float* __restrict__ dkpool, LmPool pl, int saved, int n,
                                                      int m, float kscale, float inv_lambda) {
    constexpr int D1 = D + 1;
    constexpr int NCH = D / 32;
    // Landmarks in ranges of LW: 32 at d = 32 (a 64 x 33 tile per wave, which lets three blocks
    // share a compute unit), ranges of 64 at d = 64 (whose registers allow two blocks either
    // way).  dV accumulates over the ranges (at d = 64 through its rows in memory, each range
    // adding to what the previous one stored); every sum keeps landmark order.
    constexpr int LW = D == 32 ? 32 : 64;
    constexpr int TP = LW + 1;
    __shared__ __attribute__((aligned(16))) float sdU[MPK * D1];
    __shared__ float sdv[D];
    __shared__ float sT[4 * 64 * TP];
    const int h = blockIdx.y, tid = threadIdx.x, w = tid >> 6, l = tid & 63;
    for (int e = tid; e < MPK * D1; e += 256) sdU[e] = (e < m * D1) ? dU[(size_t)h * m * D1 + e] : 0.f;
    const int ng = (m + 63) / 64;   // landmark groups of the row arrays
    if (tid < D) sdv[tid] = dvbar[(size_t)h * D + tid];
    float* tile = sT + w * 64 * TP;
    const int j0 = blockIdx.x * 256 + w * 64;
    const int j = j0 + l;
    const bool live = j < n;
    const size_t row = ((size_t)h * n + (live ? j : n - 1)) * D;
    float v[D], dk[D];
#pragma unroll
    for (int c4 = 0; c4 < D / 4; ++c4) {
        const float4 b = reinterpret_cast<const float4*>(V + row)[c4];
        v[4 * c4 + 0] = b.x; v[4 * c4 + 1] = b.y; v[4 * c4 + 2] = b.z; v[4 * c4 + 3] = b.w;
    }
    // the key row, read where a pass needs it (a cache hit after the first time): held across the
    // dV and dB products it would push the kernel past three blocks per compute unit
    float kk[D];
    auto load_key = [&]() {
        const float* kr = K + row;
        asm volatile("" : "+v"(kr));   // a fresh load each time, not a value kept from the last one
#pragma unroll
        for (int c4 = 0; c4 < D / 4; ++c4) {
            const float4 a = reinterpret_cast<const float4*>(kr)[c4];
            kk[4 * c4 + 0] = a.x; kk[4 * c4 + 1] = a.y; kk[4 * c4 + 2] = a.z; kk[4 * c4 + 3] = a.w;
        }
    };
#pragma unroll
    for (int c = 0; c < D; ++c) dk[c] = 0.f;
    __syncthreads();   // sdU, sdv
    // dV_j = sum_a B_aj dU_a[:d] on fp32 MFMA 32x32x2 (k = a landmark pair; A operand straight
    // from the tile), per 32-key half kh and 32-column block cb, accumulated over the ranges
    f32x16_t accv[2][D / 32];
#pragma unroll
    for (int kh = 0; kh < 2; ++kh)
#pragma unroll
        for (int cb = 0; cb < D / 32; ++cb)
#pragma unroll
            for (int r = 0; r < 16; ++r) accv[kh][cb][r] = 0.f;
    // dV with dvbar / n (first: the first contribution, else added to the stored rows, which this
    // lane wrote); result register r at lane l: key 32 kh + 8 (r / 4) + 4 (l / 32) + r % 4,
    // column 32 cb + l % 32
    auto store_dv = [&](bool first) {
        const float invn = 1.f / (float)n;
#pragma unroll
        for (int kh = 0; kh < 2; ++kh)
#pragma unroll
            for (int cb = 0; cb < D / 32; ++cb) {
                const int c = 32 * cb + (l & 31);
                const float add = sdv[c] * invn;
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int key = 32 * kh + 8 * (r / 4) + 4 * (l >> 5) + r % 4;
                    if (j0 + key < n) {
                        float* p = dV + ((size_t)h * n + j0 + key) * D + c;
                        *p = accv[kh][cb][r] + (first ? add : *p);
                    }
                }
            }
    };
    const int nrange = (MPK == 64 && LW == 64) ? 1 : (m + LW - 1) / LW;
    for (int ri = 0; ri < nrange; ++ri) {
        const int lo = LW * ri, mh = min(LW, m - lo);   // landmarks lo .. lo + mh - 1: tile columns 0 .. mh - 1
        const float* tab = qt + __builtin_amdgcn_readfirstlane((h * m + lo) * D);   // wave-uniform: scalar loads
        const int units = mh * NCH;
        // distance pass: B_aj into the tile (a column mh, reached only past the table, holds
        // zeros); the streaming loops read no LDS
        auto emit = [&](int a, float dist) {
            tile[l * TP + a] = (live && a < mh) ? __builtin_amdgcn_exp2f(dist * kscale) : 0.f;
        };
        float* Dg = dDk + (size_t)(h * ng + lo / 64) * n * 64;   // the range's group of rows
        if (saved) {   // the forward's key-side summary left the rows of B in dDk: copy the range's
                       // columns (each wave reads only its own rows, whose columns it overwrites
                       // with dD further down)
            if (LW == 64) load_rows64_dma(tile, Dg, j0, n);
            else load_half_rows_dma(tile, Dg, j0, n, lo % 64);
        } else {
            load_key();
            float ta[32], tb[32];
            srow32(ta, tab);
            float dist = 0.f;
            for (int u = 0; u < units; u += 2) {
                dist = l1_unit(kk + 32 * (u % NCH), ta, tb, tab + 32 * min(u + 1, units - 1), dist);
                if (NCH == 1) {
                    emit(u, dist);
                    dist = 0.f;
                }
                dist = l1_unit(kk + 32 * ((u + 1) % NCH), tb, ta, tab + 32 * min(u + 2, units - 1), dist);
                emit((u + 1) / NCH, dist);
                dist = 0.f;
            }
            asm volatile("" ::"s"(ta[0]), "s"(ta[16]));
        }
        if (mh & 1) tile[l * TP + mh] = 0.f;   // the pair loops read column mh (unwritten when d = 64)
        __builtin_amdgcn_wave_barrier();
        {
            const int npair = (mh + 1) / 2;
#pragma unroll
            for (int kh = 0; kh < 2; ++kh)
#pragma unroll
                for (int cb = 0; cb < D / 32; ++cb)
#pragma unroll 4
                    for (int p = 0; p < npair; ++p) {
                        const float av = tile[(32 * kh + (l & 31)) * TP + 2 * p + (l >> 5)];
                        const float bv = sdU[(lo + 2 * p + (l >> 5)) * D1 + 32 * cb + (l & 31)];
                        accv[kh][cb] = __builtin_amdgcn_mfma_f32_32x32x2f32(av, bv, accv[kh][cb], 0, 0, 0);
                    }
        }
        if (LW == 64) {   // the range's share of dV is complete (its accumulators free for dB)
            store_dv(ri == 0);
#pragma unroll
            for (int kh = 0; kh < 2; ++kh)
#pragma unroll
                for (int cb = 0; cb < D / 32; ++cb)
#pragma unroll
                    for (int r = 0; r < 16; ++r) accv[kh][cb][r] = 0.f;
        }
        // dB = [v | 1] dU^T on the same instruction (k = a coordinate pair; the A operands of both
        // 32-key halves from one permlane32 swap of the lane's own values), per 32-landmark block
        // and key half, and dD = -B dB / lambda in place in the tile.  Result register r at lane
        // l: key 32 kh + 8 (r / 4) + 4 (l / 32) + r % 4, landmark l % 32 of the block.
        {
            const int nlb = (mh + 31) / 32;
            for (int lb = 0; lb < nlb; ++lb) {
                const int ac = 32 * lb + (l & 31);   // tile column; landmark lo + ac
                const float u1 = sdU[(lo + ac) * D1 + D];
#pragma unroll 1
                for (int kh = 0; kh < 2; ++kh) {   // rolled: the swaps are redone, not held, per half
                    f32x16_t acc;
#pragma unroll
                    for (int r = 0; r < 16; ++r) acc[r] = 0.f;
#pragma unroll
                    for (int sp = 0; sp < D / 2; ++sp) {
                        const auto a2 = __builtin_amdgcn_permlane32_swap(__float_as_uint(v[2 * sp]),
                                                                         __float_as_uint(v[2 * sp + 1]), false, false);
                        const float bv = sdU[(lo + ac) * D1 + 2 * sp + (l >> 5)];
                        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a2[kh]), bv, acc, 0, 0, 0);
                    }
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const int key = 32 * kh + 8 * (r / 4) + 4 * (l >> 5) + r % 4;
                        float* tp = tile + key * TP + ac;
                        const float dd = -(*tp) * (acc[r] + u1) * inv_lambda;
                        if (ac < mh) *tp = dd;
                    }
                }
            }
        }
        __builtin_amdgcn_wave_barrier();
        if (LW == 64) store_rows64(Dg, tile, j0, n, mh);
        else store_half_rows(Dg, tile, j0, n, lo % 64, mh);
        // sign pass: dK_j -= dD_aj sign(qt_a - k_j), accumulated as dD sign(k_j - qt_a); each
        // unit's dD is read before the unit's first wait
        {
            load_key();
            float ta[32], tb[32];
            srow32(ta, tab);
            for (int u = 0; u < units; u += 2) {
                if (NCH == 1) {
                    const float d0 = tile[l * TP + u], d1 = tile[l * TP + u + 1];
                    __builtin_amdgcn_sched_barrier(0);
                    sgn_unit(dk, kk, ta, tb, tab + 32 * min(u + 1, units - 1), d0);
                    sgn_unit(dk, kk, tb, ta, tab + 32 * min(u + 2, units - 1), d1);
                } else {
                    const float d0 = tile[l * TP + u / NCH];
                    __builtin_amdgcn_sched_barrier(0);
                    sgn_unit(dk, kk, ta, tb, tab + 32 * min(u + 1, units - 1), d0);
                    sgn_unit(dk + 32, kk + 32, tb, ta, tab + 32 * min(u + 2, units - 1), d0);
                }
            }
            asm volatile("" ::"s"(ta[0]), "s"(ta[16]));
        }
        __builtin_amdgcn_wave_barrier();   // the next range overwrites the tile
    }
    if (LW == 32) store_dv(true);
    if (live) {   // with the pooling gradient of the key's landmark (window or segment)
        const int lp = pl.r ? ((j / pl.gw) / pl.r) * (pl.gw / pl.r) + (j % pl.gw) / pl.r : seg_of(j, n, m);
        const float4* kp = reinterpret_cast<const float4*>(dkpool + ((size_t)h * m + lp) * D);
#pragma unroll
        for (int c4 = 0; c4 < D / 4; ++c4) {
            const float4 p = kp[c4];
            reinterpret_cast<float4*>(dK + row)[c4] =
                make_float4(dk[4 * c4] + p.x, dk[4 * c4 + 1] + p.y, dk[4 * c4 + 2] + p.z, dk[4 * c4 + 3] + p.w);
        }
    }
}

// ------------------------------------------------------------------------------------------
// Landmark-major pass over keys.  grid (nlc, BH), 64 threads (lane = landmark a); block ch covers
// keys [ch * chunk, ...) in sub-tiles of 16 whose rows of K and of dDk (pitch 64) are copied to
// LDS one sub-tile ahead:  dqt_a += sum_j dD_aj sign(qt_a - k_j).  Landmarks in groups of 64:
// blockIdx.z = group g, lane = landmark 64 g + lane, reading the group's rows of dDk.
template <int D>
__global__ __launch_bounds__(64) void bwd_key_lm_kernel(const float* __restrict__ K, const float* __restrict__ qt,
                                                        const float* __restrict__ dDk, float* __restrict__ dqt_part,
                                                        int n, int m, int chunk, int nlc) {
    constexpr int BUF = 16 * D + 16 * 64;
    __shared__ __attribute__((aligned(16))) float sbuf[2 * BUF];
    const int ch = blockIdx.x, h = blockIdx.y, g = blockIdx.z, ng = gridDim.z;
    const int a = 64 * g + (int)threadIdx.x;   // landmark
    const bool live = a < m;
    const int ac = live ? a : m - 1;
    const int acol = ac - 64 * g;              // its column in the group's rows
    const float* Kh = K + (size_t)h * n * D;
    const float* DDh = dDk + (size_t)(h * ng + g) * n * 64;
    float q[D], acc[D];
#pragma unroll
    for (int c = 0; c < D; ++c) {
        q[c] = qt[((size_t)h * m + ac) * D + c];
        acc[c] = 0.f;
    }
    const int j0 = ch * chunk, j1 = min(n, j0 + chunk);
    auto stage = [&](int b, int t0) {
        stage_rows<16, D>(sbuf + b * BUF, Kh, t0, n);
        stage_rows<16, 64>(sbuf + b * BUF + 16 * D, DDh, t0, n);
    };
    if (j0 < j1) stage(0, j0);
    int buf = 0;
    for (int t0 = j0; t0 < j1; t0 += 16, buf ^= 1) {
        lds_dma_wait();
        __builtin_amdgcn_wave_barrier();
        if (t0 + 16 < j1) stage(buf ^ 1, t0 + 16);
        const float* sK = sbuf + buf * BUF;
        const float* sDD = sK + 16 * D;
#pragma unroll 4
        for (int r = 0; r < 16; ++r) {
            const float ddv = sDD[r * 64 + acol];
            const float dd = (live && t0 + r < j1) ? ddv : 0.f;
            const float dds = dd * 0x1p64f;
            const float* kr = sK + r * D;
#pragma unroll
            for (int c = 0; c < D; ++c) acc[c] = fmaf(dds, sgn_term(q[c], kr[c]), acc[c]);
        }
        __builtin_amdgcn_wave_barrier();
    }
    if (!live) return;
    const size_t o = ((size_t)h * nlc + ch) * m + a;
#pragma unroll
    for (int c = 0; c < D; ++c) dqt_part[o * D + c] = acc[c];
}

// ------------------------------------------------------------------------------------------
// Landmark-mean backward of the queries.  grid (m, BH), 256 threads: dq_l = dqtW_l + sum of the
// key-side partials (chunk order, fp64), then dQ_i += dq_l / |S_l| over the landmark's tokens:
// one contiguous run for a segment, r runs of r tokens for a window; four floats at a time.  The
// keys' share (dk_l, summed by the Newton-Schulz backward) is added by the key-major pass, which
// writes each dK row once.
__global__ __launch_bounds__(256) void bwd_pool_kernel(float* __restrict__ dQ, const float* __restrict__ dqtW,
                                                       const float* __restrict__ dqt_part, int n, int d, int m,
                                                       int nlc, LmPool pl) {
    const int l = blockIdx.x, h = blockIdx.y, tid = threadIdx.x;
    __shared__ float sq[64];
    const LmTokens tok = lm_tokens(pl, l, n, m);
    const int cntl = tok.count;
    const float inv = 1.f / (float)cntl;
    if (tid < d) {
        const size_t o = ((size_t)h * m + l) * d + tid;
        double aq = dqtW[o];
#pragma unroll 4
        for (int ch = 0; ch < nlc; ++ch) aq += dqt_part[(((size_t)h * nlc + ch) * m + l) * d + tid];
        sq[tid] = (float)aq * inv;
    }
    __syncthreads();
    const int runs = pl.r ? pl.r : 1, run_len = pl.r ? pl.r : cntl;
    for (int k = 0; k < runs; ++k) {
        const size_t base = ((size_t)h * n + tok(k * run_len)) * d;
        const int cnt4 = run_len * d / 4;
        float4* q4 = reinterpret_cast<float4*>(dQ + base);
        for (int e = tid; e < cnt4; e += 256) {
            const int c = (4 * e) % d;
            float4 a = q4[e];
            a.x += sq[c]; a.y += sq[c + 1]; a.z += sq[c + 2]; a.w += sq[c + 3];
            q4[e] = a;
        }
    }
}

// ------------------------------------------------------------------------------------------
// bf16 backward: widening of the inputs (exact) and rounding of the gradients (nearest even,
// NaN kept NaN), eight elements per thread and array, the first na of the arrays given.
// grid-stride over count / 8 groups.
__global__ __launch_bounds__(256) void widen_bf16_kernel(const uint16_t* __restrict__ a0, const uint16_t* __restrict__ a1,
                                                         const uint16_t* __restrict__ a2, const uint16_t* __restrict__ a3,
                                                         float* __restrict__ b0, float* __restrict__ b1,
                                                         float* __restrict__ b2, float* __restrict__ b3, size_t groups,
                                                         int na) {
    const uint16_t* src[4] = {a0, a1, a2, a3};
    float* dst[4] = {b0, b1, b2, b3};
    for (size_t gi = (size_t)blockIdx.x * 256 + threadIdx.x; gi < groups; gi += (size_t)gridDim.x * 256) {
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            if (t >= na) break;
            const uint4 v = reinterpret_cast<const uint4*>(src[t])[gi];
            const uint32_t w[4] = {v.x, v.y, v.z, v.w};
            float o[8];
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                o[2 * k] = __uint_as_float(w[k] << 16);
                o[2 * k + 1] = __uint_as_float(w[k] & 0xffff0000u);
            }
            reinterpret_cast<float4*>(dst[t])[2 * gi] = make_float4(o[0], o[1], o[2], o[3]);
            reinterpret_cast<float4*>(dst[t])[2 * gi + 1] = make_float4(o[4], o[5], o[6], o[7]);
        }
    }
}

__device__ __forceinline__ uint32_t bf16_rne(float x) {
    uint32_t u = __float_as_uint(x);
    if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) return (u >> 16) | 0x0040u;   // quiet NaN
    u += 0x7fffu + ((u >> 16) & 1u);
    return u >> 16;
}

__global__ __launch_bounds__(256) void narrow_bf16_kernel(const float* __restrict__ a0, const float* __restrict__ a1,
                                                          const float* __restrict__ a2, uint16_t* __restrict__ b0,
                                                          uint16_t* __restrict__ b1, uint16_t* __restrict__ b2,
                                                          size_t groups, int na) {
    const float* src[3] = {a0, a1, a2};
    uint16_t* dst[3] = {b0, b1, b2};
    for (size_t gi = (size_t)blockIdx.x * 256 + threadIdx.x; gi < groups; gi += (size_t)gridDim.x * 256) {
#pragma unroll
        for (int t = 0; t < 3; ++t) {
            if (t >= na) break;
            const float4 x = reinterpret_cast<const float4*>(src[t])[2 * gi];
            const float4 y = reinterpret_cast<const float4*>(src[t])[2 * gi + 1];
            uint4 o;
            o.x = bf16_rne(x.x) | (bf16_rne(x.y) << 16);
            o.y = bf16_rne(x.z) | (bf16_rne(x.w) << 16);
            o.z = bf16_rne(y.x) | (bf16_rne(y.y) << 16);
            o.w = bf16_rne(y.z) | (bf16_rne(y.w) << 16);
            reinterpret_cast<uint4*>(dst[t])[gi] = o;
        }
    }
}

hipError_t launch_widen_bf16(const uint16_t* Q, const uint16_t* K, const uint16_t* V, const uint16_t* G, float* wQ,
                             float* wK, float* wV, float* wG, size_t count, hipStream_t st) {
    const size_t groups = count / 8;
    const unsigned blocks = (unsigned)min((groups + 255) / 256, (size_t)4096);
    hipLaunchKernelGGL(widen_bf16_kernel, dim3(blocks), dim3(256), 0, st, Q, K, V, G, wQ, wK, wV, wG, groups,
                       G ? 4 : 3);
    return hipGetLastError();
}

hipError_t launch_narrow_bf16(const float* gQ, const float* gK, const float* gV, uint16_t* dQ, uint16_t* dK,
                              uint16_t* dV, size_t count, hipStream_t st) {
    const size_t groups = count / 8;
    const unsigned blocks = (unsigned)min((groups + 255) / 256, (size_t)4096);
    hipLaunchKernelGGL(narrow_bf16_kernel, dim3(blocks), dim3(256), 0, st, gQ, gK, gV, dQ, dK, dV, groups,
                       gK ? 3 : 1);
    return hipGetLastError();
}

// ------------------------------------------------------------------------------------------
// Launch wrappers.

hipError_t launch_bwd_query(int norm, const float* Q, const float* dO, float* dQ, const float* kt, const float* M,
                            const float* vbar, float* Aq, float* dDq, float* rs, float* dYd, float* dvbar_part,
                            float* p0_part, const float* whiten, const float* mvec, int saved, int BH, int H, int n,
                            int d, int m, float lambda, int nqb, hipStream_t st) {
    const float ks = kscale_of(lambda), il = 1.f / lambda;
    dim3 grid(nqb, BH);
#define LAPATTN_BQ(Dv, Nv, MPv)                                                                                  \
    hipLaunchKernelGGL((bwd_query_kernel<Dv, Nv, MPv>), grid, dim3(256), 0, st, Q, dO, dQ, kt, M, vbar, Aq, dDq, rs, \
                       dYd, dvbar_part, p0_part, whiten, mvec, saved, H, n, m, ks, il, nqb)
#define LAPATTN_BQN(Dv, MPv)                                        \
    do {                                                            \
        if (norm == NORM_INLINE) LAPATTN_BQ(Dv, NORM_INLINE, MPv);   \
        else if (norm == NORM_ROWSUM) LAPATTN_BQ(Dv, NORM_ROWSUM, MPv); \
        else if (norm == NORM_MSPACE) LAPATTN_BQ(Dv, NORM_MSPACE, MPv); \
        else LAPATTN_BQ(Dv, NORM_NONE, MPv);                         \
    } while (0)
    if (m <= 64) {
        if (d == 32) LAPATTN_BQN(32, 64);
        else LAPATTN_BQN(64, 64);
    } else {
        if (d == 32) LAPATTN_BQN(32, 128);
        else LAPATTN_BQN(64, 128);
    }
#undef LAPATTN_BQN
#undef LAPATTN_BQ
    return hipGetLastError();
}

hipError_t launch_bwd_query_lm(const float* Q, const float* dO, const float* kt, const float* Aq, const float* dDq,
                               const float* rs, const float* dYd, float* dM_part, float* dkt_part, int BH, int n,
                               int d, int m, int chunk, int nlc, hipStream_t st) {
    dim3 grid(nlc, BH, (m + 63) / 64);
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
                         float* dkpool, const float* dkt_part, LmPool pl, const float* p0_part, const float* whiten,
                         int mspace, float* dDW, int BH, int H, int n, int d, int m, int T, double lambda, double eps,
                         int nlc, int nqb, int MP, hipStream_t st) {
#define LAPATTN_BNS(MPv, Dv)                                                                                      \
    hipLaunchKernelGGL((bwd_ns_kernel<MPv, Dv>), dim3(BH), dim3(256), 0, st, qt, kt, Xs, cinfo, U, dM_part,       \
                       dvbar_part, dU, dvbar, dqtW, dkpool, dkt_part, pl, p0_part, whiten, mspace, dDW, H, n, m, T,  \
                       lambda, eps, nlc, nqb)
    if (MP == 32 && d == 32) LAPATTN_BNS(32, 32);
    else if (MP == 32) LAPATTN_BNS(32, 64);
    else if (d == 32) LAPATTN_BNS(64, 32);
    else LAPATTN_BNS(64, 64);
#undef LAPATTN_BNS
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_kll_backward(qt, kt, dDW, dqtW, dkpool, dkt_part, pl, BH, n, d, m, MP, nlc, st);
}

hipError_t launch_bwd_key(const float* K, const float* V, float* dK, float* dV, const float* qt, const float* dU,
                          const float* dvbar, float* dDk, const float* dkpool, LmPool pl, int saved, int BH, int n,
                          int d, int m, float lambda, hipStream_t st) {
    const float ks = kscale_of(lambda), il = 1.f / lambda;
    dim3 grid((n + 255) / 256, BH);
#define LAPATTN_BK(Dv, MPv)                                                                                      \
    hipLaunchKernelGGL((bwd_key_kernel<Dv, MPv>), grid, dim3(256), 0, st, K, V, dK, dV, qt, dU, dvbar, dDk, dkpool, \
                       pl, saved, n, m, ks, il)
    if (m <= 64) {
        if (d == 32) LAPATTN_BK(32, 64);
        else LAPATTN_BK(64, 64);
    } else {
        if (d == 32) LAPATTN_BK(32, 128);
        else LAPATTN_BK(64, 128);
    }
#undef LAPATTN_BK
    return hipGetLastError();
}

hipError_t launch_bwd_key_lm(const float* K, const float* qt, const float* dDk, float* dqt_part, int BH, int n, int d,
                             int m, int chunk, int nlc, hipStream_t st) {
    dim3 grid(nlc, BH, (m + 63) / 64);
    if (d == 32)
        hipLaunchKernelGGL((bwd_key_lm_kernel<32>), grid, dim3(64), 0, st, K, qt, dDk, dqt_part, n, m, chunk, nlc);
    else
        hipLaunchKernelGGL((bwd_key_lm_kernel<64>), grid, dim3(64), 0, st, K, qt, dDk, dqt_part, n, m, chunk, nlc);
    return hipGetLastError();
}

hipError_t launch_bwd_pool(float* dQ, const float* dqtW, const float* dqt_part, int BH, int n, int d, int m, int nlc,
                           LmPool pl, hipStream_t st) {
    hipLaunchKernelGGL(bwd_pool_kernel, dim3(m, BH), dim3(256), 0, st, dQ, dqtW, dqt_part, n, d, m, nlc, pl);
    return hipGetLastError();
}

}  // namespace lapattn
