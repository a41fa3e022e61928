// ns_mfma.hpp -- building blocks of the Newton-Schulz solve (Algorithm 2) and of its backward,
// for one workgroup of 256 threads (four waves) per head: the kernel matrix K_LL, block products
// on the fp64 matrix cores (v_mfma_f64_16x16x4_f64) and MP x MP products on the fp32 ones
// (v_mfma_f32_16x16x4f32, ns32_mm at the end).
//
// Product layout.  A product C = op(A) op(B) of R x N (R, N multiples of 16, (R/16)(N/16) a
// multiple of 4) is cut into 16 x 16 tiles numbered row-major; wave w owns tiles w, w + 4,
// w + 8, ...  Register j of a tile's accumulator at lane l holds row 16 tr + l / 16 + 4 j,
// column 16 tc + l % 16 of that tile (tr, tc): the fp64 16x16x4 result layout, which interleaves
// the rows differently from the fp32 one.  Every operand comes
// from LDS; A is R x KD row-major with pitch PA (TA: A is held transposed, KD x R), B is KD x N
// with pitch PB (TB: held transposed, N x KD).
//
// LDS pitch.  One operand read of a wave covers 16 rows x 4 consecutive columns of a row-major
// matrix (lanes l % 16 = row, l / 16 = column).  With a pitch of 4 mod 32 doubles those 64 lanes
// fall on 32 distinct 8-byte bank pairs twice over, the minimum of two passes; operands read
// the other way round (4 rows x 16 columns) take four.
#pragma once

#include <hip/hip_runtime.h>

namespace lapattn {

typedef double f64x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

// Row pitch (doubles) of an LDS matrix with `cols` columns: cols rounded up to 4 mod 32.
__host__ __device__ constexpr int ns_pitch(int cols) { return cols + ((36 - cols % 32) % 32); }

template <int R, int N>
struct ns_tiles {
    static constexpr int TC = N / 16;                  // tile columns
    static constexpr int NT = (R / 16) * TC / 4;       // tiles per wave
    static_assert(R % 16 == 0 && N % 16 == 0 && ((R / 16) * TC) % 4 == 0, "tile count");
    // Row / column of register j of this lane's t-th tile.
    static __device__ __forceinline__ int row(int t, int j) {
        const int tile = (int)(threadIdx.x >> 6) + 4 * t;
        return 16 * (tile / TC) + (int)((threadIdx.x & 63) >> 4) + 4 * j;
    }
    static __device__ __forceinline__ int col(int t) {
        const int tile = (int)(threadIdx.x >> 6) + 4 * t;
        return 16 * (tile % TC) + (int)(threadIdx.x & 15);
    }
};

// acc[t] = tile t of op(A) op(B) (overwritten).
template <int R, int N, int KD, bool TA, bool TB, int PA, int PB>
__device__ __forceinline__ void ns_mm(const double* __restrict__ A, const double* __restrict__ B,
                                      f64x4_t (&acc)[ns_tiles<R, N>::NT]) {
    using L = ns_tiles<R, N>;
    static_assert(KD % 4 == 0, "contraction length");
    const int w = (int)(threadIdx.x >> 6), li = (int)(threadIdx.x & 15), lk = (int)((threadIdx.x & 63) >> 4);
#pragma unroll
    for (int t = 0; t < L::NT; ++t) acc[t] = f64x4_t{0.0, 0.0, 0.0, 0.0};
#pragma unroll
    for (int s = 0; s < KD / 4; ++s) {
        const int k = 4 * s + lk;
#pragma unroll
        for (int t = 0; t < L::NT; ++t) {
            const int tile = w + 4 * t;
            const int r = 16 * (tile / L::TC) + li, c = 16 * (tile % L::TC) + li;
            const double a = TA ? A[k * PA + r] : A[r * PA + k];
            const double b = TB ? B[c * PB + k] : B[k * PB + c];
            acc[t] = __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, acc[t], 0, 0, 0);
        }
    }
}

// Store this wave's tiles of an R x N product (times `scale`) row-major with pitch P.
template <int R, int N, int P>
__device__ __forceinline__ void ns_store(double* __restrict__ S, const f64x4_t (&acc)[ns_tiles<R, N>::NT],
                                         double scale = 1.0) {
    using L = ns_tiles<R, N>;
#pragma unroll
    for (int t = 0; t < L::NT; ++t)
#pragma unroll
        for (int j = 0; j < 4; ++j) S[L::row(t, j) * P + L::col(t)] = scale * acc[t][j];
}

// An MP x MP fp64 matrix from global memory (pitch MP) into registers, MP*MP/256 entries per
// thread, every load issued before any is used.
template <int MP>
__device__ __forceinline__ void ns_fetch(double (&v)[MP * MP / 256], const double* __restrict__ G) {
#pragma unroll
    for (int r = 0; r < MP * MP / 256; ++r) v[r] = G[threadIdx.x + 256 * r];
}
template <int MP, int P>
__device__ __forceinline__ void ns_put(double* __restrict__ S, const double (&v)[MP * MP / 256]) {
#pragma unroll
    for (int r = 0; r < MP * MP / 256; ++r) {
        const int e = (int)threadIdx.x + 256 * r;
        S[(e / MP) * P + e % MP] = v[r];
    }
}
template <int MP, int P>
__device__ __forceinline__ void ns_load(double* __restrict__ S, const double* __restrict__ G) {
    double v[MP * MP / 256];
    ns_fetch<MP>(v, G);
    ns_put<MP, P>(S, v);
}

// The first `count` floats of src into LDS, zero-padded to MP * D; loads unconditional (clamped
// index) so that they are all in flight together.
template <int MP, int D>
__device__ __forceinline__ void ns_stage_rows(float* __restrict__ dst, const float* __restrict__ src, int count) {
    constexpr int NE = (MP * D + 255) / 256;
    float v[NE];
#pragma unroll
    for (int r = 0; r < NE; ++r) v[r] = src[min((int)threadIdx.x + 256 * r, count - 1)];
#pragma unroll
    for (int r = 0; r < NE; ++r) {
        const int e = (int)threadIdx.x + 256 * r;
        if (e < MP * D) dst[e] = (e < count) ? v[r] : 0.f;
    }
}

// W = K_LL + eps I (Algorithm 2 input; K_LL of the landmark means, Eq. (C)) into LDS, row pitch P,
// zero outside m x m.  The query landmark rows are staged in `sq` (MP x D floats of LDS, free on
// entry, still read on exit: the caller synchronises before reusing it).  Thread (a-group,
// b = tid % MP) keeps its key landmark row in registers (fp64); the L1 distance and the
// exponential are fp64.  Called by all 256 threads.
template <int MP, int D, int P>
__device__ __forceinline__ void ns_kll(const float* __restrict__ q, const float* __restrict__ k, double* __restrict__ sW,
                                       float* __restrict__ sq, int m, double lambda, double eps) {
    constexpr int AG = 256 / MP;                       // rows a handled per pass
    const int tid = (int)threadIdx.x;
    ns_stage_rows<MP, D>(sq, q, m * D);
    const int b = tid % MP;
    double kb[D];
#pragma unroll
    for (int c = 0; c < D; ++c) kb[c] = (b < m) ? (double)k[b * D + c] : 0.0;
    __syncthreads();
    for (int a = tid / MP; a < MP; a += AG) {
        double w = 0.0;
        if (a < m && b < m) {
            const float* qa = sq + a * D;
            double dist = 0.0;
#pragma unroll
            for (int c = 0; c < D; ++c) dist += fabs((double)qa[c] - kb[c]);
            w = exp(-dist / lambda);
            if (a == b) w += eps;
        }
        sW[a * P + b] = w;
    }
}

// Maximum of v over each group of G consecutive lanes (G a power of two, at most 64) and the
// lowest index within the group that holds it (butterfly: every lane ends with its group's
// result).  NaN must be mapped below every candidate by the caller.
template <int G>
__device__ __forceinline__ void ns_group_argmax(double& v, int& idx) {
#pragma unroll
    for (int off = G / 2; off >= 1; off >>= 1) {
        const double ov = __shfl_xor(v, off, 64);
        const int oi = __shfl_xor(idx, off, 64);
        if (ov > v || (ov == v && oi < idx)) {
            v = ov;
            idx = oi;
        }
    }
}


// fp32 products C = A B of MP x MP matrices (MP = 32 or 64) on v_mfma_f32_16x16x4f32 (ns32_mm),
// for the Newton-Schulz iterations and their backward: 16 x 16 tiles, wave w owns column block w
// (MP = 64: all four row blocks) or tile (w / 2, w % 2) (MP = 32).  The contraction is split over
// the four lane groups (group g takes k = g MP/4 .. g MP/4 + MP/4 - 1, one per MFMA), so that a
// lane's operands are contiguous runs of A's row and of B's column: B is passed transposed.
// LDS matrices have a row pitch of MP + 4 floats (16-byte reads of 16 rows fall on distinct
// banks).
template <int MP>
struct ns32_tiles {
    static constexpr int KS = MP / 4;               // k values per lane group
    static constexpr int NT = MP == 64 ? 4 : 1;     // tiles per wave
    static constexpr int P = MP + 4;                // row pitch (floats) of the LDS matrices
    static __device__ __forceinline__ int tc() {
        const int w = (int)(threadIdx.x >> 6);
        return MP == 64 ? w : (w & 1);
    }
    static __device__ __forceinline__ int tr(int t) {
        const int w = (int)(threadIdx.x >> 6);
        return MP == 64 ? t : (w >> 1);
    }
};

// acc[t] = tile t of A B, A row-major and BT = B^T row-major (pitch P each).  Register r of tile t
// at lane l holds row 16 tr(t) + 4 (l / 16) + r, column 16 tc + l % 16.
template <int MP>
__device__ __forceinline__ void ns32_mm(const float* __restrict__ A, const float* __restrict__ BT,
                                        f32x4_t (&acc)[ns32_tiles<MP>::NT]) {
    using L = ns32_tiles<MP>;
    const int l = (int)(threadIdx.x & 63), li = l & 15, g = l >> 4;
    float b[L::KS];
    const float* bp = BT + (16 * L::tc() + li) * L::P + g * L::KS;
#pragma unroll
    for (int s4 = 0; s4 < L::KS / 4; ++s4) {
        const float4 v = reinterpret_cast<const float4*>(bp)[s4];
        b[4 * s4] = v.x; b[4 * s4 + 1] = v.y; b[4 * s4 + 2] = v.z; b[4 * s4 + 3] = v.w;
    }
    float a[L::NT][L::KS];
#pragma unroll
    for (int t = 0; t < L::NT; ++t) {
        const float* ap = A + (16 * L::tr(t) + li) * L::P + g * L::KS;
#pragma unroll
        for (int s4 = 0; s4 < L::KS / 4; ++s4) {
            const float4 v = reinterpret_cast<const float4*>(ap)[s4];
            a[t][4 * s4] = v.x; a[t][4 * s4 + 1] = v.y; a[t][4 * s4 + 2] = v.z; a[t][4 * s4 + 3] = v.w;
        }
        acc[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    }
    // k outer, tiles inner: consecutive MFMAs are independent
#pragma unroll
    for (int s = 0; s < L::KS; ++s)
#pragma unroll
        for (int t = 0; t < L::NT; ++t) acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[t][s], b[s], acc[t], 0, 0, 0);
}

// Row and column of register j of tile t of an ns32_mm result at this lane.
template <int MP>
__device__ __forceinline__ int ns32_row(int t, int j) {
    return 16 * ns32_tiles<MP>::tr(t) + 4 * (int)((threadIdx.x & 63) >> 4) + j;
}
template <int MP>
__device__ __forceinline__ int ns32_col() {
    return 16 * ns32_tiles<MP>::tc() + (int)(threadIdx.x & 15);
}

}  // namespace lapattn
