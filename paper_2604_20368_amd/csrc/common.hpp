// common.hpp -- small device helpers shared by the lapattn HIP kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lapattn {

enum { DT_F32 = 0, DT_BF16 = 1 };
enum { NORM_INLINE = 0, NORM_ROWSUM = 1, NORM_NONE = 2, NORM_MSPACE = 3 };

// Element access for the two storage types.  bf16 is carried as raw 16-bit
// patterns; widening is exact, narrowing rounds to nearest even.
template <int DT> struct elem;
template <> struct elem<DT_F32> {
    using type = float;
    static __device__ __forceinline__ float load(const float* p, size_t i) { return p[i]; }
    static __device__ __forceinline__ void store(float* p, size_t i, float v) { p[i] = v; }
};
template <> struct elem<DT_BF16> {
    using type = uint16_t;
    static __device__ __forceinline__ float load(const uint16_t* p, size_t i) {
        return __uint_as_float(((uint32_t)p[i]) << 16);
    }
    static __device__ __forceinline__ void store(uint16_t* p, size_t i, float v) {
        uint32_t u = __float_as_uint(v);
        if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu)) {
            p[i] = (uint16_t)((u >> 16) | 0x0040u);           // quiet NaN stays NaN
        } else {
            u += 0x7fffu + ((u >> 16) & 1u);                  // round to nearest even
            p[i] = (uint16_t)(u >> 16);
        }
    }
};

// Fixed-point L1 distances of the one-launch small-head forward.  Every kernel value of a head is
// exp(-||x - y||_1 / lambda) with x, y rows of Q, K or their landmark means, all of magnitude at
// most R = max |x| over the head's Q and K.  With s = 2^(22 - e), R < 2^e, a coordinate is coded as the bits of
// fmaf(x, s, 1.5 2^23): for |x s| <= 2^22 that float lies in [2^23, 2^24], where consecutive
// floats are consecutive integers, so the bits are 0x4B000000 + 2^22 + round(x s) and the
// difference of two codes is the difference of the rounded scaled coordinates.  One v_sad_u32
// per coordinate then adds |x_c - y_c| s exactly (a row's sum stays below 64 2^23 = 2^29).  The
// rounding moves a coordinate by at most 2^(e - 23) <= R 2^-22, a distance by at most d times
// that (typically a few times); the fp32 sums of differences carry errors of the same order.
// fgrid: s and kss = -log2(e) / (lambda s) from R and ks = -log2(e) / lambda; e >= -100 (a tiny R
// gets a coarser grid: its distances are below 2^-100).  R must be finite.
__device__ __forceinline__ void fgrid(float R, float ks, float& s, float& kss) {
    int e = 0;
    (void)frexpf(R, &e);   // R < 2^e (e = 0 for R = 0)
    e = e < -100 ? -100 : e;
    s = __uint_as_float((uint32_t)(127 + 22 - e) << 23);
    kss = ks * __uint_as_float((uint32_t)(127 - 22 + e) << 23);
}
__device__ __forceinline__ uint32_t fcode(float x, float s) { return __float_as_uint(fmaf(x, s, 12582912.f)); }
// Kernel value from a coded distance.
__device__ __forceinline__ float fkval(uint32_t dist, float kss) { return __builtin_amdgcn_exp2f((float)dist * kss); }
// |x - y| + acc on unsigned 32-bit integers (v_sad_u32).
__device__ __forceinline__ uint32_t sad32(uint32_t x, uint32_t y, uint32_t acc) {
    uint32_t r;
    asm("v_sad_u32 %0, %1, %2, %3" : "=v"(r) : "v"(x), "v"(y), "v"(acc));
    return r;
}

// Landmark segments: segment l covers tokens [floor(l n/m), floor((l+1) n/m)).
__device__ __host__ __forceinline__ int seg_start(int l, int n, int m) {
    return (int)(((long long)l * n) / m);
}
// The segment holding token i: the largest l with seg_start(l) <= i.
__device__ __host__ __forceinline__ int seg_of(int i, int n, int m) {
    return (int)((((long long)i + 1) * m - 1) / n);
}

// Landmark l's tokens (Sec. 4.2 sampling): with r == 0 the balanced segment above; otherwise
// the tokens form a row-major map of width gw (height n / gw, both multiples of r) and
// landmark l = Y (gw / r) + X averages the r x r window at rows Y r.., columns X r.. .
struct LmPool {
    int gw, r;
};
// One landmark's tokens: count, and the t-th token (window tokens in row-major order).
struct LmTokens {
    int count, s0, r, gw, y0, x0;
    __device__ __host__ __forceinline__ int operator()(int t) const {
        return r ? (y0 + t / r) * gw + x0 + t % r : s0 + t;
    }
};
__device__ __host__ __forceinline__ LmTokens lm_tokens(LmPool p, int l, int n, int m) {
    LmTokens k;
    k.r = p.r;
    k.gw = p.gw;
    if (!p.r) {
        k.s0 = seg_start(l, n, m);
        k.count = seg_start(l + 1, n, m) - k.s0;
        k.y0 = k.x0 = 0;
    } else {
        const int mw = p.gw / p.r;
        k.s0 = 0;
        k.count = p.r * p.r;
        k.y0 = (l / mw) * p.r;
        k.x0 = (l % mw) * p.r;
    }
    return k;
}

// A wave's [row][column] tile of pitch 65 (rows r0 .. r0+63) into a [n][64] row array: lane l
// moves column l of 16 rows at a time, so that 16 accesses are in flight; rows past n and
// columns past m are skipped.
__device__ __forceinline__ void store_rows64(float* __restrict__ dst, const float* __restrict__ tile, int r0, int n,
                                             int m) {
    const int l = (int)(threadIdx.x & 63);
    float* col = dst + (size_t)r0 * 64 + l;   // rows at constant offsets from one address
#pragma unroll 1
    for (int b = 0; b < 64; b += 16) {
        float v[16];
#pragma unroll
        for (int t = 0; t < 16; ++t) v[t] = tile[(b + t) * 65 + l];
#pragma unroll
        for (int t = 0; t < 16; ++t)
            if (l < m && r0 + b + t < n) col[(b + t) * 64] = v[t];
    }
}

// Rows r0 .. r0 + 63 of a 64 x 32 half tile (pitch 33) into columns c0 .. c0 + mh - 1 of dst
// ([n][64]); rows past n are skipped.  Lanes 0..31 and 32..63 take two rows per store.
__device__ __forceinline__ void store_half_rows(float* __restrict__ dst, const float* __restrict__ tile, int r0,
                                                int n, int c0, int mh) {
    const int l = (int)(threadIdx.x & 63), c = l & 31, rh = l >> 5;
    float* col = dst + (size_t)(r0 + rh) * 64 + c0 + c;   // rows at constant offsets from one address
#pragma unroll 1
    for (int b = 0; b < 64; b += 32) {
        float v[16];
#pragma unroll
        for (int t = 0; t < 16; ++t) v[t] = tile[(b + 2 * t + rh) * 33 + c];
#pragma unroll
        for (int t = 0; t < 16; ++t)
            if (c < mh && r0 + rh + b + 2 * t < n) col[(b + 2 * t) * 64] = v[t];
    }
}

// Blocks are dispatched to the 8 XCDs round-robin (block i to XCD i % 8).  xcd_order maps block i
// of n to a logical index such that each XCD's blocks get a contiguous range: a bijection of [0, n).
__device__ __forceinline__ int xcd_order(int i, int n) {
    const int x = i & 7, y = i >> 3;
    int off = 0;
    for (int xp = 0; xp < x; ++xp) off += xp < n ? (n - xp + 7) >> 3 : 0;
    return off + y;
}

__device__ __forceinline__ float sgnf(float x) { return (float)((x > 0.f) - (x < 0.f)); }
__device__ __forceinline__ double sgnd(double x) { return (double)((x > 0.0) - (x < 0.0)); }

}  // namespace lapattn
