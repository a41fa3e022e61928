// dwc.hip -- the depth-wise convolution branch of Eq. (7), Out = Z V + DWC(V): each value
// channel c of head h is cross-correlated over the row-major H' x W' token map with its own
// k x k filter (k odd, stride 1, zero padding (k-1)/2), plus an optional per-channel bias.
// Filters are [H][d][k][k] fp32 and shared by the batch.
//
//   dwc_fwd_kernel       E = DWC(V) + bias in fp32; the query kernels add E to the normalised
//                        output before rounding it to the output type
//   dwc_bwd_dv_kernel    dV += DWC^T(dOut): the filter applied at the mirrored offsets
//   dwc_bwd_w_kernel     per token chunk: sum_i dOut_i V_{i + offset} for every tap, and
//                        sum_i dOut_i for the bias
//   dwc_bwd_w_reduce     the chunk partials summed over the batch and the chunks in a fixed order
//
// HBM-bound elementwise stencils: a thread owns one token and four consecutive channels, so a
// wave's loads of one tap cover whole 128- or 256-byte rows of V (or dOut); the neighbours'
// rows come back from L1/L2, each row of V being read by up to k^2 tokens.
#include "kernels.hpp"

namespace lapattn {

constexpr int kDwcMaxK = 7;

template <int DT>
__device__ __forceinline__ float4 load4(const typename elem<DT>::type* __restrict__ p, size_t i);
template <>
__device__ __forceinline__ float4 load4<DT_F32>(const float* __restrict__ p, size_t i) {
    return *reinterpret_cast<const float4*>(p + i);
}
template <>
__device__ __forceinline__ float4 load4<DT_BF16>(const uint16_t* __restrict__ p, size_t i) {
    const uint2 u = *reinterpret_cast<const uint2*>(p + i);
    return make_float4(__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u), __uint_as_float(u.y << 16),
                       __uint_as_float(u.y & 0xffff0000u));
}

__device__ __forceinline__ void fma4(float4& acc, float4 a, float4 b) {
    acc.x = fmaf(a.x, b.x, acc.x);
    acc.y = fmaf(a.y, b.y, acc.y);
    acc.z = fmaf(a.z, b.z, acc.z);
    acc.w = fmaf(a.w, b.w, acc.w);
}

// The head's filters in LDS as [tap][c], so that four channels of one tap are one float4.
template <int D>
__device__ __forceinline__ void stage_filters(float* __restrict__ sw, const float* __restrict__ W, int h, int kk) {
    for (int e = threadIdx.x; e < kk * D; e += blockDim.x) sw[e] = W[((size_t)h * D + e % D) * kk + e / D];
}

// grid (ceil(n D/4 / 256), B*H), 256 threads; thread = (token i, channels c0 .. c0+3).
template <int DT, int D>
__global__ __launch_bounds__(256) void dwc_fwd_kernel(const typename elem<DT>::type* __restrict__ V,
                                                      const float* __restrict__ W, const float* __restrict__ bias,
                                                      float* __restrict__ E, int n, int H, int gw, int k) {
    constexpr int NG = D / 4;
    __shared__ __attribute__((aligned(16))) float sw[kDwcMaxK * kDwcMaxK * D];
    __shared__ __attribute__((aligned(16))) float sb[D];
    const int bh = blockIdx.y, h = bh % H, kk = k * k, tid = threadIdx.x;
    stage_filters<D>(sw, W, h, kk);
    if (tid < D) sb[tid] = bias ? bias[h * D + tid] : 0.f;
    __syncthreads();
    const long long gid = (long long)blockIdx.x * 256 + tid;
    const int i = (int)(gid / NG), c0 = (int)(gid % NG) * 4;
    if (i >= n) return;
    const int gh = n / gw, y = i / gw, x = i % gw, p = (k - 1) / 2;
    const size_t base = (size_t)bh * n * D + c0;
    float4 acc = *reinterpret_cast<const float4*>(sb + c0);
    for (int u = 0; u < k; ++u) {
        const int yy = y + u - p;
        if (yy < 0 || yy >= gh) continue;
        for (int t = 0; t < k; ++t) {
            const int xx = x + t - p;
            if (xx < 0 || xx >= gw) continue;
            fma4(acc, *reinterpret_cast<const float4*>(sw + (u * k + t) * D + c0),
                 load4<DT>(V, base + (size_t)(yy * gw + xx) * D));
        }
    }
    *reinterpret_cast<float4*>(E + base + (size_t)i * D) = acc;
}

// dV_j += sum over taps of w[u][t] dOut_{j - (u - p, t - p)}; same grid as the forward.
template <int D>
__global__ __launch_bounds__(256) void dwc_bwd_dv_kernel(const float* __restrict__ G, const float* __restrict__ W,
                                                         float* __restrict__ dV, int n, int H, int gw, int k) {
    constexpr int NG = D / 4;
    __shared__ __attribute__((aligned(16))) float sw[kDwcMaxK * kDwcMaxK * D];
    const int bh = blockIdx.y, h = bh % H, kk = k * k, tid = threadIdx.x;
    stage_filters<D>(sw, W, h, kk);
    __syncthreads();
    const long long gid = (long long)blockIdx.x * 256 + tid;
    const int j = (int)(gid / NG), c0 = (int)(gid % NG) * 4;
    if (j >= n) return;
    const int gh = n / gw, y = j / gw, x = j % gw, p = (k - 1) / 2;
    const size_t base = (size_t)bh * n * D + c0;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int u = 0; u < k; ++u) {
        const int yy = y - (u - p);
        if (yy < 0 || yy >= gh) continue;
        for (int t = 0; t < k; ++t) {
            const int xx = x - (t - p);
            if (xx < 0 || xx >= gw) continue;
            fma4(acc, *reinterpret_cast<const float4*>(sw + (u * k + t) * D + c0),
                 *reinterpret_cast<const float4*>(G + base + (size_t)(yy * gw + xx) * D));
        }
    }
    float4* o = reinterpret_cast<float4*>(dV + base + (size_t)j * D);
    float4 v = *o;
    v.x += acc.x;
    v.y += acc.y;
    v.z += acc.z;
    v.w += acc.w;
    *o = v;
}

// grid (nch, B*H), 256 threads.  Chunk ch covers tokens [ch*chunk, min(n, (ch+1)*chunk)).
// Thread job = (tap, channels c0..c0+3); tap k*k is the bias.  part[bh][ch][c][tap], k*k+1 taps.
template <int D>
__global__ __launch_bounds__(256) void dwc_bwd_w_kernel(const float* __restrict__ G, const float* __restrict__ V,
                                                        float* __restrict__ part, int n, int gw, int k, int chunk,
                                                        int nch) {
    constexpr int NG = D / 4;
    const int bh = blockIdx.y, ch = blockIdx.x, kk = k * k, ntap = kk + 1;
    const int i0 = ch * chunk, i1 = min(n, i0 + chunk);
    const int gh = n / gw, p = (k - 1) / 2;
    const float* g = G + (size_t)bh * n * D;
    const float* v = V + (size_t)bh * n * D;
    float* dst = part + ((size_t)bh * nch + ch) * D * ntap;
    for (int job = threadIdx.x; job < NG * ntap; job += 256) {
        const int c0 = (job % NG) * 4, tap = job / NG;
        float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
        if (tap == kk) {
            for (int i = i0; i < i1; ++i) {
                const float4 gi = *reinterpret_cast<const float4*>(g + (size_t)i * D + c0);
                acc.x += gi.x;
                acc.y += gi.y;
                acc.z += gi.z;
                acc.w += gi.w;
            }
        } else {
            const int du = tap / k - p, dx = tap % k - p;
            int y = i0 / gw, x = i0 % gw;
            for (int i = i0; i < i1; ++i) {
                const int yy = y + du, xx = x + dx;
                if (yy >= 0 && yy < gh && xx >= 0 && xx < gw)
                    fma4(acc, *reinterpret_cast<const float4*>(g + (size_t)i * D + c0),
                         *reinterpret_cast<const float4*>(v + (size_t)(yy * gw + xx) * D + c0));
                if (++x == gw) {
                    x = 0;
                    ++y;
                }
            }
        }
        dst[(c0 + 0) * ntap + tap] = acc.x;
        dst[(c0 + 1) * ntap + tap] = acc.y;
        dst[(c0 + 2) * ntap + tap] = acc.z;
        dst[(c0 + 3) * ntap + tap] = acc.w;
    }
}

// One thread per (h, c, tap): the partials of every batch entry and chunk, in that order, in fp64.
__global__ __launch_bounds__(256) void dwc_bwd_w_reduce(const float* __restrict__ part, float* __restrict__ dW,
                                                        float* __restrict__ db, int B, int H, int d, int k, int nch) {
    const int kk = k * k, ntap = kk + 1;
    const int e = blockIdx.x * 256 + threadIdx.x;
    if (e >= H * d * ntap) return;
    const int h = e / (d * ntap), c = (e / ntap) % d, tap = e % ntap;
    double s = 0.0;
    for (int b = 0; b < B; ++b)
        for (int ch = 0; ch < nch; ++ch) s += part[(((size_t)(b * H + h) * nch + ch) * d + c) * ntap + tap];
    if (tap < kk) {
        if (dW) dW[((size_t)h * d + c) * kk + tap] = (float)s;
    } else if (db) {
        db[h * d + c] = (float)s;
    }
}

// ------------------------------------------------------------------------------------------
// Launch wrappers.

static dim3 dwc_grid(int BH, int n, int d) { return dim3((unsigned)(((long long)n * (d / 4) + 255) / 256), BH); }

hipError_t launch_dwc_fwd(int dt, const void* V, const float* W, const float* bias, float* E, int BH, int H, int n,
                          int d, int gw, int k, hipStream_t st) {
    if (k < 1 || k > kDwcMaxK || k % 2 == 0 || gw < 1 || n % gw) return hipErrorInvalidValue;
    const dim3 grid = dwc_grid(BH, n, d);
#define LAPATTN_DWC(DTv, Dv)                                                                                        \
    hipLaunchKernelGGL((dwc_fwd_kernel<DTv, Dv>), grid, dim3(256), 0, st,                                          \
                       static_cast<const typename elem<DTv>::type*>(V), W, bias, E, n, H, gw, k)
    if (dt == DT_F32 && d == 32) LAPATTN_DWC(DT_F32, 32);
    else if (dt == DT_F32) LAPATTN_DWC(DT_F32, 64);
    else if (d == 32) LAPATTN_DWC(DT_BF16, 32);
    else LAPATTN_DWC(DT_BF16, 64);
#undef LAPATTN_DWC
    return hipGetLastError();
}

hipError_t launch_dwc_bwd_dv(const float* G, const float* W, float* dV, int BH, int H, int n, int d, int gw, int k,
                             hipStream_t st) {
    if (k < 1 || k > kDwcMaxK || k % 2 == 0 || gw < 1 || n % gw) return hipErrorInvalidValue;
    const dim3 grid = dwc_grid(BH, n, d);
    if (d == 32) hipLaunchKernelGGL((dwc_bwd_dv_kernel<32>), grid, dim3(256), 0, st, G, W, dV, n, H, gw, k);
    else hipLaunchKernelGGL((dwc_bwd_dv_kernel<64>), grid, dim3(256), 0, st, G, W, dV, n, H, gw, k);
    return hipGetLastError();
}

hipError_t launch_dwc_bwd_w(const float* G, const float* V, float* part, float* dW, float* db, int B, int H, int n,
                            int d, int gw, int k, int chunk, hipStream_t st) {
    if (k < 1 || k > kDwcMaxK || k % 2 == 0 || gw < 1 || n % gw || chunk < 1) return hipErrorInvalidValue;
    const int nch = (n + chunk - 1) / chunk;
    const dim3 grid(nch, B * H);
    if (d == 32) hipLaunchKernelGGL((dwc_bwd_w_kernel<32>), grid, dim3(256), 0, st, G, V, part, n, gw, k, chunk, nch);
    else hipLaunchKernelGGL((dwc_bwd_w_kernel<64>), grid, dim3(256), 0, st, G, V, part, n, gw, k, chunk, nch);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int jobs = H * d * (k * k + 1);
    hipLaunchKernelGGL(dwc_bwd_w_reduce, dim3((jobs + 255) / 256), dim3(256), 0, st, part, dW, db, B, H, d, k, nch);
    return hipGetLastError();
}

}  // namespace lapattn
