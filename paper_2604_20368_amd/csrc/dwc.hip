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

// The neighbour of map position (y, x) at offset (dy, dx): its token, clamped into the map, and
// whether it lies on the map.  The loads of all taps are issued unconditionally (a tap off the
// map reads a clamped row and is given weight 0), so they are in flight together.
struct Nbr {
    int j;
    bool in;
};
__device__ __forceinline__ Nbr nbr(int y, int x, int dy, int dx, int gh, int gw) {
    const int yy = y + dy, xx = x + dx;
    Nbr r;
    r.in = yy >= 0 && yy < gh && xx >= 0 && xx < gw;
    r.j = min(max(yy, 0), gh - 1) * gw + min(max(xx, 0), gw - 1);
    return r;
}

// grid (x, B*H), 256 threads; a thread takes (token i, channels c0 .. c0+3) items of its head
// with a stride of x * 256 items, so that each block stages its head's filters once for
// several items.
template <int DT, int D, int K>
__global__ __launch_bounds__(256) void dwc_fwd_kernel(const typename elem<DT>::type* __restrict__ V,
                                                      const float* __restrict__ W, const float* __restrict__ bias,
                                                      float* __restrict__ E, int n, int H, int gw) {
    constexpr int NG = D / 4, P = (K - 1) / 2;
    __shared__ __attribute__((aligned(16))) float sw[K * K * D];
    __shared__ __attribute__((aligned(16))) float sb[D];
    const int bh = blockIdx.y, h = bh % H, tid = threadIdx.x;
    stage_filters<D>(sw, W, h, K * K);
    if (tid < D) sb[tid] = bias ? bias[h * D + tid] : 0.f;
    __syncthreads();
    const long long items = (long long)n * NG, stride = (long long)gridDim.x * 256;
    for (long long gid = (long long)blockIdx.x * 256 + tid; gid < items; gid += stride) {
        const int i = (int)(gid / NG), c0 = (int)(gid % NG) * 4;
        const int gh = n / gw, y = i / gw, x = i % gw;
        const size_t base = (size_t)bh * n * D + c0;
        float4 acc = *reinterpret_cast<const float4*>(sb + c0);
        auto row = [&](int u) {   // one filter row: its K loads in flight together
            float4 v[K];
            bool in[K];
#pragma unroll
            for (int t = 0; t < K; ++t) {
                const Nbr q = nbr(y, x, u - P, t - P, gh, gw);
                in[t] = q.in;
                v[t] = load4<DT>(V, base + (size_t)q.j * D);
            }
#pragma unroll
            for (int t = 0; t < K; ++t) {
                float4 wv = *reinterpret_cast<const float4*>(sw + (u * K + t) * D + c0);
                if (!in[t]) wv = make_float4(0.f, 0.f, 0.f, 0.f);
                fma4(acc, wv, v[t]);
            }
        };
        if constexpr (K <= 3) {   // every tap's load in flight at once
#pragma unroll
            for (int u = 0; u < K; ++u) row(u);
        } else {                  // wide filters: a row at a time, to keep the registers for more waves
#pragma unroll 1
            for (int u = 0; u < K; ++u) row(u);
        }
        *reinterpret_cast<float4*>(E + base + (size_t)i * D) = acc;
    }
}

// dV_j += sum over taps of w[u][t] dOut_{j - (u - p, t - p)}; same grid as the forward.
template <int D, int K>
__global__ __launch_bounds__(256) void dwc_bwd_dv_kernel(const float* __restrict__ G, const float* __restrict__ W,
                                                         float* __restrict__ dV, int n, int H, int gw) {
    constexpr int NG = D / 4, P = (K - 1) / 2;
    __shared__ __attribute__((aligned(16))) float sw[K * K * D];
    const int bh = blockIdx.y, h = bh % H, tid = threadIdx.x;
    stage_filters<D>(sw, W, h, K * K);
    __syncthreads();
    const long long items = (long long)n * NG, stride = (long long)gridDim.x * 256;
    for (long long gid = (long long)blockIdx.x * 256 + tid; gid < items; gid += stride) {
        const int j = (int)(gid / NG), c0 = (int)(gid % NG) * 4;
        const int gh = n / gw, y = j / gw, x = j % gw;
        const size_t base = (size_t)bh * n * D + c0;
        float4* o = reinterpret_cast<float4*>(dV + base + (size_t)j * D);
        float4 acc = *o;
        auto row = [&](int u) {
            float4 g[K];
            bool in[K];
#pragma unroll
            for (int t = 0; t < K; ++t) {
                const Nbr q = nbr(y, x, P - u, P - t, gh, gw);
                in[t] = q.in;
                g[t] = *reinterpret_cast<const float4*>(G + base + (size_t)q.j * D);
            }
#pragma unroll
            for (int t = 0; t < K; ++t) {
                float4 wv = *reinterpret_cast<const float4*>(sw + (u * K + t) * D + c0);
                if (!in[t]) wv = make_float4(0.f, 0.f, 0.f, 0.f);
                fma4(acc, wv, g[t]);
            }
        };
        if constexpr (K <= 3) {
#pragma unroll
            for (int u = 0; u < K; ++u) row(u);
        } else {
#pragma unroll 1
            for (int u = 0; u < K; ++u) row(u);
        }
        *o = acc;
    }
}

// Filter and bias gradients of one token chunk.  grid (nch, B*H), 256 threads: thread
// (token lane tl, channel group cg) takes tokens i0 + tl, i0 + tl + TL, ... of chunk
// [i0, min(n, i0 + chunk)).  Taps k*k+1 (the last is the bias) go in passes of up to TB, each
// thread keeping TB float4 sums; the sums are added over the token lanes of a wave by xor
// shuffles, then over the four waves through LDS, both in a fixed order.
// part[h][c][tap][b * nch + ch]: the terms of one sum are contiguous for the reduction.
template <int D, int K>
__global__ __launch_bounds__(256) void dwc_bwd_w_kernel(const float* __restrict__ G, const float* __restrict__ V,
                                                        float* __restrict__ part, int n, int H, int gw, int chunk,
                                                        int nch, int BN) {
    constexpr int NG = D / 4, TL = 256 / NG, P = (K - 1) / 2;
    constexpr int NTAP = K * K + 1, TB = NTAP < 10 ? NTAP : 10, NPASS = (NTAP + TB - 1) / TB;
    __shared__ __attribute__((aligned(16))) float4 red[4 * NG * TB];
    const int bh = blockIdx.y, ch = blockIdx.x, tid = threadIdx.x, cg = tid % NG, tl = tid / NG;
    const int w = tid >> 6, lane = tid & 63;
    const int i0 = ch * chunk, i1 = min(n, i0 + chunk), gh = n / gw;
    const size_t base = (size_t)bh * n * D + 4 * cg;
    float* dst = part + (size_t)(bh % H) * D * NTAP * BN + (size_t)(bh / H) * nch + ch;
#pragma unroll 1
    for (int pass = 0; pass < NPASS; ++pass) {
        float4 acc[TB];
#pragma unroll
        for (int b = 0; b < TB; ++b) acc[b] = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll 2
        for (int i = i0 + tl; i < i1; i += TL) {
            const int y = i / gw, x = i % gw;
            const float4 gi = *reinterpret_cast<const float4*>(G + base + (size_t)i * D);
            float4 vv[TB];
            bool in[TB];
#pragma unroll
            for (int b = 0; b < TB; ++b) {
                const int tap = pass * TB + b;   // K*K: the bias; past NTAP: unused
                const int tt = tap < K * K ? tap : P * K + P;
                const Nbr q = nbr(y, x, tt / K - P, tt % K - P, gh, gw);
                in[b] = q.in && tap < K * K;
                vv[b] = *reinterpret_cast<const float4*>(V + base + (size_t)q.j * D);
                if (tap == K * K) {
                    in[b] = true;
                    vv[b] = make_float4(1.f, 1.f, 1.f, 1.f);
                }
            }
#pragma unroll
            for (int b = 0; b < TB; ++b) {
                float4 v = vv[b];
                if (!in[b]) v = make_float4(0.f, 0.f, 0.f, 0.f);
                fma4(acc[b], gi, v);
            }
        }
        // lanes cg, cg + NG, ... of a wave share a channel group
#pragma unroll
        for (int off = NG; off < 64; off <<= 1)
#pragma unroll
            for (int b = 0; b < TB; ++b) {
                acc[b].x += __shfl_xor(acc[b].x, off, 64);
                acc[b].y += __shfl_xor(acc[b].y, off, 64);
                acc[b].z += __shfl_xor(acc[b].z, off, 64);
                acc[b].w += __shfl_xor(acc[b].w, off, 64);
            }
        if (lane < NG) {
#pragma unroll
            for (int b = 0; b < TB; ++b) red[(w * NG + lane) * TB + b] = acc[b];
        }
        __syncthreads();
        for (int job = tid; job < NG * TB; job += 256) {
            const int jc = job % NG, b = job / NG, tap = pass * TB + b;
            const float4 r0 = red[(0 * NG + jc) * TB + b], r1 = red[(1 * NG + jc) * TB + b],
                         r2 = red[(2 * NG + jc) * TB + b], r3 = red[(3 * NG + jc) * TB + b];
            if (tap < NTAP) {
                dst[(size_t)((4 * jc + 0) * NTAP + tap) * BN] = ((r0.x + r1.x) + r2.x) + r3.x;
                dst[(size_t)((4 * jc + 1) * NTAP + tap) * BN] = ((r0.y + r1.y) + r2.y) + r3.y;
                dst[(size_t)((4 * jc + 2) * NTAP + tap) * BN] = ((r0.z + r1.z) + r2.z) + r3.z;
                dst[(size_t)((4 * jc + 3) * NTAP + tap) * BN] = ((r0.w + r1.w) + r2.w) + r3.w;
            }
        }
        __syncthreads();   // red is rewritten by the next pass
    }
}

// One wave per sum (h, c, tap), four per block: lane t adds terms t, t + 64, ... of the BN
// contiguous partials in fp64, then the lanes are combined by xor shuffles (a fixed order).
__global__ __launch_bounds__(256) void dwc_bwd_w_reduce(const float* __restrict__ part, float* __restrict__ dW,
                                                        float* __restrict__ db, int H, int d, int k, int BN) {
    const int kk = k * k, ntap = kk + 1;
    const int e = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
    if (e >= H * d * ntap) return;   // whole waves leave together
    const float* src = part + (size_t)e * BN;
    double s = 0.0;
    for (int t = lane; t < BN; t += 64) s += src[t];
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) s += __shfl_xor(s, off, 64);
    if (lane) return;
    const int h = e / (d * ntap), c = (e / ntap) % d, tap = e % ntap;
    if (tap < kk) {
        if (dW) dW[((size_t)h * d + c) * kk + tap] = (float)s;
    } else if (db) {
        db[h * d + c] = (float)s;
    }
}

// ------------------------------------------------------------------------------------------
// Launch wrappers.

constexpr int kDwcItemsPerThread = 4;
static dim3 dwc_grid(int BH, int n, int d) {
    return dim3((unsigned)(((long long)n * (d / 4) + 256 * kDwcItemsPerThread - 1) / (256 * kDwcItemsPerThread)), BH);
}
static bool dwc_ok(int k, int n, int gw) { return (k == 1 || k == 3 || k == 5 || k == kDwcMaxK) && gw >= 1 && n % gw == 0; }

template <int DT, int D>
static void dwc_fwd_k(const void* V, const float* W, const float* bias, float* E, int BH, int H, int n, int gw, int k,
                      hipStream_t st) {
    const auto* v = static_cast<const typename elem<DT>::type*>(V);
    const dim3 grid = dwc_grid(BH, n, D);
    if (k == 1) hipLaunchKernelGGL((dwc_fwd_kernel<DT, D, 1>), grid, dim3(256), 0, st, v, W, bias, E, n, H, gw);
    else if (k == 3) hipLaunchKernelGGL((dwc_fwd_kernel<DT, D, 3>), grid, dim3(256), 0, st, v, W, bias, E, n, H, gw);
    else if (k == 5) hipLaunchKernelGGL((dwc_fwd_kernel<DT, D, 5>), grid, dim3(256), 0, st, v, W, bias, E, n, H, gw);
    else hipLaunchKernelGGL((dwc_fwd_kernel<DT, D, 7>), grid, dim3(256), 0, st, v, W, bias, E, n, H, gw);
}

hipError_t launch_dwc_fwd(int dt, const void* V, const float* W, const float* bias, float* E, int BH, int H, int n,
                          int d, int gw, int k, hipStream_t st) {
    if (!dwc_ok(k, n, gw)) return hipErrorInvalidValue;
    if (dt == DT_F32 && d == 32) dwc_fwd_k<DT_F32, 32>(V, W, bias, E, BH, H, n, gw, k, st);
    else if (dt == DT_F32) dwc_fwd_k<DT_F32, 64>(V, W, bias, E, BH, H, n, gw, k, st);
    else if (d == 32) dwc_fwd_k<DT_BF16, 32>(V, W, bias, E, BH, H, n, gw, k, st);
    else dwc_fwd_k<DT_BF16, 64>(V, W, bias, E, BH, H, n, gw, k, st);
    return hipGetLastError();
}

template <int D>
static void dwc_dv_k(const float* G, const float* W, float* dV, int BH, int H, int n, int gw, int k, hipStream_t st) {
    const dim3 grid = dwc_grid(BH, n, D);
    if (k == 1) hipLaunchKernelGGL((dwc_bwd_dv_kernel<D, 1>), grid, dim3(256), 0, st, G, W, dV, n, H, gw);
    else if (k == 3) hipLaunchKernelGGL((dwc_bwd_dv_kernel<D, 3>), grid, dim3(256), 0, st, G, W, dV, n, H, gw);
    else if (k == 5) hipLaunchKernelGGL((dwc_bwd_dv_kernel<D, 5>), grid, dim3(256), 0, st, G, W, dV, n, H, gw);
    else hipLaunchKernelGGL((dwc_bwd_dv_kernel<D, 7>), grid, dim3(256), 0, st, G, W, dV, n, H, gw);
}

hipError_t launch_dwc_bwd_dv(const float* G, const float* W, float* dV, int BH, int H, int n, int d, int gw, int k,
                             hipStream_t st) {
    if (!dwc_ok(k, n, gw)) return hipErrorInvalidValue;
    if (d == 32) dwc_dv_k<32>(G, W, dV, BH, H, n, gw, k, st);
    else dwc_dv_k<64>(G, W, dV, BH, H, n, gw, k, st);
    return hipGetLastError();
}

template <int D>
static void dwc_w_k(const float* G, const float* V, float* part, int BH, int H, int n, int gw, int k, int chunk,
                    int nch, int BN, hipStream_t st) {
    const dim3 grid(nch, BH);
#define LAPATTN_DWCW(Kv) \
    hipLaunchKernelGGL((dwc_bwd_w_kernel<D, Kv>), grid, dim3(256), 0, st, G, V, part, n, H, gw, chunk, nch, BN)
    if (k == 1) LAPATTN_DWCW(1);
    else if (k == 3) LAPATTN_DWCW(3);
    else if (k == 5) LAPATTN_DWCW(5);
    else LAPATTN_DWCW(7);
#undef LAPATTN_DWCW
}

hipError_t launch_dwc_bwd_w(const float* G, const float* V, float* part, float* dW, float* db, int B, int H, int n,
                            int d, int gw, int k, int chunk, hipStream_t st) {
    if (!dwc_ok(k, n, gw) || chunk < 1) return hipErrorInvalidValue;
    const int nch = (n + chunk - 1) / chunk, BN = B * nch;
    if (d == 32) dwc_w_k<32>(G, V, part, B * H, H, n, gw, k, chunk, nch, BN, st);
    else dwc_w_k<64>(G, V, part, B * H, H, n, gw, k, chunk, nch, BN, st);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int sums = H * d * (k * k + 1);
    hipLaunchKernelGGL(dwc_bwd_w_reduce, dim3((sums + 3) / 4), dim3(256), 0, st, part, dW, db, H, d, k, BN);
    return hipGetLastError();
}

}  // namespace lapattn
