// fast.hip -- the bf16 forward path: fixed-point L1 distances on the VALU (v_sad_u16),
// contractions on the matrix cores (fp16 MFMA), Newton-Schulz on fp32 MFMA.
//
//   pool2_kernel     landmark means (Sec. 4.2, sampling; 1-D segments) and per-segment
//                    value sums / magnitudes, 16-byte vector loads
//   frame_kernel     per head: the fixed-point frame of the L1 distances, the landmark
//                    tables in that frame, the value mean and the value prescale
//   nskey_kernel     one launch, two roles: blocks [0, BH) run Algorithm 2 on K_LL with
//                    fp32 MFMA; the other blocks form U = K_LK [V | 1] over key chunks
//                    (Sec. 3.2 key summaries) with v_sad_u16 distances and fp16 MFMA
//   mfinal_kernel    U = sum of the chunk partials, M = X_T U, split into fp16 hi/lo
//                    MFMA operand tiles with a power-of-two scale per column
//   query2_kernel    Y = K_QL M (Eq. (8)) and the normalisation (Eq. (4) / Eq. (3))
//
// Distances.  Per head, with R = max(|Q|, |K|) over the head and S = 65535 / (2R), every
// coordinate x becomes u(x) = rint((x + R) S) in [0, 65535] (v_cvt_pknorm_u16_f32 of
// (x + R) / (2R), two coordinates per instruction).  Then
// sum_c |u(x_c) - u(y_c)| = S ||x - y||_1 + e with |e| <= d (each rounding moves a
// coordinate by at most 1/2 a step), so the distance error is at most d / S = 2 R d / 65535.
// v_sad_u16 adds |a.lo - b.lo| + |a.hi - b.hi| to an accumulator: two coordinates per lane
// and instruction, exact integer arithmetic.  The accumulator starts at the bit pattern of
// 2^23, so after the sum it reads as the float 2^23 + D (D < 2^23 for d <= 64), and one fma
// maps it to the exp2 argument -D log2(e) / (lambda S).
#include "common.hpp"
#include "kernels.hpp"

namespace lapattn {

typedef _Float16 h8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

constexpr int kLP = 72;            // LDS row pitch (halves) of the 64 x 64 fp16 tiles
constexpr float kTwo23 = 8388608.f;

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

typedef unsigned short u16x2_t __attribute__((ext_vector_type(2)));
typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));

// Two coordinates to the fixed-point frame: u = rint(clamp((x + R) / (2R)) * 65535), packed.
__device__ __forceinline__ uint32_t fix2(float x0, float x1, float inv2R) {
    const u16x2_t u = __builtin_amdgcn_cvt_pknorm_u16(fmaf(x0, inv2R, 0.5f), fmaf(x1, inv2R, 0.5f));
    return __builtin_bit_cast(uint32_t, u);
}
// A packed bf16 pair (one dword) to the fixed-point frame.
__device__ __forceinline__ uint32_t fix2_bf16(uint32_t w, float inv2R) {
    return fix2(bf16_lo(w), bf16_hi(w), inv2R);
}
__device__ __forceinline__ uint32_t pk_f16(float a, float b) {
    const f16x2_t h = {(_Float16)a, (_Float16)b};
    return __builtin_bit_cast(uint32_t, h);
}

// ------------------------------------------------------------------------------------------
// Landmark means and per-segment statistics.  grid (m, BH), 256 threads.  Thread t always
// reads the 8-column group t % (D/8) of its rows; partial sums are combined in a fixed order.
template <int D>
__global__ __launch_bounds__(256) void pool2_kernel(const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
                                                    const uint16_t* __restrict__ V, float* __restrict__ qt,
                                                    float* __restrict__ kt, double* __restrict__ vseg,
                                                    float* __restrict__ segmax, float* __restrict__ vsegmax, int n,
                                                    int m) {
    constexpr int CPR = D / 8;      // 16-byte chunks per row
    constexpr int RPI = 256 / CPR;  // rows per block iteration
    const int l = blockIdx.x, h = blockIdx.y, tid = threadIdx.x;
    const int s0 = seg_start(l, n, m), s1 = seg_start(l + 1, n, m);
    const int cg = tid % CPR, r0 = tid / CPR;
    float sq[8], sk[8], sv[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) sq[j] = sk[j] = sv[j] = 0.f;
    float mx = 0.f, vmx = 0.f;
    const size_t base = (size_t)h * n * D + cg * 8;
#pragma unroll 4
    for (int i = s0 + r0; i < s1; i += RPI) {
        const size_t off = base + (size_t)i * D;
        const uint4 a = *reinterpret_cast<const uint4*>(Q + off);
        const uint4 b = *reinterpret_cast<const uint4*>(K + off);
        const uint4 c = *reinterpret_cast<const uint4*>(V + off);
        const uint32_t aw[4] = {a.x, a.y, a.z, a.w}, bw[4] = {b.x, b.y, b.z, b.w}, cw[4] = {c.x, c.y, c.z, c.w};
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const float q0 = bf16_lo(aw[j]), q1 = bf16_hi(aw[j]);
            const float k0 = bf16_lo(bw[j]), k1 = bf16_hi(bw[j]);
            const float v0 = bf16_lo(cw[j]), v1 = bf16_hi(cw[j]);
            sq[2 * j] += q0; sq[2 * j + 1] += q1;
            sk[2 * j] += k0; sk[2 * j + 1] += k1;
            sv[2 * j] += v0; sv[2 * j + 1] += v1;
            mx = fmaxf(fmaxf(mx, fabsf(q0)), fmaxf(fabsf(q1), fmaxf(fabsf(k0), fabsf(k1))));
            vmx = fmaxf(vmx, fmaxf(fabsf(v0), fabsf(v1)));
        }
    }
    // A non-finite input makes its column sum non-finite (fmaxf alone would hide a NaN).
    __shared__ double red[256 * 8];
    __shared__ float smx[256], svmx[256];
    __shared__ int sbad[64];
    const double cnt = (double)(s1 - s0);
    for (int pass = 0; pass < 3; ++pass) {
        const float* src = pass == 0 ? sq : (pass == 1 ? sk : sv);
#pragma unroll
        for (int j = 0; j < 8; ++j) red[tid * 8 + j] = (double)src[j];
        if (pass == 0) {
            smx[tid] = mx;
            svmx[tid] = vmx;
        }
        __syncthreads();
        if (tid < D) {
            const int g = tid / 8, j = tid % 8;
            double t = 0.0;
            for (int r = 0; r < RPI; ++r) t += red[(g + CPR * r) * 8 + j];
            const size_t o = ((size_t)h * m + l) * D + tid;
            if (pass == 0) qt[o] = (float)(t / cnt);
            else if (pass == 1) kt[o] = (float)(t / cnt);
            else vseg[o] = t;
            sbad[tid] = (pass == 0 ? 0 : sbad[tid]) | (isfinite(t) ? 0 : 1);
        }
        __syncthreads();
    }
    if (tid == 0) {
        float a = 0.f, b = 0.f;
        int anybad = 0;
        for (int r = 0; r < 256; ++r) {
            a = fmaxf(a, smx[r]);
            b = fmaxf(b, svmx[r]);
        }
        for (int c = 0; c < D; ++c) anybad |= sbad[c];
        segmax[(size_t)h * m + l] = anybad ? __builtin_nanf("") : a;
        vsegmax[(size_t)h * m + l] = anybad ? __builtin_nanf("") : b;
    }
}

// ------------------------------------------------------------------------------------------
// Per-head frame.  grid (BH), 256 threads.
//   frame[h] = {R, 1/(2R), escale = -log2(e) / (lambda S), vscale}; R is NaN when Q, K or V hold a
//   non-finite value (the outputs of that head are then NaN, as the plain computation gives).
//   qfix/kfix[h][a][c/2] = u(x_{a,c}) | u(x_{a,c+1}) << 16 for landmarks a < 64 (zero rows >= m).
//   vbar[h] = mean of the values; vscale = 2^-e keeps the fp16 copies of V below 2^14.
template <int D>
__global__ __launch_bounds__(256) void frame_kernel(const float* __restrict__ qt, const float* __restrict__ kt,
                                                    const double* __restrict__ vseg,
                                                    const float* __restrict__ segmax,
                                                    const float* __restrict__ vsegmax, float* __restrict__ frame,
                                                    uint32_t* __restrict__ qfix, uint32_t* __restrict__ kfix,
                                                    float* __restrict__ vbar, int n, int m, float lambda) {
    const int h = blockIdx.x, tid = threadIdx.x;
    __shared__ float sR, sS, smx[64], svm[64];   // sS: 1 / (2R)
    __shared__ int sbad[64];
    if (tid < 64) {
        float a = 0.f, b = 0.f;
        if (tid < m) {
            a = segmax[(size_t)h * m + tid];
            b = vsegmax[(size_t)h * m + tid];
        }
        sbad[tid] = (isfinite(a) && isfinite(b)) ? 0 : 1;
        smx[tid] = a;
        svm[tid] = b;
    }
    __syncthreads();
    if (tid == 0) {
        float R = 0.f, vm = 0.f;
        int bad = 0;
        for (int l = 0; l < 64; ++l) {
            bad |= sbad[l];
            R = fmaxf(R, smx[l]);
            vm = fmaxf(vm, svm[l]);
        }
        if (R == 0.f) R = 1.f;
        const float S = (float)(65535.0 / (2.0 * (double)R));
        float vscale = 1.f;
        if (vm > 16384.f) vscale = exp2f(-ceilf(log2f(vm / 16384.f)));
        if (bad) R = __builtin_nanf("");
        sR = R;
        sS = (float)(0.5 / (double)R);
        frame[h * 4 + 0] = R;
        frame[h * 4 + 1] = sS;
        frame[h * 4 + 2] = (float)(-1.4426950408889634 / ((double)lambda * (double)S));
        frame[h * 4 + 3] = vscale;
    }
    __syncthreads();
    const float inv2R = sS;
    for (int e = tid; e < 64 * (D / 2); e += 256) {
        const int a = e / (D / 2), c2 = e % (D / 2);
        uint32_t wq = 0, wk = 0;
        if (a < m) {
            const float* q = qt + ((size_t)h * m + a) * D + 2 * c2;
            const float* k = kt + ((size_t)h * m + a) * D + 2 * c2;
            wq = fix2(q[0], q[1], inv2R);
            wk = fix2(k[0], k[1], inv2R);
        }
        qfix[(size_t)h * 64 * (D / 2) + e] = wq;
        kfix[(size_t)h * 64 * (D / 2) + e] = wk;
    }
    for (int c = tid; c < D; c += 256) {
        double s = 0.0;
#pragma unroll 16
        for (int l = 0; l < m; ++l) s += vseg[((size_t)h * m + l) * D + c];
        vbar[(size_t)h * D + c] = (float)(s / n);
    }
}

// ------------------------------------------------------------------------------------------
// fp32 64 x 64 product on the matrix cores for one wave: the 32 x 32 block (rb, cb) of A B,
// A and B in LDS with row pitch 65.  v_mfma_f32_32x32x2_f32: lane l supplies A[32rb + l%32][2s + l/32]
// and B[2s + l/32][32cb + l%32]; result register r holds row 32rb + 8(r/4) + 4(l/32) + r%4,
// column 32cb + l%32.
__device__ __forceinline__ f32x16_t mm64_f32(const float* __restrict__ A, const float* __restrict__ B, int rb,
                                             int cb) {
    const int l = threadIdx.x & 63;
    f32x16_t acc = {};
    const float* a = A + (32 * rb + (l & 31)) * 65 + (l >> 5);
    const float* b = B + (l >> 5) * 65 + 32 * cb + (l & 31);
#pragma unroll 8
    for (int s = 0; s < 32; ++s) acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a[2 * s], b[2 * s * 65], acc, 0, 0, 0);
    return acc;
}

__device__ __forceinline__ int c_row(int r, int l) { return 8 * (r >> 2) + 4 * (l >> 5) + (r & 3); }

// ------------------------------------------------------------------------------------------
// Newton-Schulz role (one block per head, 4 waves): W = K_LL + eps I padded to 64 x 64,
// c = ||W||_1 ||W||_inf (first maximising column / row), X0 = W^T / c (0 if c = 0),
// X_{t+1} = X_t (2I - W X_t).  Writes X_T (fp32, [64][64]) and cinfo = {c, n1, ninf, code}.
__device__ void ns_role(int h, float* lds, const float* __restrict__ qt, const float* __restrict__ kt, int m, int D,
                        int T, float kscale, float eps, float* __restrict__ XT, float* __restrict__ cinfo) {
    float* sW = lds;
    float* sX0 = lds + 64 * 65;
    float* sX1 = lds + 2 * 64 * 65;
    float* sT = lds + 3 * 64 * 65;
    float* sred = lds + 4 * 64 * 65;   // 130 floats
    const int tid = threadIdx.x, w = tid >> 6, l = tid & 63;
    // landmarks staged in the X1 / T regions (m x D <= 64 x 64 floats each)
    float* q = sX1;
    float* k = sT;
    for (int e = tid; e < m * D; e += 256) {
        q[e] = qt[(size_t)h * m * D + e];
        k[e] = kt[(size_t)h * m * D + e];
    }
    __syncthreads();
    for (int e = tid; e < 64 * 64; e += 256) {
        const int a = e >> 6, b = e & 63;
        float v = 0.f;
        if (a < m && b < m) {
            float dist = 0.f;
            for (int c = 0; c < D; ++c) dist += fabsf(q[a * D + c] - k[b * D + c]);
            v = exp2f(dist * kscale);
            if (a == b) v += eps;
        }
        sW[a * 65 + b] = v;
    }
    __syncthreads();
    if (tid < 128) {
        const int i = tid & 63;
        float s = 0.f;
        if (tid < 64)
            for (int a = 0; a < 64; ++a) s += fabsf(sW[a * 65 + i]);   // column sums
        else
            for (int b = 0; b < 64; ++b) s += fabsf(sW[i * 65 + b]);   // row sums
        sred[tid] = s;
    }
    __syncthreads();
    if (tid == 0) {
        float n1 = -1.f, ninf = -1.f;
        int bs = 0, as = 0;
        for (int b = 0; b < 64; ++b)
            if (sred[b] > n1) { n1 = sred[b]; bs = b; }
        for (int a = 0; a < 64; ++a)
            if (sred[64 + a] > ninf) { ninf = sred[64 + a]; as = a; }
        const float c = n1 * ninf;
        sred[128] = c;
        cinfo[h * 4 + 0] = c;
        cinfo[h * 4 + 1] = n1;
        cinfo[h * 4 + 2] = ninf;
        cinfo[h * 4 + 3] = (float)(as * 256 + bs);
    }
    __syncthreads();
    const float c = sred[128];
    const float inv_c = c > 0.f ? 1.f / c : 0.f;
    for (int e = tid; e < 64 * 64; e += 256) {
        const int a = e >> 6, b = e & 63;
        sX0[a * 65 + b] = sW[b * 65 + a] * inv_c;
    }
    __syncthreads();
    const int rb = w >> 1, cb = w & 1;
    float* Xc = sX0;
    float* Xn = sX1;
    for (int t = 0; t < T; ++t) {
        f32x16_t p = mm64_f32(sW, Xc, rb, cb);          // W X
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int row = 32 * rb + c_row(r, l), col = 32 * cb + (l & 31);
            sT[row * 65 + col] = (row == col ? 2.f : 0.f) - p[r];
        }
        __syncthreads();
        p = mm64_f32(Xc, sT, rb, cb);                     // X (2I - W X)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int row = 32 * rb + c_row(r, l), col = 32 * cb + (l & 31);
            Xn[row * 65 + col] = p[r];
        }
        __syncthreads();
        float* tmp = Xc;
        Xc = Xn;
        Xn = tmp;
    }
    for (int e = tid; e < 64 * 64; e += 256) XT[(size_t)h * 4096 + e] = Xc[(e >> 6) * 65 + (e & 63)];
}

// ------------------------------------------------------------------------------------------
// Key-summary role: block kb of head h covers keys [kb*kpb, min(n, (kb+1)*kpb)); each wave
// takes 64-key tiles (lane = key) on its own, with its own LDS region (no block barrier in the
// loop).  Per tile: u(k_j) in registers, the value row to fp16 in LDS transposed ([c][j]), the
// m kernel values exp(-||qt_a - k_j||_1/lambda) from v_sad_u16 against the landmark table
// (wave-uniform, scalar loads) into LDS as [a][j], then U[a][c] += sum_j B[a][j] V[j][c] (and
// the ones column) on fp16 MFMA 32x32x16.  The raw rows of the next tile are loaded while the
// current one is computed.
__device__ __forceinline__ void wave_lds_sync() {
    // LDS requests of one wave complete in order; this only keeps the compiler from moving
    // the reads of other lanes' writes above the writes.
    __builtin_amdgcn_s_waitcnt(0xc07f);
    __builtin_amdgcn_wave_barrier();
}

template <int D>
__device__ void key_role(int h, int kb, char* lds_raw, const uint16_t* __restrict__ K,
                         const uint16_t* __restrict__ V, const uint32_t* __restrict__ qfix,
                         const float* __restrict__ frame, float* __restrict__ Upart, int n, int m, int kpb, int nkb) {
    constexpr int D2 = D / 2;
    constexpr int D8 = D / 8;
    constexpr int CB = D / 32;
    const int tid = threadIdx.x, w = tid >> 6, l = tid & 63;
    _Float16* sB = reinterpret_cast<_Float16*>(lds_raw) + w * (2 * 64 * kLP);
    _Float16* sV = sB + 64 * kLP;
    const float inv2R = frame[h * 4 + 1], esc = frame[h * 4 + 2], vsc = frame[h * 4 + 3];
    const float ebias = -kTwo23 * esc;
    const uint32_t* tab = qfix + (size_t)h * 64 * D2;
    const int j_begin = kb * kpb, j_end = min(n, j_begin + kpb);
    const int ntiles = (j_end - j_begin + 63) / 64;
    const int RB = m > 32 ? 2 : 1;
    f32x16_t acc[2][CB + 1];
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
        for (int cb = 0; cb <= CB; ++cb) acc[rb][cb] = (f32x16_t){};
    h8_t ones;
#pragma unroll
    for (int i = 0; i < 8; ++i) ones[i] = (l & 31) == 0 ? (_Float16)1.f : (_Float16)0.f;
    for (int a = m; a < 64; ++a) sB[a * kLP + l] = (_Float16)0.f;   // rows a >= m stay zero

    uint4 kr[D8], vr[D8];
    auto load_rows = [&](int tile) {
        const int j = j_begin + tile * 64 + l;
        if (tile < ntiles && j < j_end) {
            const uint4* kp = reinterpret_cast<const uint4*>(K + ((size_t)h * n + j) * D);
            const uint4* vp = reinterpret_cast<const uint4*>(V + ((size_t)h * n + j) * D);
#pragma unroll
            for (int c8 = 0; c8 < D8; ++c8) {
                kr[c8] = kp[c8];
                vr[c8] = vp[c8];
            }
        }
    };
    load_rows(w);
    for (int tile = w; tile < ntiles; tile += 4) {
        const int j = j_begin + tile * 64 + l;
        const bool valid = j < j_end;
        uint32_t kf[D2];
        if (valid) {
#pragma unroll
            for (int c8 = 0; c8 < D8; ++c8) {
                const uint32_t xw[4] = {kr[c8].x, kr[c8].y, kr[c8].z, kr[c8].w};
                const uint32_t yw[4] = {vr[c8].x, vr[c8].y, vr[c8].z, vr[c8].w};
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    kf[4 * c8 + t] = fix2_bf16(xw[t], inv2R);
                    sV[(8 * c8 + 2 * t) * kLP + l] = (_Float16)(bf16_lo(yw[t]) * vsc);
                    sV[(8 * c8 + 2 * t + 1) * kLP + l] = (_Float16)(bf16_hi(yw[t]) * vsc);
                }
            }
        } else {
#pragma unroll
            for (int c = 0; c < D2; ++c) kf[c] = 0u;
#pragma unroll
            for (int c = 0; c < D; ++c) sV[c * kLP + l] = (_Float16)0.f;
        }
        load_rows(tile + 4);
        for (int a = 0; a < m; ++a) {
            const uint32_t* ta = tab + a * D2;
            uint32_t acc_u = 0x4B000000u;
#pragma unroll
            for (int c = 0; c < D2; ++c) acc_u = __builtin_amdgcn_sad_u16(kf[c], ta[c], acc_u);
            const float b = __builtin_amdgcn_exp2f(fmaf(__uint_as_float(acc_u), esc, ebias));
            sB[a * kLP + l] = valid ? (_Float16)b : (_Float16)0.f;
        }
        wave_lds_sync();
#pragma unroll
        for (int s4 = 0; s4 < 4; ++s4) {
#pragma unroll
            for (int rb = 0; rb < 2; ++rb) {
                if (rb < RB) {
                    const h8_t A =
                        *reinterpret_cast<const h8_t*>(sB + (32 * rb + (l & 31)) * kLP + 16 * s4 + 8 * (l >> 5));
#pragma unroll
                    for (int cb = 0; cb < CB; ++cb) {
                        const h8_t Bv =
                            *reinterpret_cast<const h8_t*>(sV + (32 * cb + (l & 31)) * kLP + 16 * s4 + 8 * (l >> 5));
                        acc[rb][cb] = __builtin_amdgcn_mfma_f32_32x32x16_f16(A, Bv, acc[rb][cb], 0, 0, 0);
                    }
                    acc[rb][CB] = __builtin_amdgcn_mfma_f32_32x32x16_f16(A, ones, acc[rb][CB], 0, 0, 0);
                }
            }
        }
        wave_lds_sync();
    }
    __syncthreads();
    // per-wave partials to LDS as [a][c] (64 x (D+1) floats), then a fixed-order block sum;
    // the value columns were formed from V * vscale
    const float inv_vsc = 1.f / vsc;
    float* sP = reinterpret_cast<float*>(lds_raw) + w * (64 * (D + 1));
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
        for (int cb = 0; cb <= CB; ++cb)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int a = 32 * rb + c_row(r, l);
                const int c = cb < CB ? 32 * cb + (l & 31) : D;
                if (cb < CB || (l & 31) == 0) sP[a * (D + 1) + c] = acc[rb][cb][r] * (cb < CB ? inv_vsc : 1.f);
            }
    __syncthreads();
    const float* base = reinterpret_cast<const float*>(lds_raw);
    for (int e = tid; e < m * (D + 1); e += 256) {
        float t = 0.f;
#pragma unroll
        for (int ww = 0; ww < 4; ++ww) t += base[ww * 64 * (D + 1) + e];
        Upart[((size_t)h * nkb + kb) * m * (D + 1) + e] = t;
    }
}

// ------------------------------------------------------------------------------------------
// One launch for both independent halves of the middle of the forward: blocks [0, BH) solve
// Newton-Schulz (they only need the landmarks), blocks [BH, BH + BH*nkb) form the key-side
// partial sums.  The solver blocks come first so they start at once.
constexpr int kNsLds = (4 * 64 * 65 + 132) * 4;
constexpr int kKeyLds = 4 * 2 * 64 * kLP * 2;
constexpr int kNsKeyLds = kNsLds > kKeyLds ? kNsLds : kKeyLds;

template <int D>
__global__ __launch_bounds__(256) void nskey_kernel(const float* __restrict__ qt, const float* __restrict__ kt,
                                                    float* __restrict__ XT, float* __restrict__ cinfo,
                                                    const uint16_t* __restrict__ K, const uint16_t* __restrict__ V,
                                                    const uint32_t* __restrict__ qfix, const float* __restrict__ frame,
                                                    float* __restrict__ Upart, int BH, int n, int m, int T,
                                                    float kscale, float eps, int kpb, int nkb) {
    __shared__ __attribute__((aligned(16))) char lds[kNsKeyLds];
    const int b = blockIdx.x;
    if (b < BH) {
        ns_role(b, reinterpret_cast<float*>(lds), qt, kt, m, D, T, kscale, eps, XT, cinfo);
    } else {
        const int kbb = b - BH;
        key_role<D>(kbb / nkb, kbb % nkb, lds, K, V, qfix, frame, Upart, n, m, kpb, nkb);
    }
}

// ------------------------------------------------------------------------------------------
// U = sum over key chunks, M = X_T U, and the MFMA operand tiles of M for the query side.
// grid (BH), 1024 threads.  Tiles: Mt[h][s][cb][part][lane][i] = part of
// M[16s + 8(lane/32) + i][column of (cb, lane%32)] * 2^-e, part 0 = fp16 value, part 1 = fp16
// residual; column (cb, j) is 32cb + j for cb < D/32 and, for cb = D/32, the ones column d
// when j = 0 (else zero).  One power-of-two scale for the value columns and one for the ones
// column (mscale[h][0], mscale[h][1] = 2^e): the largest magnitude lands in [2^14, 2^15).
template <int D>
__global__ __launch_bounds__(1024) void mfinal_kernel(const float* __restrict__ Upart, const float* __restrict__ XT,
                                                      _Float16* __restrict__ Mt, float* __restrict__ mscale,
                                                      float* __restrict__ U, float* __restrict__ Mout, int m,
                                                      int nkb) {
    constexpr int D1 = D + 1;
    constexpr int CB = D / 32;
    __shared__ float sU[64 * D1];
    __shared__ float sX[64 * 65];
    __shared__ float sM[64 * D1];
    __shared__ float sred[2][1024];
    __shared__ float sE[2];
    const int h = blockIdx.x, tid = threadIdx.x;
    const float* up = Upart + (size_t)h * nkb * m * D1;
    for (int e = tid; e < 64 * D1; e += 1024) {
        const int a = e / D1;
        float t = 0.f;
        if (a < m) {
#pragma unroll 32
            for (int k = 0; k < nkb; ++k) t += up[(size_t)k * m * D1 + e];
            U[(size_t)h * m * D1 + e] = t;
        }
        sU[e] = t;
    }
    for (int e = tid; e < 4096; e += 1024) sX[(e >> 6) * 65 + (e & 63)] = XT[(size_t)h * 4096 + e];
    __syncthreads();
    float mv = 0.f, m1 = 0.f;
    for (int e = tid; e < 64 * D1; e += 1024) {
        const int a = e / D1, c = e % D1;
        float t = 0.f;
        if (a < m) {
#pragma unroll 8
            for (int b = 0; b < m; ++b) t = fmaf(sX[a * 65 + b], sU[b * D1 + c], t);
            Mout[(size_t)h * m * D1 + e] = t;
        }
        sM[e] = t;
        if (c < D) mv = fmaxf(mv, fabsf(t));
        else m1 = fmaxf(m1, fabsf(t));
    }
    sred[0][tid] = mv;
    sred[1][tid] = m1;
    __syncthreads();
    if (tid < 2) {
        float mx = 0.f;
        for (int r = 0; r < 1024; ++r) mx = fmaxf(mx, sred[tid][r]);
        sE[tid] = (mx > 0.f && isfinite(mx)) ? (float)(ilogbf(mx) - 14) : 0.f;
        mscale[h * 2 + tid] = ldexpf(1.f, (int)sE[tid]);
    }
    __syncthreads();
    const int ev = (int)sE[0], e1 = (int)sE[1];
    for (int e = tid; e < 4 * (CB + 1) * 64 * 8; e += 1024) {
        const int i = e & 7, lane = (e >> 3) & 63, cb = (e >> 9) % (CB + 1), s4 = (e >> 9) / (CB + 1);
        const int row = 16 * s4 + 8 * (lane >> 5) + i, j = lane & 31;
        float v = 0.f;
        if (cb < CB) v = ldexpf(sM[row * D1 + 32 * cb + j], -ev);
        else if (j == 0) v = ldexpf(sM[row * D1 + D], -e1);
        const _Float16 hi = (_Float16)v;
        const _Float16 lo = (_Float16)(v - (float)hi);
        const size_t o = ((((size_t)h * 4 + s4) * (CB + 1) + cb) * 2) * 512 + lane * 8 + i;
        Mt[o] = hi;
        Mt[o + 512] = lo;
    }
}

// ------------------------------------------------------------------------------------------
// Query side.  grid (ceil(n/256), BH), 256 threads, lane = query.  Per wave: u(q_i) in
// registers, the m kernel values a_il from v_sad_u16 against the landmark-key table
// (wave-uniform, scalar loads) packed as fp16 pairs, a permlane32 swap that turns "query per
// lane" into the 32x32x16 operand layout for both 32-query halves, then Y^T = (M_hi + M_lo)^T A^T
// on fp16 MFMA: the result holds, per lane, 16 output columns of one query, so the
// normalisation and the bf16 stores happen straight from registers.
template <int D, int NORM>
__global__ __launch_bounds__(256) void query2_kernel(const uint16_t* __restrict__ Q, uint16_t* __restrict__ Out,
                                                     const uint32_t* __restrict__ kfix,
                                                     const float* __restrict__ frame, const _Float16* __restrict__ Mt,
                                                     const float* __restrict__ mscale, const float* __restrict__ vbar,
                                                     int n, int m) {
    constexpr int D2 = D / 2;
    constexpr int D8 = D / 8;
    constexpr int CB = D / 32;
    __shared__ __attribute__((aligned(16))) _Float16 sM[4 * (CB + 1) * 2 * 512];
    __shared__ __attribute__((aligned(16))) float sVb[D];
    const int h = blockIdx.y, tid = threadIdx.x, w = tid >> 6, l = tid & 63;
    {
        const uint4* src = reinterpret_cast<const uint4*>(Mt + (size_t)h * 4 * (CB + 1) * 2 * 512);
        uint4* dst = reinterpret_cast<uint4*>(sM);
        for (int e = tid; e < 4 * (CB + 1) * 2 * 64; e += 256) dst[e] = src[e];
        if (tid < D) sVb[tid] = vbar[(size_t)h * D + tid];
    }
    const float R = frame[h * 4 + 0], inv2R = frame[h * 4 + 1], esc = frame[h * 4 + 2];
    const float ebias = -kTwo23 * esc;
    const float scv = mscale[h * 2 + 0], sc1 = mscale[h * 2 + 1];
    const uint32_t* tab = kfix + (size_t)h * 64 * D2;
    const int i0 = blockIdx.x * 256 + w * 64;
    const int i = i0 + l;
    uint32_t qf[D2];
    if (i < n) {
        const uint4* qr = reinterpret_cast<const uint4*>(Q + ((size_t)h * n + i) * D);
        uint4 raw[D8];
#pragma unroll
        for (int c8 = 0; c8 < D8; ++c8) raw[c8] = qr[c8];
#pragma unroll
        for (int c8 = 0; c8 < D8; ++c8) {
            qf[4 * c8 + 0] = fix2_bf16(raw[c8].x, inv2R);
            qf[4 * c8 + 1] = fix2_bf16(raw[c8].y, inv2R);
            qf[4 * c8 + 2] = fix2_bf16(raw[c8].z, inv2R);
            qf[4 * c8 + 3] = fix2_bf16(raw[c8].w, inv2R);
        }
    } else {
#pragma unroll
        for (int c = 0; c < D2; ++c) qf[c] = 0u;
    }
    // kernel values, two landmarks per fp16 pair register (landmarks >= m give 0)
    uint32_t ah[32];
#pragma unroll
    for (int p = 0; p < 32; ++p) {
        uint32_t v = 0u;
        if (2 * p < m) {
            const uint32_t* t0 = tab + (2 * p) * D2;
            const uint32_t* t1 = tab + (2 * p + 1) * D2;
            uint32_t u0 = 0x4B000000u, u1 = 0x4B000000u;
#pragma unroll
            for (int c = 0; c < D2; ++c) {
                u0 = __builtin_amdgcn_sad_u16(qf[c], t0[c], u0);
                u1 = __builtin_amdgcn_sad_u16(qf[c], t1[c], u1);
            }
            const float a0 = __builtin_amdgcn_exp2f(fmaf(__uint_as_float(u0), esc, ebias));
            float a1 = __builtin_amdgcn_exp2f(fmaf(__uint_as_float(u1), esc, ebias));
            if (2 * p + 1 >= m) a1 = 0.f;
            v = pk_f16(a0, a1);
        }
        ah[p] = v;
    }
    // lower half keeps ah[8s+t] (queries 0..31, landmarks 16s..16s+7) and receives queries
    // 32..63 / landmarks 16s..16s+7; the upper half receives queries 0..31 / 16s+8..16s+15
    // and keeps queries 32..63 / 16s+8..16s+15.
#pragma unroll
    for (int s4 = 0; s4 < 4; ++s4)
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const auto r = __builtin_amdgcn_permlane32_swap(ah[8 * s4 + t], ah[8 * s4 + 4 + t], false, false);
            ah[8 * s4 + t] = r[0];
            ah[8 * s4 + 4 + t] = r[1];
        }
    __syncthreads();   // sM, sVb
    const int NSTEP = (m + 15) / 16;
    const bool nan_head = !isfinite(R);
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
        h8_t A[4];
#pragma unroll
        for (int s4 = 0; s4 < 4; ++s4)
            A[s4] = __builtin_bit_cast(h8_t, (uint4){ah[8 * s4 + 4 * qb], ah[8 * s4 + 4 * qb + 1],
                                                     ah[8 * s4 + 4 * qb + 2], ah[8 * s4 + 4 * qb + 3]});
        // ones column: s_i of query 32qb + l%32 lands in register 0 of lane l%32
        f32x16_t acc = {};
#pragma unroll
        for (int s4 = 0; s4 < 4; ++s4) {
            if (s4 < NSTEP) {
                const _Float16* bt = sM + ((s4 * (CB + 1) + CB) * 2) * 512 + l * 8;
                acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(*reinterpret_cast<const h8_t*>(bt), A[s4], acc, 0, 0, 0);
                acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(*reinterpret_cast<const h8_t*>(bt + 512), A[s4], acc, 0,
                                                             0, 0);
            }
        }
        const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(acc[0]), __float_as_uint(acc[0]), false,
                                                         false);
        const float si = __uint_as_float(sw[0]) * sc1;
        float tmul, tadd;   // o = y * tmul + tadd * vbar
        if (NORM == NORM_INLINE) { tmul = scv; tadd = 1.f - si; }
        else if (NORM == NORM_ROWSUM) { tmul = scv / si; tadd = 0.f; }
        else { tmul = scv; tadd = 0.f; }
        const int iq = i0 + 32 * qb + (l & 31);
        uint16_t* orow = Out + ((size_t)h * n + iq) * D;
#pragma unroll
        for (int cb = 0; cb < CB; ++cb) {
            f32x16_t y = {};
#pragma unroll
            for (int s4 = 0; s4 < 4; ++s4) {
                if (s4 < NSTEP) {
                    const _Float16* bt = sM + ((s4 * (CB + 1) + cb) * 2) * 512 + l * 8;
                    y = __builtin_amdgcn_mfma_f32_32x32x16_f16(*reinterpret_cast<const h8_t*>(bt), A[s4], y, 0, 0, 0);
                    y = __builtin_amdgcn_mfma_f32_32x32x16_f16(*reinterpret_cast<const h8_t*>(bt + 512), A[s4], y, 0, 0,
                                                               0);
                }
            }
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int c0 = 32 * cb + 8 * g + 4 * (l >> 5);
                const float4 vb = *reinterpret_cast<const float4*>(&sVb[c0]);
                float o0 = fmaf(y[4 * g + 0], tmul, tadd * vb.x);
                float o1 = fmaf(y[4 * g + 1], tmul, tadd * vb.y);
                float o2 = fmaf(y[4 * g + 2], tmul, tadd * vb.z);
                float o3 = fmaf(y[4 * g + 3], tmul, tadd * vb.w);
                if (nan_head) o0 = o1 = o2 = o3 = __builtin_nanf("");
                typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
                const bf16x2_t p0 = {(__bf16)o0, (__bf16)o1}, p1 = {(__bf16)o2, (__bf16)o3};
                if (iq < n) {
                    uint2 st;
                    st.x = __builtin_bit_cast(uint32_t, p0);
                    st.y = __builtin_bit_cast(uint32_t, p1);
                    *reinterpret_cast<uint2*>(orow + c0) = st;
                }
            }
        }
    }
}

// ------------------------------------------------------------------------------------------
// Launch wrappers.

hipError_t launch_fast_pool(const void* Q, const void* K, const void* V, float* qt, float* kt, double* vseg,
                            float* segmax, float* vsegmax, int BH, int n, int d, int m, hipStream_t st) {
    dim3 grid(m, BH);
    if (d == 32)
        hipLaunchKernelGGL(pool2_kernel<32>, grid, dim3(256), 0, st, (const uint16_t*)Q, (const uint16_t*)K,
                           (const uint16_t*)V, qt, kt, vseg, segmax, vsegmax, n, m);
    else
        hipLaunchKernelGGL(pool2_kernel<64>, grid, dim3(256), 0, st, (const uint16_t*)Q, (const uint16_t*)K,
                           (const uint16_t*)V, qt, kt, vseg, segmax, vsegmax, n, m);
    return hipGetLastError();
}

hipError_t launch_fast_frame(const float* qt, const float* kt, const double* vseg, const float* segmax,
                             const float* vsegmax, float* frame, uint32_t* qfix, uint32_t* kfix, float* vbar, int BH,
                             int n, int d, int m, float lambda, hipStream_t st) {
    if (d == 32)
        hipLaunchKernelGGL(frame_kernel<32>, dim3(BH), dim3(256), 0, st, qt, kt, vseg, segmax, vsegmax, frame, qfix,
                           kfix, vbar, n, m, lambda);
    else
        hipLaunchKernelGGL(frame_kernel<64>, dim3(BH), dim3(256), 0, st, qt, kt, vseg, segmax, vsegmax, frame, qfix,
                           kfix, vbar, n, m, lambda);
    return hipGetLastError();
}

hipError_t launch_fast_nskey(const float* qt, const float* kt, float* XT, float* cinfo, const void* K, const void* V,
                             const uint32_t* qfix, const float* frame, float* Upart, int BH, int n, int d, int m,
                             int T, float lambda, float eps, int kpb, int nkb, hipStream_t st) {
    const float ks = (float)(-1.4426950408889634 / (double)lambda);
    dim3 grid(BH + BH * nkb);
    if (d == 32)
        hipLaunchKernelGGL(nskey_kernel<32>, grid, dim3(256), 0, st, qt, kt, XT, cinfo, (const uint16_t*)K,
                           (const uint16_t*)V, qfix, frame, Upart, BH, n, m, T, ks, eps, kpb, nkb);
    else
        hipLaunchKernelGGL(nskey_kernel<64>, grid, dim3(256), 0, st, qt, kt, XT, cinfo, (const uint16_t*)K,
                           (const uint16_t*)V, qfix, frame, Upart, BH, n, m, T, ks, eps, kpb, nkb);
    return hipGetLastError();
}

hipError_t launch_fast_mfinal(const float* Upart, const float* XT, _Float16* Mt, float* mscale, float* U, float* M,
                              int BH, int d, int m, int nkb, hipStream_t st) {
    if (d == 32)
        hipLaunchKernelGGL(mfinal_kernel<32>, dim3(BH), dim3(1024), 0, st, Upart, XT, Mt, mscale, U, M, m, nkb);
    else
        hipLaunchKernelGGL(mfinal_kernel<64>, dim3(BH), dim3(1024), 0, st, Upart, XT, Mt, mscale, U, M, m, nkb);
    return hipGetLastError();
}

hipError_t launch_fast_query(int norm, const void* Q, void* Out, const uint32_t* kfix, const float* frame,
                             const _Float16* Mt, const float* mscale, const float* vbar, int BH, int n, int d, int m,
                             hipStream_t st) {
    dim3 grid((n + 255) / 256, BH);
#define LAPATTN_Q2(Dv, Nv)                                                                                        \
    hipLaunchKernelGGL((query2_kernel<Dv, Nv>), grid, dim3(256), 0, st, (const uint16_t*)Q, (uint16_t*)Out, kfix, \
                       frame, Mt, mscale, vbar, n, m)
    if (d == 32) {
        if (norm == NORM_INLINE) LAPATTN_Q2(32, NORM_INLINE);
        else if (norm == NORM_ROWSUM) LAPATTN_Q2(32, NORM_ROWSUM);
        else LAPATTN_Q2(32, NORM_NONE);
    } else {
        if (norm == NORM_INLINE) LAPATTN_Q2(64, NORM_INLINE);
        else if (norm == NORM_ROWSUM) LAPATTN_Q2(64, NORM_ROWSUM);
        else LAPATTN_Q2(64, NORM_NONE);
    }
#undef LAPATTN_Q2
    return hipGetLastError();
}

}  // namespace lapattn
