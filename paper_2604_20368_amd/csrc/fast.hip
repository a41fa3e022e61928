// fast.hip -- the bf16 forward path: fixed-point L1 distances on the VALU (v_sad_u16),
// contractions on the matrix cores (fp16 MFMA), Newton-Schulz on fp32 MFMA.
//
//   pool2_kernel     landmark means (Sec. 4.2, sampling; 1-D segments) and per-segment
//                    value sums / magnitudes, 16-byte vector loads
//   frame_kernel     per head: the fixed-point frame of the L1 distances, the landmark
//                    tables in that frame, the value mean and the value prescale
//   nskey_kernel     one launch, two roles: blocks [0, BH) run Algorithm 2 on K_LL with
//                    fp16-pair MFMA; the other blocks form U = K_LK [V | 1] over key chunks
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
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
    return v;
}

// Maximum of a non-negative value over the wave with DPP lane moves (no LDS round trips);
// the result is wave-uniform.
__device__ __forceinline__ float wave_max_dpp(float v) {
    int x = __float_as_int(v);
    x = max(x, __builtin_amdgcn_update_dpp(0, x, 0xB1, 0xF, 0xF, false));   // quad_perm [1,0,3,2]
    x = max(x, __builtin_amdgcn_update_dpp(0, x, 0x4E, 0xF, 0xF, false));   // quad_perm [2,3,0,1]
    x = max(x, __builtin_amdgcn_update_dpp(0, x, 0x141, 0xF, 0xF, false));  // row_half_mirror
    x = max(x, __builtin_amdgcn_update_dpp(0, x, 0x140, 0xF, 0xF, false));  // row_mirror
    x = max(x, __builtin_amdgcn_update_dpp(0, x, 0x142, 0xA, 0xF, false));  // row_bcast:15
    x = max(x, __builtin_amdgcn_update_dpp(0, x, 0x143, 0xC, 0xF, false));  // row_bcast:31
    return __int_as_float(__builtin_amdgcn_readlane(x, 63));
}

// Maximum over the wave and the lowest lane index holding it.
__device__ __forceinline__ void wave_argmax(float& v, int& idx) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        const float v2 = __shfl_xor(v, off, 64);
        const int i2 = __shfl_xor(idx, off, 64);
        if (v2 > v || (v2 == v && i2 < idx)) {
            v = v2;
            idx = i2;
        }
    }
}

typedef float f32x2_t __attribute__((ext_vector_type(2)));

// Two floats to a packed fp16 pair, round to nearest even (v_cvt_pk_f16_f32).
__device__ __forceinline__ uint32_t pk_f16(float a, float b) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){a, b}, f16x2_t));
}

// Workgroups are dispatched to the 8 XCDs round-robin (block id mod 8); each XCD has its own
// L2 and its CUs share scalar caches.  xcd_rank maps the i-th of n consecutive blocks (first
// block id `base`) to a logical index such that the blocks running on one XCD get a
// contiguous range -- so they work on the same one or two heads and share their landmark
// tables and operand tiles in cache.  It is a bijection of [0, n).
__device__ __forceinline__ int xcd_rank(int i, int n, int base) {
    const int x = (base + i) & 7;
    const int y = (i - ((x - base) & 7)) >> 3;
    int off = 0;
    for (int xp = 0; xp < x; ++xp) {
        const int j0 = (xp - base) & 7;
        off += j0 < n ? (n - j0 + 7) >> 3 : 0;
    }
    return off + y;
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
    __shared__ float smx[4], svmx[4];
    mx = wave_max(mx);
    vmx = wave_max(vmx);
    if ((tid & 63) == 0) {
        smx[tid >> 6] = mx;
        svmx[tid >> 6] = vmx;
    }
    const double cnt = (double)(s1 - s0);
    bool bad = false;
    for (int pass = 0; pass < 3; ++pass) {
        const float* src = pass == 0 ? sq : (pass == 1 ? sk : sv);
#pragma unroll
        for (int j = 0; j < 8; ++j) red[tid * 8 + j] = (double)src[j];
        __syncthreads();
        if (tid < D) {
            const int g = tid / 8, j = tid % 8;
            double t = 0.0;
#pragma unroll
            for (int r = 0; r < RPI; ++r) t += red[(g + CPR * r) * 8 + j];
            const size_t o = ((size_t)h * m + l) * D + tid;
            if (pass == 0) qt[o] = (float)(t / cnt);
            else if (pass == 1) kt[o] = (float)(t / cnt);
            else vseg[o] = t;
            bad |= !isfinite(t);
        }
        __syncthreads();
    }
    if (tid < 64) {   // D <= 64: every column flag lives in wave 0
        const bool anybad = __any(bad);
        if (tid == 0) {
            const float a = fmaxf(fmaxf(smx[0], smx[1]), fmaxf(smx[2], smx[3]));
            const float b = fmaxf(fmaxf(svmx[0], svmx[1]), fmaxf(svmx[2], svmx[3]));
            segmax[(size_t)h * m + l] = anybad ? __builtin_nanf("") : a;
            vsegmax[(size_t)h * m + l] = anybad ? __builtin_nanf("") : b;
        }
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
    constexpr int D2 = D / 2;
    constexpr int PER = 64 * D2 / 256;   // table words per thread
    const int h = blockIdx.x, tid = threadIdx.x;
    __shared__ float sS;   // 1 / (2R)
    // every global read this block needs, issued before the first use
    float q0[PER], q1[PER], k0[PER], k1[PER];
#pragma unroll
    for (int r = 0; r < PER; ++r) {
        const int e = tid + 256 * r, a = e / D2, c2 = e % D2;
        const size_t o = ((size_t)h * m + (a < m ? a : 0)) * D + 2 * c2;
        q0[r] = qt[o]; q1[r] = qt[o + 1]; k0[r] = kt[o]; k1[r] = kt[o + 1];
    }
    double vs = 0.0;
    if (tid < D) {
#pragma unroll 16
        for (int l = 0; l < m; ++l) vs += vseg[((size_t)h * m + l) * D + tid];
    }
    if (tid < 64) {
        float a = 0.f, b = 0.f;
        if (tid < m) {
            a = segmax[(size_t)h * m + tid];
            b = vsegmax[(size_t)h * m + tid];
        }
        const bool bad = __any(!(isfinite(a) && isfinite(b)));
        float R = wave_max(a);
        const float vm = wave_max(b);
        if (tid == 0) {
            if (R == 0.f) R = 1.f;
            const float S = (float)(65535.0 / (2.0 * (double)R));
            float vscale = 1.f;
            if (vm > 16384.f) vscale = exp2f(-ceilf(log2f(vm / 16384.f)));
            sS = (float)(0.5 / (double)R);
            frame[h * 4 + 0] = bad ? __builtin_nanf("") : R;
            frame[h * 4 + 1] = sS;
            frame[h * 4 + 2] = (float)(-1.4426950408889634 / ((double)lambda * (double)S));
            frame[h * 4 + 3] = vscale;
        }
    }
    if (tid < D) vbar[(size_t)h * D + tid] = (float)(vs / n);
    __syncthreads();
    const float inv2R = sS;
#pragma unroll
    for (int r = 0; r < PER; ++r) {
        const int e = tid + 256 * r, a = e / D2;
        qfix[(size_t)h * 64 * D2 + e] = a < m ? fix2(q0[r], q1[r], inv2R) : 0u;
        kfix[(size_t)h * 64 * D2 + e] = a < m ? fix2(k0[r], k1[r], inv2R) : 0u;
    }
}

__device__ __forceinline__ int c_row(int r, int l) { return 8 * (r >> 2) + 4 * (l >> 5) + (r & 3); }

__device__ __forceinline__ void split_f16(float v, _Float16& hi, _Float16& lo) {
    hi = (_Float16)v;
    lo = (_Float16)(v - (float)hi);
}

// One wave's 32 x 32 block (rb, cb) of the 64 x 64 product A B with both factors carried as an
// fp16 pair (value + residual, ~22 significant bits): A row-major and B transposed ([col][k]),
// LDS row pitch kLP.  A B ~ Ahi Bhi + Ahi Blo + Alo Bhi on v_mfma_f32_32x32x16_f16; lane l
// supplies A[row l%32][k 8(l/32)..+8] and B^T[col l%32][k 8(l/32)..+8]; result register r holds
// row 32rb + c_row(r, l), column 32cb + l%32.
__device__ __forceinline__ f32x16_t mm_split(const _Float16* __restrict__ Ah, const _Float16* __restrict__ Al,
                                             const _Float16* __restrict__ BTh, const _Float16* __restrict__ BTl,
                                             int rb, int cb) {
    const int l = threadIdx.x & 63;
    f32x16_t acc = {};
    const int ao = (32 * rb + (l & 31)) * kLP + 8 * (l >> 5);
    const int bo = (32 * cb + (l & 31)) * kLP + 8 * (l >> 5);
#pragma unroll
    for (int s4 = 0; s4 < 4; ++s4) {
        const h8_t ah = *reinterpret_cast<const h8_t*>(Ah + ao + 16 * s4);
        const h8_t al = *reinterpret_cast<const h8_t*>(Al + ao + 16 * s4);
        const h8_t bh = *reinterpret_cast<const h8_t*>(BTh + bo + 16 * s4);
        const h8_t bl = *reinterpret_cast<const h8_t*>(BTl + bo + 16 * s4);
        acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(ah, bh, acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(ah, bl, acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_32x32x16_f16(al, bh, acc, 0, 0, 0);
    }
    return acc;
}

// Store one wave's C block (scaled by `scale`) as an fp16 pair, row-major (Mh/Ml) and, when
// MTh is given, transposed (MTh/MTl, four consecutive rows per 8-byte write).
__device__ __forceinline__ void store_split(const f32x16_t& v, float scale, int rb, int cb, _Float16* Mh,
                                            _Float16* Ml, _Float16* MTh, _Float16* MTl) {
    const int l = threadIdx.x & 63;
    const int col = 32 * cb + (l & 31);
#pragma unroll
    for (int g = 0; g < 4; ++g) {
        _Float16 hi[4], lo[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            split_f16(v[4 * g + i] * scale, hi[i], lo[i]);
            const int row = 32 * rb + 8 * g + 4 * (l >> 5) + i;
            if (Mh) {
                Mh[row * kLP + col] = hi[i];
                Ml[row * kLP + col] = lo[i];
            }
        }
        if (MTh) {
            const int row0 = 32 * rb + 8 * g + 4 * (l >> 5);
            typedef _Float16 h4_t __attribute__((ext_vector_type(4)));
            *reinterpret_cast<h4_t*>(MTh + col * kLP + row0) = (h4_t){hi[0], hi[1], hi[2], hi[3]};
            *reinterpret_cast<h4_t*>(MTl + col * kLP + row0) = (h4_t){lo[0], lo[1], lo[2], lo[3]};
        }
    }
}

// Power-of-two exponent that brings a maximum magnitude into [2^14, 2^15) (0 when mx is 0).
__device__ __forceinline__ int pow2_exp(float mx) { return (mx > 0.f && isfinite(mx)) ? ilogbf(mx) - 14 : 0; }

// ------------------------------------------------------------------------------------------
// Newton-Schulz role (one block per head, 4 waves; wave w owns the 32 x 32 block (w/2, w%2)).
//   W = K_LL + eps I padded to 64 x 64, from the landmark tables in the fixed-point frame
//   (v_sad_u16, lane = row a, the landmark-key row b wave-uniform);
//   c = ||W||_1 ||W||_inf (first maximising column / row); X0 = W^T / c (0 if c = 0);
//   X_{t+1} = X_t (2I - W X_t) with both products on fp16-pair MFMA, X carried with a
//   power-of-two scale so its largest entry sits in [2^14, 2^15).
//   Writes X_T (fp32, [64][64]) and cinfo = {c, n1, ninf, a* 256 + b*}.
constexpr int kNsLds = 8 * 64 * kLP * 2 + 16 * 4 + 128 * 4;

template <int D>
__device__ void ns_role(int h, char* lds_raw, const uint32_t* __restrict__ qfix, const uint32_t* __restrict__ kfix,
                        const float* __restrict__ frame, int m, int T, float eps, float* __restrict__ XT,
                        float* __restrict__ cinfo) {
    constexpr int D2 = D / 2;
    const int tid = threadIdx.x, w = tid >> 6, l = tid & 63;
    const int rb = w >> 1, cb = w & 1;
    _Float16* base = reinterpret_cast<_Float16*>(lds_raw);
    _Float16* Wh = base;
    _Float16* Wl = base + 1 * 64 * kLP;
    _Float16* Xh = base + 2 * 64 * kLP;
    _Float16* Xl = base + 3 * 64 * kLP;
    _Float16* XTh = base + 4 * 64 * kLP;
    _Float16* XTl = base + 5 * 64 * kLP;
    _Float16* TTh = base + 6 * 64 * kLP;
    _Float16* TTl = base + 7 * 64 * kLP;
    // set-up only: W in fp32 and the landmark-key table (alias XT*/TT* and X*)
    float* sWf = reinterpret_cast<float*>(base + 4 * 64 * kLP);
    uint32_t* sK = reinterpret_cast<uint32_t*>(base + 2 * 64 * kLP);
    unsigned* sred = reinterpret_cast<unsigned*>(base + 8 * 64 * kLP);   // 16 words
    const float esc = frame[h * 4 + 2];
    const float ebias = -kTwo23 * esc;

    // landmark-query row of lane a in registers, landmark-key table in LDS (one round trip each)
    uint32_t qa[D2];
    {
        const uint4* qp = reinterpret_cast<const uint4*>(qfix + ((size_t)h * 64 + l) * D2);
#pragma unroll
        for (int c4 = 0; c4 < D2 / 4; ++c4) {
            const uint4 x = qp[c4];
            qa[4 * c4] = x.x; qa[4 * c4 + 1] = x.y; qa[4 * c4 + 2] = x.z; qa[4 * c4 + 3] = x.w;
        }
        const uint4* kp = reinterpret_cast<const uint4*>(kfix + (size_t)h * 64 * D2);
        uint4* sk4 = reinterpret_cast<uint4*>(sK);
#pragma unroll
        for (int r = 0; r < 64 * D2 / 4 / 256; ++r) sk4[tid + 256 * r] = kp[tid + 256 * r];
    }
    if (tid < 16) sred[tid] = 0u;
    __syncthreads();
    // W[a][b] = k(qt_a, kt_b) (+ eps on the diagonal): lane a, wave w takes b in [16w, 16w+16)
#pragma unroll 2
    for (int bb = 0; bb < 16; ++bb) {
        const int b = 16 * w + bb;
        const uint4* kr = reinterpret_cast<const uint4*>(sK + b * D2);
        uint32_t u0 = 0x4B000000u, u1 = 0u;
#pragma unroll
        for (int c4 = 0; c4 < D2 / 4; ++c4) {
            const uint4 t = kr[c4];
            u0 = __builtin_amdgcn_sad_u16(qa[4 * c4 + 0], t.x, u0);
            u1 = __builtin_amdgcn_sad_u16(qa[4 * c4 + 1], t.y, u1);
            u0 = __builtin_amdgcn_sad_u16(qa[4 * c4 + 2], t.z, u0);
            u1 = __builtin_amdgcn_sad_u16(qa[4 * c4 + 3], t.w, u1);
        }
        float v = __builtin_amdgcn_exp2f(fmaf(__uint_as_float(u0 + u1), esc, ebias));
        if (l == b) v += eps;
        sWf[l * 65 + b] = (l < m && b < m) ? v : 0.f;
    }
    __syncthreads();
    // column sums (wave 0) and row sums (wave 1) into LDS, the largest |W| by LDS atomic max
    float* csum = reinterpret_cast<float*>(sred + 16);   // 128 floats after the 16 words
    if (w < 2) {
        float sum = 0.f, mx = 0.f;
#pragma unroll
        for (int i = 0; i < 64; ++i) {
            const float x = fabsf(w == 0 ? sWf[i * 65 + l] : sWf[l * 65 + i]);
            sum += x;
            mx = fmaxf(mx, x);
        }
        csum[64 * w + l] = sum;
        mx = wave_max_dpp(mx);
        if (l == 0 && w == 0) sred[0] = __float_as_uint(mx);
    }
    __syncthreads();
    // first maximising column / row (all 128 sums loaded at once, then a serial scan)
    if (tid == 0) {
        float sums[128];
#pragma unroll
        for (int i = 0; i < 128; ++i) sums[i] = csum[i];
        float n1 = -1.f, ninf = -1.f;
        int bs = 0, as = 0;
#pragma unroll
        for (int i = 0; i < 64; ++i) {
            if (sums[i] > n1) { n1 = sums[i]; bs = i; }
            if (sums[64 + i] > ninf) { ninf = sums[64 + i]; as = i; }
        }
        const float c = n1 * ninf;
        reinterpret_cast<float*>(sred)[1] = c;
        cinfo[h * 4 + 0] = c;
        cinfo[h * 4 + 1] = n1;
        cinfo[h * 4 + 2] = ninf;
        cinfo[h * 4 + 3] = (float)(as * 256 + bs);
    }
    // W and X0 = W^T / c into the fp16-pair tiles (all of sWf is read before it is overwritten)
    float wv[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) wv[k] = sWf[((tid + 256 * k) >> 6) * 65 + ((tid + 256 * k) & 63)];
    __syncthreads();
    const float c = reinterpret_cast<float*>(sred)[1];
    const float inv_c = c > 0.f ? 1.f / c : 0.f;
    float xs = ldexpf(1.f, pow2_exp(__uint_as_float(sred[0]) * inv_c));   // X_true = X_stored * xs
    const float x0s = inv_c / xs;
#pragma unroll
    for (int k = 0; k < 16; ++k) {
        const int e = tid + 256 * k, a = e >> 6, b = e & 63;
        _Float16 hi, lo;
        split_f16(wv[k], hi, lo);
        Wh[a * kLP + b] = hi;
        Wl[a * kLP + b] = lo;
        split_f16(wv[k] * x0s, hi, lo);   // X0[b][a]
        Xh[b * kLP + a] = hi;
        Xl[b * kLP + a] = lo;
        XTh[a * kLP + b] = hi;
        XTl[a * kLP + b] = lo;
        if (T == 0) XT[(size_t)h * 4096 + b * 64 + a] = wv[k] * inv_c;
    }
    __syncthreads();
    for (int t = 0; t < T; ++t) {
        // T1 = 2I - W X
        f32x16_t p = mm_split(Wh, Wl, XTh, XTl, rb, cb);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int row = 32 * rb + c_row(r, l), col = 32 * cb + (l & 31);
            p[r] = (row == col ? 2.f : 0.f) - p[r] * xs;
        }
        store_split(p, 1.f, rb, cb, nullptr, nullptr, TTh, TTl);
        __syncthreads();
        // X_{t+1} = X T1, its largest magnitude by LDS atomic max (slot 2 + t % 8, reset ahead)
        f32x16_t xn = mm_split(Xh, Xl, TTh, TTl, rb, cb);
        float mx = 0.f;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            xn[r] *= xs;
            mx = fmaxf(mx, fabsf(xn[r]));
        }
        mx = wave_max_dpp(mx);
        float* slot = reinterpret_cast<float*>(&sred[4 + 4 * (t & 1)]);   // alternating sets of 4
        if (l == 0) slot[w] = mx;
        __syncthreads();
        if (t + 1 < T) {
            xs = ldexpf(1.f, pow2_exp(fmaxf(fmaxf(slot[0], slot[1]), fmaxf(slot[2], slot[3]))));
            store_split(xn, 1.f / xs, rb, cb, Xh, Xl, XTh, XTl);
            __syncthreads();
        } else {
#pragma unroll
            for (int r = 0; r < 16; ++r)
                XT[(size_t)h * 4096 + (32 * rb + c_row(r, l)) * 64 + 32 * cb + (l & 31)] = xn[r];
        }
    }
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
        // two landmarks per step: one scalar fetch of 2 table rows, two independent sad chains;
        // rows 2p, 2p+1 of the [a][j] tile (rows >= m were zeroed once; an odd m writes the
        // zero of landmark m into row m, which stays zero)
        uint16_t* brow = reinterpret_cast<uint16_t*>(sB) + l;
#pragma unroll 1
        for (int p = 0; 2 * p < m; ++p) {
            const uint32_t* t0 = tab + (2 * p) * D2;
            const uint32_t* t1 = t0 + D2;
            uint32_t u0 = 0x4B000000u, u1 = 0x4B000000u;
#pragma unroll
            for (int c = 0; c < D2; ++c) {
                u0 = __builtin_amdgcn_sad_u16(kf[c], t0[c], u0);
                u1 = __builtin_amdgcn_sad_u16(kf[c], t1[c], u1);
            }
            const float b0 = __builtin_amdgcn_exp2f(fmaf(__uint_as_float(u0), esc, ebias));
            const float b1 = __builtin_amdgcn_exp2f(fmaf(__uint_as_float(u1), esc, ebias));
            const uint32_t v = valid ? pk_f16(b0, 2 * p + 1 < m ? b1 : 0.f) : 0u;
            brow[(2 * p) * kLP] = (uint16_t)(v & 0xffffu);
            brow[(2 * p + 1) * kLP] = (uint16_t)(v >> 16);
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
constexpr int kKeyLds = 4 * 2 * 64 * kLP * 2;
constexpr int kNsKeyLds = kNsLds > kKeyLds ? kNsLds : kKeyLds;

template <int D>
__global__ __launch_bounds__(256) void nskey_kernel(float* __restrict__ XT, float* __restrict__ cinfo,
                                                    const uint16_t* __restrict__ K, const uint16_t* __restrict__ V,
                                                    const uint32_t* __restrict__ qfix,
                                                    const uint32_t* __restrict__ kfix,
                                                    const float* __restrict__ frame, float* __restrict__ Upart,
                                                    int BH, int n, int m, int T, float eps, int kpb, int nkb) {
    __shared__ __attribute__((aligned(16))) char lds[kNsKeyLds];
    const int b = blockIdx.x;
    if (b < BH) {
        ns_role<D>(b, lds, qfix, kfix, frame, m, T, eps, XT, cinfo);
    } else {
        const int kbb = xcd_rank(b - BH, BH * nkb, BH);
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
    constexpr int NC = 32 * (CB + 1);       // padded columns of U and M
    constexpr int PER = (64 * D1 + 1023) / 1024;
    __shared__ float sU[64 * NC];
    __shared__ float sX[64 * 65];
    __shared__ float sM[64 * NC];
    __shared__ unsigned smax[2];
    const int h = blockIdx.x, tid = threadIdx.x, w = tid >> 6, l = tid & 63;
    if (tid < 2) smax[tid] = 0u;
    // U = sum of the key-chunk partials: every thread owns PER entries and keeps PER loads in flight
    const float* up = Upart + (size_t)h * nkb * m * D1;
    const int mD1 = m * D1;
    float acc[PER];
#pragma unroll
    for (int r = 0; r < PER; ++r) acc[r] = 0.f;
    for (int k0 = 0; k0 < nkb; k0 += 8) {
        float t[8][PER];
#pragma unroll
        for (int kk = 0; kk < 8; ++kk)
#pragma unroll
            for (int r = 0; r < PER; ++r) {
                const int e = tid + 1024 * r;
                t[kk][r] = (k0 + kk < nkb && e < mD1) ? up[(size_t)(k0 + kk) * mD1 + e] : 0.f;
            }
#pragma unroll
        for (int kk = 0; kk < 8; ++kk)
#pragma unroll
            for (int r = 0; r < PER; ++r) acc[r] += t[kk][r];
    }
    for (int e = tid; e < 64 * NC; e += 1024) sU[e] = 0.f;
    for (int e = tid; e < 4096; e += 1024) sX[(e >> 6) * 65 + (e & 63)] = XT[(size_t)h * 4096 + e];
    __syncthreads();
#pragma unroll
    for (int r = 0; r < PER; ++r) {
        const int e = tid + 1024 * r;
        if (e < mD1) {
            sU[(e / D1) * NC + e % D1] = acc[r];
            U[(size_t)h * mD1 + e] = acc[r];
        }
    }
    __syncthreads();
    // M = X_T U on fp32 MFMA 32x32x2: wave w < 2 (CB + 1) owns block (w % 2, w / 2)
    if (w < 2 * (CB + 1)) {
        const int rb = w & 1, cb = w >> 1;
        typedef float f32x16_t2 __attribute__((ext_vector_type(16)));
        f32x16_t2 c = {};
        const float* a = sX + (32 * rb + (l & 31)) * 65 + (l >> 5);
        const float* b = sU + (l >> 5) * NC + 32 * cb + (l & 31);
#pragma unroll 8
        for (int s2 = 0; s2 < 32; ++s2) c = __builtin_amdgcn_mfma_f32_32x32x2f32(a[2 * s2], b[2 * s2 * NC], c, 0, 0, 0);
        float mv = 0.f;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int row = 32 * rb + 8 * (r >> 2) + 4 * (l >> 5) + (r & 3), col = 32 * cb + (l & 31);
            sM[row * NC + col] = c[r];
            if (row < m && col < D1) {
                Mout[(size_t)h * mD1 + row * D1 + col] = c[r];
                mv = fmaxf(mv, fabsf(c[r]));
            }
        }
        // magnitudes are non-negative: their bit patterns order like the values
        mv = wave_max_dpp(mv);
        if (l == 0) atomicMax(&smax[cb == CB ? 1 : 0], __float_as_uint(mv));
    }
    __syncthreads();
    const int ev = pow2_exp(__uint_as_float(smax[0])), e1 = pow2_exp(__uint_as_float(smax[1]));
    if (tid < 2) mscale[h * 2 + tid] = ldexpf(1.f, tid == 0 ? ev : e1);
    for (int e = tid; e < 4 * (CB + 1) * 64 * 8; e += 1024) {
        const int i = e & 7, lane = (e >> 3) & 63, cb = (e >> 9) % (CB + 1), s4 = (e >> 9) / (CB + 1);
        const int row = 16 * s4 + 8 * (lane >> 5) + i, j = lane & 31;
        float v = 0.f;
        if (cb < CB) v = ldexpf(sM[row * NC + 32 * cb + j], -ev);
        else if (j == 0) v = ldexpf(sM[row * NC + D], -e1);
        const _Float16 hi = (_Float16)v;
        const _Float16 lo = (_Float16)(v - (float)hi);
        const size_t o = ((((size_t)h * 4 + s4) * (CB + 1) + cb) * 2) * 512 + lane * 8 + i;
        Mt[o] = hi;
        Mt[o + 512] = lo;
    }
}

// ------------------------------------------------------------------------------------------
// Query side.  grid (ceil(n/256) * BH) (XCD-aware order), 256 threads, lane = query.  Per wave: u(q_i) in
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
                                                     int n, int m, int nqb, int BH) {
    constexpr int D2 = D / 2;
    constexpr int D8 = D / 8;
    constexpr int CB = D / 32;
    __shared__ __attribute__((aligned(16))) _Float16 sM[4 * (CB + 1) * 2 * 512];
    __shared__ __attribute__((aligned(16))) float sVb[D];
    const int lin = xcd_rank(blockIdx.x, nqb * BH, 0);
    const int h = lin / nqb, qblk = lin % nqb;
    const int tid = threadIdx.x, w = tid >> 6, l = tid & 63;
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
    const int i0 = qblk * 256 + w * 64;
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

hipError_t launch_fast_nskey(float* XT, float* cinfo, const void* K, const void* V, const uint32_t* qfix,
                             const uint32_t* kfix, const float* frame, float* Upart, int BH, int n, int d, int m,
                             int T, float eps, int kpb, int nkb, hipStream_t st) {
    dim3 grid(BH + BH * nkb);
    if (d == 32)
        hipLaunchKernelGGL(nskey_kernel<32>, grid, dim3(256), 0, st, XT, cinfo, (const uint16_t*)K,
                           (const uint16_t*)V, qfix, kfix, frame, Upart, BH, n, m, T, eps, kpb, nkb);
    else
        hipLaunchKernelGGL(nskey_kernel<64>, grid, dim3(256), 0, st, XT, cinfo, (const uint16_t*)K,
                           (const uint16_t*)V, qfix, kfix, frame, Upart, BH, n, m, T, eps, kpb, nkb);
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
    const int nqb = (n + 255) / 256;
    dim3 grid(nqb * BH);
#define LAPATTN_Q2(Dv, Nv)                                                                                        \
    hipLaunchKernelGGL((query2_kernel<Dv, Nv>), grid, dim3(256), 0, st, (const uint16_t*)Q, (uint16_t*)Out, kfix, \
                       frame, Mt, mscale, vbar, n, m, nqb, BH)
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
