// fast.hip -- the bf16 forward path: fixed-point L1 distances on the VALU (v_sad_u16),
// contractions on the matrix cores (fp16 MFMA), Newton-Schulz on fp32 MFMA.
//
//   pool2_kernel     landmark means (Sec. 4.2, sampling; 1-D segments) and per-segment
//                    value sums / magnitudes, 16-byte vector loads
//   frame_ns_kernel  per head: the fixed-point frame of the L1 distances, the landmark
//                    tables in that frame, the value mean and prescale, then Algorithm 2
//                    on K_LL with fp16-pair MFMA
//   key_kernel       U = K_LK [V | 1] over key chunks (Sec. 3.2 key summaries) with
//                    v_sad_u16 distances and fp16 MFMA
//   mfinal_kernel    U = sum of the chunk partials, M = X_T U, split into fp16 hi/lo
//                    MFMA operand tiles with a power-of-two scale per column
//   query2_kernel    Y = K_QL M (Eq. (8)) and the normalisation (Eq. (4) / Eq. (3))
//
// Distances.  Per head, a range R covering every landmark coordinate (below) and
// S = 65535 / (2R): a coordinate x becomes u(x) = rint((clamp(x, -R, R) + R) S) in [0, 65535]
// (v_cvt_pknorm_u16_f32 of (x + R) / (2R), which saturates, two coordinates per instruction).
// For a token x and a landmark y (|y_c| <= R for every c),
//   ||x - y||_1 = ||clamp(x) - y||_1 + E(x),  E(x) = sum_c max(|x_c| - R, 0),
// exactly: a coordinate beyond R lies on the far side of every landmark coordinate.  So
// sum_c |u(x_c) - u(y_c)| = S ||clamp(x) - y||_1 + e with |e| <= d (each rounding moves a
// coordinate by at most 1/2 a step): the error of the clamped part is at most 2 R d / 65535,
// and E(x) is formed in fp32 once per token and enters the exponent as a per-token bias.
// R = max(landmark max, min(head max, 2 x the median over landmarks of their tokens' max));
// a head without far tokens keeps R = its max |Q|, |K| and E = 0, and one or a few outlier
// tokens no longer coarsen every distance of their head.
// v_sad_u16 adds |a.lo - b.lo| + |a.hi - b.hi| to an accumulator: two coordinates per lane
// and instruction, exact integer arithmetic.  The accumulator starts at the bit pattern of
// 2^23, so after the sum it reads as the float 2^23 + D (D < 2^23 for d <= 64), and one fma
// maps it to the exp2 argument -(D / S + E) log2(e) / lambda.
#include "common.hpp"
#include "kernels.hpp"
#include "ns_split.hpp"

namespace lapattn {

constexpr float kTwo23 = 8388608.f;
// Word 3 of a raw (unswizzled, stride 0) buffer resource on CDNA: 32-bit data format, so that
// loads are range-checked against the byte count in word 2 and return 0 past it.
constexpr int kRawBufferWord3 = 0x00020000;

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

typedef unsigned short u16x2_t __attribute__((ext_vector_type(2)));

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

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

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
// Landmark means and per-landmark statistics.  grid (m, BH), 256 threads.  Thread t always
// reads the 8-column group t % (D/8) of its rows (the landmark's tokens t / (D/8) + (256 / (D/8)) i
// of its segment or window, lm_tokens), four rows per thread in flight at a time.  Sums: per thread in fp32, then over the
// lanes of a wave that share a column group (a butterfly), then over the four waves in a fixed
// order in fp64.  RV = false (the key side with the landmarks split over its waves, which forms
// the value statistics itself): Q and K only, vseg and vsegmax untouched.
template <int D, bool RV>
__global__ __launch_bounds__(256) void pool2_kernel(const uint16_t* __restrict__ Q, const uint16_t* __restrict__ K,
                                                    const uint16_t* __restrict__ V, float* __restrict__ qt,
                                                    float* __restrict__ kt, double* __restrict__ vseg,
                                                    float* __restrict__ segmax, float* __restrict__ vsegmax, int n,
                                                    int m, LmPool pl) {
    constexpr int CPR = D / 8;      // 16-byte chunks per row
    constexpr int RPI = 256 / CPR;  // rows per block iteration
    constexpr int UNR = 4;          // row iterations in flight
    const int l = blockIdx.x, h = blockIdx.y, tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
    const LmTokens tok = lm_tokens(pl, l, n, m);   // the landmark's tokens tok(0 .. count - 1)
    const int cntl = tok.count;
    const int cg = tid % CPR, r0 = tid / CPR;
    float sq[8], sk[8], sv[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) sq[j] = sk[j] = sv[j] = 0.f;
    float mx = 0.f, vmx = 0.f;
    const size_t base = (size_t)h * n * D + cg * 8;
    for (int t0 = r0; t0 < cntl; t0 += UNR * RPI) {
        uint4 a[UNR], b[UNR], c[UNR];
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
            const int t = t0 + u * RPI;
            if (t < cntl) {
                const size_t off = base + (size_t)tok(t) * D;
                a[u] = *reinterpret_cast<const uint4*>(Q + off);
                b[u] = *reinterpret_cast<const uint4*>(K + off);
                c[u] = RV ? *reinterpret_cast<const uint4*>(V + off) : make_uint4(0u, 0u, 0u, 0u);
            } else {
                a[u] = b[u] = c[u] = make_uint4(0u, 0u, 0u, 0u);   // +0: no effect on sums or maxima
            }
        }
#pragma unroll
        for (int u = 0; u < UNR; ++u) {
            const uint32_t aw[4] = {a[u].x, a[u].y, a[u].z, a[u].w}, bw[4] = {b[u].x, b[u].y, b[u].z, b[u].w},
                           cw[4] = {c[u].x, c[u].y, c[u].z, c[u].w};
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const float q0 = bf16_lo(aw[j]), q1 = bf16_hi(aw[j]);
                const float k0 = bf16_lo(bw[j]), k1 = bf16_hi(bw[j]);
                const float v0 = bf16_lo(cw[j]), v1 = bf16_hi(cw[j]);
                sq[2 * j] += q0; sq[2 * j + 1] += q1;
                sk[2 * j] += k0; sk[2 * j + 1] += k1;
                mx = fmaxf(fmaxf(mx, fabsf(q0)), fmaxf(fabsf(q1), fmaxf(fabsf(k0), fabsf(k1))));
                if (RV) {
                    sv[2 * j] += v0; sv[2 * j + 1] += v1;
                    vmx = fmaxf(vmx, fmaxf(fabsf(v0), fabsf(v1)));
                }
            }
        }
    }
    // Within a wave, the lanes with one column group are lane % CPR == cg.  Reduce over the
    // other lane bits by a butterfly; lane cg's result (always the same order) is the one kept.
    float* sums[3] = {sq, sk, sv};
#pragma unroll
    for (int a3 = 0; a3 < (RV ? 3 : 2); ++a3)
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            float v = sums[a3][j];
            if (CPR <= 4) v += __shfl_xor(v, 4, 64);
            v += __shfl_xor(v, 8, 64);
            v += __shfl_xor(v, 16, 64);
            v += __shfl_xor(v, 32, 64);
            sums[a3][j] = v;
        }
    mx = wave_max(mx);
    vmx = wave_max(vmx);
    __shared__ double red[3][4][D];
    __shared__ float smx[4], svmx[4];
    if (lane < CPR) {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            red[0][w][lane * 8 + j] = (double)sq[j];
            red[1][w][lane * 8 + j] = (double)sk[j];
            if (RV) red[2][w][lane * 8 + j] = (double)sv[j];
        }
    }
    if (lane == 0) {
        smx[w] = mx;
        svmx[w] = vmx;
    }
    __syncthreads();
    const double cnt = (double)cntl;
    bool bad = false;
    if (tid < (RV ? 3 : 2) * D) {
        const int a3 = tid / D, col = tid % D;
        const double t = ((red[a3][0][col] + red[a3][1][col]) + red[a3][2][col]) + red[a3][3][col];
        const size_t o = ((size_t)h * m + l) * D + col;
        if (a3 == 0) qt[o] = (float)(t / cnt);
        else if (a3 == 1) kt[o] = (float)(t / cnt);
        else vseg[o] = t;
        bad = !isfinite(t);
    }
    // A non-finite input makes its column sum non-finite (fmaxf alone would hide a NaN).
    const bool anybad = __syncthreads_or(bad);
    if (tid == 0) {
        const float a = fmaxf(fmaxf(smx[0], smx[1]), fmaxf(smx[2], smx[3]));
        const float b = fmaxf(fmaxf(svmx[0], svmx[1]), fmaxf(svmx[2], svmx[3]));
        segmax[(size_t)h * m + l] = anybad ? __builtin_nanf("") : a;
        if (RV) vsegmax[(size_t)h * m + l] = anybad ? __builtin_nanf("") : b;
    }
}

// Scalar loads of one landmark row (D/2 words) into `t`.  The row is read through the
// constant address space: the tables are written by earlier launches and never within the
// reading kernel, and this keeps the loads scalar (s_load) wherever the compiler cannot prove
// the pointer free of the kernel's own stores.
typedef const __attribute__((address_space(4))) uint32_t cu32_t;

template <int D2>
__device__ __forceinline__ void load_row(uint32_t (&t)[D2], const uint32_t* __restrict__ row) {
    cu32_t* q = (cu32_t*)row;
#pragma unroll
    for (int c = 0; c < D2; ++c) t[c] = q[c];
}

// The sad chains start at 0 (an inline operand beside the scalar row word) and meet the 2^23
// bias in their final add, through an operand held in a scalar register: a literal start value
// would cost a move per row.
__device__ __forceinline__ uint32_t bias23() {
    uint32_t b;
    asm("s_mov_b32 %0, 0x4b000000" : "=s"(b));
    return b;
}

// The exp2 argument (lap_arg) and the kernel value (lap_row) of one (lane's token, landmark
// row) pair: two sad chains over the even and odd coordinate pairs; the first sad (the wait
// point for `t`) is issued before the scalar loads of the next row, which go into `nt`.
template <int D2>
__device__ __forceinline__ float lap_arg(const uint32_t (&kf)[D2], const uint32_t (&t)[D2], uint32_t (&nt)[D2],
                                         const uint32_t* __restrict__ next_row, float esc, float ebias) {
    uint32_t u0 = __builtin_amdgcn_sad_u16(kf[0], t[0], 0u);
    __builtin_amdgcn_sched_barrier(0);
    load_row<D2>(nt, next_row);
    __builtin_amdgcn_sched_barrier(0);
    uint32_t u1 = __builtin_amdgcn_sad_u16(kf[1], t[1], 0u);
#pragma unroll
    for (int c = 2; c < D2; c += 2) {
        u0 = __builtin_amdgcn_sad_u16(kf[c], t[c], u0);
        u1 = __builtin_amdgcn_sad_u16(kf[c + 1], t[c + 1], u1);
    }
    return fmaf(__uint_as_float(u0 + u1 + bias23()), esc, ebias);
}
template <int D2>
__device__ __forceinline__ float lap_row(const uint32_t (&kf)[D2], const uint32_t (&t)[D2], uint32_t (&nt)[D2],
                                         const uint32_t* __restrict__ next_row, float esc, float ebias) {
    return __builtin_amdgcn_exp2f(lap_arg<D2>(kf, t, nt, next_row, esc, ebias));
}

// As lap_arg, with the next row read from LDS (all lanes at one address) into registers: the
// rows of one table alternate between the scalar cache and LDS, so that neither path alone has
// to deliver a row per 32 v_sad_u16 of a wave.
template <int D2>
__device__ __forceinline__ float lap_arg_lds(const uint32_t (&kf)[D2], const uint32_t (&t)[D2], uint32_t (&nt)[D2],
                                             const uint32_t* next_row, float esc, float ebias) {
    uint32_t u0 = __builtin_amdgcn_sad_u16(kf[0], t[0], 0u);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int c4 = 0; c4 < D2 / 4; ++c4) {
        const uint4 r = reinterpret_cast<const uint4*>(next_row)[c4];
        nt[4 * c4] = r.x; nt[4 * c4 + 1] = r.y; nt[4 * c4 + 2] = r.z; nt[4 * c4 + 3] = r.w;
    }
    __builtin_amdgcn_sched_barrier(0);
    uint32_t u1 = __builtin_amdgcn_sad_u16(kf[1], t[1], 0u);
#pragma unroll
    for (int c = 2; c < D2; c += 2) {
        u0 = __builtin_amdgcn_sad_u16(kf[c], t[c], u0);
        u1 = __builtin_amdgcn_sad_u16(kf[c + 1], t[c + 1], u1);
    }
    return fmaf(__uint_as_float(u0 + u1 + bias23()), esc, ebias);
}

// The exp2 arguments of two tokens (x, y) against one landmark row: four sad chains, the loads
// of the next row into `nt` issued after the first sad (the wait point for `t`).  Each row
// fetched through the scalar cache feeds twice the VALU work of lap_arg.
template <int D2>
__device__ __forceinline__ void lap_arg2(const uint32_t (&xf)[D2], const uint32_t (&yf)[D2], const uint32_t (&t)[D2],
                                         uint32_t (&nt)[D2], const uint32_t* __restrict__ next_row, float esc,
                                         float xbias, float ybias, float& gx, float& gy) {
    uint32_t u0 = __builtin_amdgcn_sad_u16(xf[0], t[0], 0u);
    __builtin_amdgcn_sched_barrier(0);
    load_row<D2>(nt, next_row);
    __builtin_amdgcn_sched_barrier(0);
    uint32_t u1 = __builtin_amdgcn_sad_u16(xf[1], t[1], 0u);
    uint32_t v0 = __builtin_amdgcn_sad_u16(yf[0], t[0], 0u);
    uint32_t v1 = __builtin_amdgcn_sad_u16(yf[1], t[1], 0u);
#pragma unroll
    for (int c = 2; c < D2; c += 2) {
        u0 = __builtin_amdgcn_sad_u16(xf[c], t[c], u0);
        u1 = __builtin_amdgcn_sad_u16(xf[c + 1], t[c + 1], u1);
        v0 = __builtin_amdgcn_sad_u16(yf[c], t[c], v0);
        v1 = __builtin_amdgcn_sad_u16(yf[c + 1], t[c + 1], v1);
    }
    const uint32_t b23 = bias23();
    gx = fmaf(__uint_as_float(u0 + u1 + b23), esc, xbias);
    gy = fmaf(__uint_as_float(v0 + v1 + b23), esc, ybias);
}

// ------------------------------------------------------------------------------------------
// Per-head frame and Newton-Schulz solve.  grid (BH), 512 threads (8 waves).
//
// Frame: frame[h][0..7] = {R, 1/(2R), escale = -log2(e) / (lambda S), vscale,
// xscale = -log2(e) / lambda, clamped, rho (written by mfinal_kernel), 0}; R is NaN when Q, K or
// V hold a non-finite value
// (the outputs of that head are then NaN, as the plain computation gives); clamped = 1 when
// some |x| of Q or K exceeds R (the key and query sides then add the excess E(x) of each
// token).  qfix/kfix[h][a][c/2] = u(x_{a,c}) | u(x_{a,c+1}) << 16 for landmarks a < 64 (zero
// rows >= m).  vbar[h] = mean of the values; vscale = 2^e puts the largest |v| of the head in
// [2^13, 2^14), so that the fp16 copies of V (exact for bf16 values in fp16's normal range)
// neither overflow nor fall into fp16's subnormal range for small values.
//
// Solve (Algorithm 2): W = K_LL + eps I padded to 64 x 64 (lane = row a, eight columns b per
// wave, v_sad_u16 against the key-landmark rows read by the whole wave at one LDS address);
// c = ||W||_1 ||W||_inf (first maximising column / row); X0 = W^T / c (0 if c = 0); then the
// T updates X_{t+1} = X_t (2I - W X_t).  The updates satisfy I - W X_t = E^(2^t) with
// E = I - W X0, hence X_{t+1} = X_t (I + E^(2^t)) and
//   X_T = X0 (I + E_0)(I + E_1) ... (I + E_{T-1}),  E_0 = E,  E_{k+1} = E_k E_k,
// the same iterates in exact arithmetic.  The two products of a step -- Z <- Z + Z E_k
// (waves 0-3) and E_{k+1} = E_k E_k (waves 4-7) -- are independent, so a step costs one
// product and one barrier, and the two chains share every SIMD.  Both run on fp16-pair MFMA
// 32x32x16 (A B ~ Ahi Bhi + Ahi Blo + Alo Bhi, ~22 significant bits); Z is accumulated in fp32
// registers.  Only transposed copies are stored (Z^T, E^T), with 8-byte writes straight from the
// MFMA result layout, each alternating between two buffers; the A factors come through
// transposing LDS reads.
// Scales: ||E_k||_2 <= 1 (E's spectrum lies in [0, 1)), so E is stored unscaled.  Z carries a
// power-of-two scale: Z_0's from its exact maximum (largest entry in [2^14, 2^15)), Z_{k+1}'s
// from the maximum of Z_k, placing that maximum in [2^7, 2^8); ||I + E_k||_2 <= 2 bounds the
// growth of the largest entry by 2 * 64 = 2^7 per step, so stored values stay below 2^15.
//   Writes X_T (fp32, row-major [64][64]) and cinfo = {c, n1, ninf, a* 256 + b*}.
constexpr int kSolveLds = 8 * 64 * kLP * 2 + 64 * 4;
constexpr int kSolveThreads = 512;

// One DPP step of wave_argmax_dpp: keep the larger (value bits, 63 - lane) key.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ void argmax_step(int& hi, int& lo) {
    const int h2 = __builtin_amdgcn_update_dpp(0, hi, CTRL, ROW_MASK, 0xF, false);
    const int l2 = __builtin_amdgcn_update_dpp(0, lo, CTRL, ROW_MASK, 0xF, false);
    if (h2 > hi || (h2 == hi && l2 > lo)) {
        hi = h2;
        lo = l2;
    }
}

// Maximum of a non-negative v over the wave and the lowest lane holding it, by DPP on
// (value bits, 63 - lane): a larger key is a larger value or, on a tie, a lower lane.  The
// result is wave-uniform.
__device__ __forceinline__ void wave_argmax_dpp(float& v, int& idx) {
    int hi = __float_as_int(v), lo = 63 - (int)(threadIdx.x & 63);
    argmax_step<0xB1, 0xF>(hi, lo);    // quad_perm [1,0,3,2]
    argmax_step<0x4E, 0xF>(hi, lo);    // quad_perm [2,3,0,1]
    argmax_step<0x141, 0xF>(hi, lo);   // row_half_mirror
    argmax_step<0x140, 0xF>(hi, lo);   // row_mirror
    argmax_step<0x142, 0xA>(hi, lo);   // row_bcast:15
    argmax_step<0x143, 0xC>(hi, lo);   // row_bcast:31
    v = __int_as_float(__builtin_amdgcn_readlane(hi, 63));
    idx = 63 - __builtin_amdgcn_readlane(lo, 63);
}

// SOLVE = false: the frame and the code tables only (the solve then runs beside the key side,
// ns_role in key2_kernel, whose key blocks also form the value statistics: vseg, vsegmax, vbar
// and vscale are then neither read nor written, and R reflects Q and K only).
template <int D, bool SOLVE>
__global__ __launch_bounds__(kSolveThreads) void frame_ns_kernel(
    const float* __restrict__ qt, const float* __restrict__ kt, const double* __restrict__ vseg,
    const float* __restrict__ segmax, const float* __restrict__ vsegmax, float* __restrict__ frame,
    uint32_t* __restrict__ qfix, uint32_t* __restrict__ kfix, float* __restrict__ vbar, float* __restrict__ XT,
    float* __restrict__ cinfo, int n, int m, float lambda, int T, float eps) {
    constexpr int NT = kSolveThreads;
    constexpr int NW = NT / 64;          // 8 waves
    constexpr int D2 = D / 2;
    constexpr int WPT = 64 * D2 / NT;    // table words per thread (4 at d = 64, 2 at d = 32)
    constexpr int G = NT / D;            // landmark groups of the value-mean partial sums
    constexpr int LPG = 64 / G;          // landmarks per group
    constexpr int BPW = 64 / NW;         // columns b of W per wave
    constexpr int WP = 68;               // fp32 pitch of the set-up copy of W
    __shared__ __attribute__((aligned(16))) char lds[kSolveLds];
    const int h = blockIdx.x, tid = threadIdx.x, w = tid >> 6, l = tid & 63;
    _Float16* base = reinterpret_cast<_Float16*>(lds);
    // transposed copies, two buffers each: Z^T (ZTh/ZTl(k & 1)) and E^T (ETh/ETl(k & 1)).
    // Offsets from the LDS base, not an array of pointers: a pointer picked from a local array
    // by a run-time index loses its address space and would be accessed with flat loads.
    constexpr int TB = 64 * kLP;
    auto ZTh = [&](int i) { return base + (2 * i) * TB; };
    auto ZTl = [&](int i) { return base + (2 * i + 1) * TB; };
    auto ETh = [&](int i) { return base + (4 + 2 * i) * TB; };
    auto ETl = [&](int i) { return base + (5 + 2 * i) * TB; };
    float* sred = reinterpret_cast<float*>(base + 8 * 64 * kLP);   // 64 floats
    // set-up aliases, each dead before the first write to its buffer: the landmark tables in
    // Z^T[1]; the norm partials and the value partials in E^T[0]; W in fp32 in E^T[1] (read
    // until the barrier after E_0, which precedes the first write of E^T[1])
    uint32_t* sQ = reinterpret_cast<uint32_t*>(ZTh(1));
    uint32_t* sK = sQ + 64 * D2;
    float* part = reinterpret_cast<float*>(ETh(0));          // 2 x NW x 64 floats
    double* vpart = reinterpret_cast<double*>(ETh(0)) + 512;  // G x D doubles, after part
    float* sWf = reinterpret_cast<float*>(ETh(1));
    static_assert(2 * 64 * D2 * 4 <= 2 * 64 * kLP * 2, "landmark tables exceed Z^T[1]");
    static_assert(2 * NW * 64 * 4 <= 512 * 8 && 512 * 8 + G * D * 8 <= 2 * 64 * kLP * 2, "partials exceed E^T[0]");
    static_assert(64 * WP * 4 <= 2 * 64 * kLP * 2, "fp32 W exceeds E^T[1]");
    static_assert(G * D == NT && G * LPG == 64, "value partials");

    // ---- frame: every global read first
    float q0[WPT], q1[WPT], k0[WPT], k1[WPT];
#pragma unroll
    for (int r = 0; r < WPT; ++r) {
        const int e = tid + NT * r, a = e / D2, c2 = e % D2;
        const size_t o = ((size_t)h * m + (a < m ? a : 0)) * D + 2 * c2;
        q0[r] = qt[o]; q1[r] = qt[o + 1]; k0[r] = kt[o]; k1[r] = kt[o + 1];
    }
    double vs = 0.0;
    if (SOLVE) {
        // all loads issued before the first add (landmarks past m read row 0 and are dropped)
        const int c = tid % D, g = tid / D;
        double vv[LPG];
#pragma unroll
        for (int i = 0; i < LPG; ++i) {
            const int lm = g * LPG + i;
            vv[i] = vseg[((size_t)h * m + (lm < m ? lm : 0)) * D + c];
        }
#pragma unroll
        for (int i = 0; i < LPG; ++i) vs += g * LPG + i < m ? vv[i] : 0.0;
    }
    const int tm = tid < m ? tid : 0;
    float sa = segmax[(size_t)h * m + tm], sb = SOLVE ? vsegmax[(size_t)h * m + tm] : 0.f;
    if (tid >= m) sa = sb = 0.f;
    vpart[tid] = vs;   // [g][c]
    {
        // largest landmark coordinate (rows past m were loaded from row 0 and are left out)
        float lmx = 0.f;
#pragma unroll
        for (int r = 0; r < WPT; ++r)
            if ((tid + NT * r) / D2 < m)
                lmx = fmaxf(lmx, fmaxf(fmaxf(fabsf(q0[r]), fabsf(q1[r])), fmaxf(fabsf(k0[r]), fabsf(k1[r]))));
        lmx = wave_max_dpp(lmx);
        if (l == 0) sred[48 + w] = lmx;
    }
    __syncthreads();
    if (w == 0) {
        const bool bad = __any(!(isfinite(sa) && isfinite(sb)));
        const float xmax = wave_max_dpp(sa);
        const float vm = wave_max_dpp(sb);
        // median of the landmarks' token maxima (lane l < m holds landmark l's): the value of
        // rank (m - 1) / 2, ties ranked by landmark index (landmark j's value read as a scalar)
        int rank = 0;
        for (int j = 0; j < m; ++j) {
            const float sj = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(sa), j));
            rank += (sj < sa || (sj == sa && j < l)) ? 1 : 0;
        }
        const unsigned long long pick = __ballot(l < m && rank == (m - 1) / 2);
        const float med = pick ? __int_as_float(__builtin_amdgcn_readlane(__float_as_int(sa), (int)__builtin_ctzll(pick)))
                               : xmax;   // none: a NaN maximum
        float lmax = sred[48];
#pragma unroll
        for (int i = 1; i < NW; ++i) lmax = fmaxf(lmax, sred[48 + i]);
        if (l == 0) {
            float R = fmaxf(lmax, fminf(xmax, 2.f * med));
            if (!(R > 0.f)) R = 1.f;
            const float S = (float)(65535.0 / (2.0 * (double)R));
            const float vscale = (vm > 0.f && isfinite(vm)) ? ldexpf(1.f, 13 - ilogbf(vm)) : 1.f;
            const float inv2R = (float)(0.5 / (double)R);
            const float escale = (float)(-1.4426950408889634 / ((double)lambda * (double)S));
            frame[h * 8 + 0] = bad ? __builtin_nanf("") : R;
            frame[h * 8 + 1] = inv2R;
            frame[h * 8 + 2] = escale;
            frame[h * 8 + 3] = vscale;
            frame[h * 8 + 4] = (float)(-1.4426950408889634 / (double)lambda);
            frame[h * 8 + 5] = xmax > R ? 1.f : 0.f;
            frame[h * 8 + 7] = 0.f;
            sred[0] = inv2R;
            sred[1] = escale;
        }
    }
    __syncthreads();
    if (SOLVE && tid < D) {
        double t = 0.0;
#pragma unroll
        for (int g = 0; g < G; ++g) t += vpart[g * D + tid];
        vbar[(size_t)h * D + tid] = (float)(t / n);
    }
    const float inv2R = sred[0], esc = sred[1];
    const float ebias = -kTwo23 * esc;
    uint32_t* qtab = qfix + (size_t)h * 64 * D2;
    uint32_t* ktab = kfix + (size_t)h * 64 * D2;
#pragma unroll
    for (int r = 0; r < WPT; ++r) {
        const int e = tid + NT * r, a = e / D2;
        const uint32_t uq = a < m ? fix2(q0[r], q1[r], inv2R) : 0u;
        const uint32_t uk = a < m ? fix2(k0[r], k1[r], inv2R) : 0u;
        qtab[e] = uq;
        ktab[e] = uk;
        sQ[e] = uq;
        sK[e] = uk;
    }
    if (!SOLVE) return;
    __syncthreads();
    // ---- W[a][b] = k(qt_a, kt_b) (+ eps on the diagonal): lane a, columns b = BPW w..+BPW
    uint32_t qa[D2];
#pragma unroll
    for (int c4 = 0; c4 < D2 / 4; ++c4) {
        const uint4 x = reinterpret_cast<const uint4*>(sQ + l * D2)[c4];
        qa[4 * c4] = x.x; qa[4 * c4 + 1] = x.y; qa[4 * c4 + 2] = x.z; qa[4 * c4 + 3] = x.w;
    }
    // the key-landmark rows b are read by the whole wave at one address (LDS broadcast), two
    // rows' reads in flight at a time (fully unrolled: wv stays in registers)
    float wv[BPW];
    const uint4* krow = reinterpret_cast<const uint4*>(sK + BPW * w * D2);
#pragma unroll
    for (int bb = 0; bb < BPW; bb += 2) {
        uint4 t0[D2 / 4], t1[D2 / 4];
#pragma unroll
        for (int c4 = 0; c4 < D2 / 4; ++c4) {
            t0[c4] = krow[bb * (D2 / 4) + c4];
            t1[c4] = krow[(bb + 1) * (D2 / 4) + c4];
        }
        uint32_t u0 = 0x4B000000u, u1 = 0u, v0 = 0x4B000000u, v1 = 0u;
#pragma unroll
        for (int c4 = 0; c4 < D2 / 4; ++c4) {
            u0 = __builtin_amdgcn_sad_u16(qa[4 * c4 + 0], t0[c4].x, u0);
            u1 = __builtin_amdgcn_sad_u16(qa[4 * c4 + 1], t0[c4].y, u1);
            v0 = __builtin_amdgcn_sad_u16(qa[4 * c4 + 0], t1[c4].x, v0);
            v1 = __builtin_amdgcn_sad_u16(qa[4 * c4 + 1], t1[c4].y, v1);
            u0 = __builtin_amdgcn_sad_u16(qa[4 * c4 + 2], t0[c4].z, u0);
            u1 = __builtin_amdgcn_sad_u16(qa[4 * c4 + 3], t0[c4].w, u1);
            v0 = __builtin_amdgcn_sad_u16(qa[4 * c4 + 2], t1[c4].z, v0);
            v1 = __builtin_amdgcn_sad_u16(qa[4 * c4 + 3], t1[c4].w, v1);
        }
        wv[bb] = __builtin_amdgcn_exp2f(fmaf(__uint_as_float(u0 + u1), esc, ebias));
        wv[bb + 1] = __builtin_amdgcn_exp2f(fmaf(__uint_as_float(v0 + v1), esc, ebias));
    }
#pragma unroll
    for (int bb = 0; bb < BPW; ++bb) {
        const int b = BPW * w + bb;
        if (l == b) wv[bb] += eps;
        wv[bb] = (l < m && b < m) ? wv[bb] : 0.f;
    }
    // row partial sums from registers, W (fp32) to LDS for the column partial sums
    float rsum = 0.f, wmax = 0.f;
#pragma unroll
    for (int bb = 0; bb < BPW; ++bb) {
        rsum += fabsf(wv[bb]);
        wmax = fmaxf(wmax, fabsf(wv[bb]));
    }
#pragma unroll
    for (int q = 0; q < BPW / 4; ++q)
        *reinterpret_cast<float4*>(sWf + l * WP + BPW * w + 4 * q) =
            make_float4(wv[4 * q], wv[4 * q + 1], wv[4 * q + 2], wv[4 * q + 3]);
    wmax = wave_max_dpp(wmax);
    if (l == 0) sred[16 + w] = wmax;
    __syncthreads();
    {
        float csum = 0.f;   // column l, rows BPW w..+BPW
#pragma unroll
        for (int i = 0; i < BPW; ++i) csum += fabsf(sWf[(BPW * w + i) * WP + l]);
        part[w * 64 + l] = csum;
        part[NW * 64 + w * 64 + l] = rsum;   // row l, columns BPW w..+BPW
    }
    __syncthreads();
    if (w == 0) {
        // column and row sums in a fixed order, then the first maximising column / row
        float n1 = 0.f, ninf = 0.f, mx = 0.f;
#pragma unroll
        for (int g = 0; g < NW; ++g) {
            n1 += part[g * 64 + l];
            ninf += part[NW * 64 + g * 64 + l];
            mx = fmaxf(mx, sred[16 + g]);
        }
        int bs, as;
        wave_argmax_dpp(n1, bs);
        wave_argmax_dpp(ninf, as);
        if (l == 0) {
            const float c = n1 * ninf;
            sred[2] = c;
            sred[3] = mx;
            cinfo[h * 4 + 0] = c;
            cinfo[h * 4 + 1] = n1;
            cinfo[h * 4 + 2] = ninf;
            cinfo[h * 4 + 3] = (float)(as * 256 + bs);
        }
    }
    __syncthreads();
    const float c = sred[2];
    const float inv_c = c > 0.f ? 1.f / c : 0.f;
    float mx = sred[3] * inv_c;             // max |X0| = max |Z_0|
    float zs = ldexpf(1.f, pow2_exp(mx));   // Z_true = Z_stored * zs
    // Z_0^T = X0^T = W / c: BPW consecutive b of row a
    {
        const float x0s = inv_c / zs;
        uint32_t xh[BPW / 2], xl[BPW / 2];
#pragma unroll
        for (int q = 0; q < BPW / 2; ++q) split_pk(wv[2 * q] * x0s, wv[2 * q + 1] * x0s, xh[q], xl[q]);
        const int o = l * kLP + BPW * w;
#pragma unroll
        for (int q = 0; q < BPW / 8; ++q) {
            *reinterpret_cast<uint4*>(ZTh(0) + o + 8 * q) = make_uint4(xh[4 * q], xh[4 * q + 1], xh[4 * q + 2], xh[4 * q + 3]);
            *reinterpret_cast<uint4*>(ZTl(0) + o + 8 * q) = make_uint4(xl[4 * q], xl[4 * q + 1], xl[4 * q + 2], xl[4 * q + 3]);
        }
        if (T == 0) {
#pragma unroll
            for (int bb = 0; bb < BPW; ++bb) XT[(size_t)h * 4096 + (BPW * w + bb) * 64 + l] = wv[bb] * inv_c;
        }
    }
    __syncthreads();
    if (T == 0) return;
    // waves 0-3: the Z chain; waves 4-7: the E chain; block (rb, cb) = ((w & 3) / 2, w & 1)
    const bool zchain = w < 4;
    const int rb = (w & 3) >> 1, cb = w & 1;
    f32x16_t zreg;   // Z chain: this wave's block of Z_k (true values, fp32)
    if (zchain) {
        // Z_0 = X0: X0[row][col] = W[col][row] / c
#pragma unroll
        for (int r = 0; r < 16; ++r) zreg[r] = sWf[(32 * cb + (l & 31)) * WP + 32 * rb + c_row(r, l)] * inv_c;
    } else {
        // E_0 = I - W X0 (A = W from the fp32 copy, B = X0 through Z^T[0])
        h8_t wah[4], wal[4];
#pragma unroll
        for (int s4 = 0; s4 < 4; ++s4) {
            const float* src = sWf + (32 * rb + (l & 31)) * WP + 16 * s4 + 8 * (l >> 5);
            uint32_t hq[4], lq[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) split_pk(src[2 * q], src[2 * q + 1], hq[q], lq[q]);
            wah[s4] = __builtin_bit_cast(h8_t, make_uint4(hq[0], hq[1], hq[2], hq[3]));
            wal[s4] = __builtin_bit_cast(h8_t, make_uint4(lq[0], lq[1], lq[2], lq[3]));
        }
        f32x16_t e0 = mm32_split(wah, wal, ZTh(0), ZTl(0), cb);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int row = 32 * rb + c_row(r, l), col = 32 * cb + (l & 31);
            e0[r] = (row == col ? 1.f : 0.f) - e0[r] * zs;
        }
        store32_t(e0, 1.f, rb, cb, ETh(0), ETl(0));
    }
    __syncthreads();
    for (int k = 0; k < T; ++k) {
        const int cur = k & 1;
        if (zchain) {
            // Z_{k+1} = Z_k + Z_k E_k
            h8_t zah[4], zal[4];
#pragma unroll
            for (int s4 = 0; s4 < 4; ++s4) {
                zah[s4] = a_from_transposed(ZTh(cur), rb, 16 * s4);
                zal[s4] = a_from_transposed(ZTl(cur), rb, 16 * s4);
            }
            const f32x16_t d = mm32_split(zah, zal, ETh(cur), ETl(cur), cb);
#pragma unroll
            for (int r = 0; r < 16; ++r) zreg[r] = fmaf(d[r], zs, zreg[r]);
            if (k + 1 < T) {
                // scale of Z_{k+1} from the maximum of Z_k (mx)
                zs = ldexpf(1.f, (mx > 0.f && isfinite(mx)) ? ilogbf(mx) - 7 : 0);
                store32_t(zreg, 1.f / zs, rb, cb, ZTh(cur ^ 1), ZTl(cur ^ 1));
                float lm = 0.f;
#pragma unroll
                for (int r = 0; r < 16; ++r) lm = fmaxf(lm, fabsf(zreg[r]));
                lm = wave_max_dpp(lm);
                if (l == 0) sred[32 + 4 * cur + w] = lm;
            } else {
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    XT[(size_t)h * 4096 + (32 * rb + c_row(r, l)) * 64 + 32 * cb + (l & 31)] = zreg[r];
            }
        } else if (k + 1 < T) {
            // E_{k+1} = E_k E_k
            h8_t eah[4], eal[4];
#pragma unroll
            for (int s4 = 0; s4 < 4; ++s4) {
                eah[s4] = a_from_transposed(ETh(cur), rb, 16 * s4);
                eal[s4] = a_from_transposed(ETl(cur), rb, 16 * s4);
            }
            const f32x16_t e = mm32_split(eah, eal, ETh(cur), ETl(cur), cb);
            store32_t(e, 1.f, rb, cb, ETh(cur ^ 1), ETl(cur ^ 1));
        }
        if (k + 1 < T) {
            __syncthreads();
            mx = fmaxf(fmaxf(sred[32 + 4 * cur], sred[33 + 4 * cur]), fmaxf(sred[34 + 4 * cur], sred[35 + 4 * cur]));
        }
    }
}

// ------------------------------------------------------------------------------------------
// Key-summary role: block kb of head h covers keys [kb*kpb, min(n, (kb+1)*kpb)) in steps of
// 256 keys, one 64-key tile per wave (lane = key).  Per step, each wave: u(k_j) in registers,
// the m kernel values exp(-||qt_a - k_j||_1/lambda) from v_sad_u16 against the landmark table
// into its LDS tile as [a][j], its value rows to fp16, transposed, into LDS as [c][j]; then,
// after a block barrier, U[a][c] += sum_j B[a][j] V[j][c] over the block's 256 keys on fp16
// MFMA 16x16x32, wave w forming the rows a in [16w, 16w + 16) for every value column and the
// ones column.  The raw rows of the next step are loaded while the current one is computed.
//
// The landmark rows are wave-uniform and come through scalar registers, one row per step in
// two alternating buffers: the scalar loads of row a+1 are issued right after the first use
// of row a (which is the point where the wave waits for row a), so each row's load has a
// whole step of 32 v_sad_u16 to arrive.  Scalar loads complete out of order, so the wait
// cannot be narrowed to one of several outstanding rows; issuing after the wait keeps exactly
// one row in flight.
constexpr int kKeyTileLds = 4 * 2 * 64 * kLP * 2;   // four waves' [a][j] and [c][j] fp16 tiles

typedef float f32x4_t __attribute__((ext_vector_type(4)));

// Writes Upart[h][kb][c][a] (a < 64; rows >= m finite, multiplied by zero columns of X_T).
template <int D>
__device__ void key_role(int h, int kb, char* lds_raw, const uint16_t* __restrict__ K,
                         const uint16_t* __restrict__ V, const uint32_t* __restrict__ qfix,
                         const float* __restrict__ frame, float* __restrict__ Upart, int n, int m, int kpb, int nkb) {
    constexpr int D2 = D / 2;
    constexpr int D8 = D / 8;
    constexpr int C16 = D / 16;   // value column blocks of the 16 x 16 products
    const int tid = threadIdx.x, w = tid >> 6, l = tid & 63;
    _Float16* const tiles = reinterpret_cast<_Float16*>(lds_raw);
    _Float16* sB = tiles + w * (2 * 64 * kLP);   // this wave's [a][j]
    _Float16* sV = sB + 64 * kLP;                 // this wave's [c][j]
    const float inv2R = frame[h * 8 + 1], esc = frame[h * 8 + 2], vsc = frame[h * 8 + 3];
    const float R = frame[h * 8 + 0], xsc = frame[h * 8 + 4];
    const bool clamped = __float_as_uint(frame[h * 8 + 5]) != 0u;   // integer test: a scalar branch
    const uint32_t* tab = qfix + (size_t)h * 64 * D2;
    const float ebias = -kTwo23 * esc;
    const int j_begin = kb * kpb, j_end = min(n, j_begin + kpb);
    const int ntiles = (j_end - j_begin + 63) / 64;
    const int nsteps = (ntiles + 3) / 4;
    const int mp = (m + 1) & ~1;   // landmark rows written per tile (an odd m writes one zero row)
    const bool rows_live = 16 * w < m;   // this wave's rows of U are not all zero
    f32x4_t acc[C16 + 1];
#pragma unroll
    for (int cc = 0; cc <= C16; ++cc) acc[cc] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
    h8_t ones;   // B operand of the ones column: 1 in column 0
#pragma unroll
    for (int i = 0; i < 8; ++i) ones[i] = (l & 15) == 0 ? (_Float16)1.f : (_Float16)0.f;
    for (int a = mp; a < 64; ++a) sB[a * kLP + l] = (_Float16)0.f;   // rows a >= m stay zero

    // rows of keys past the end keep stale values: their kernel values and value pairs are
    // masked to zero below
    uint4 kr[D8] = {}, vr[D8] = {};
    auto row_ptrs = [&](int tile, const uint4*& kp, const uint4*& vp) {
        const int j = j_begin + tile * 64 + l;
        const bool ok = tile < ntiles && j < j_end;
        kp = ok ? reinterpret_cast<const uint4*>(K + ((size_t)h * n + j) * D) : nullptr;
        vp = ok ? reinterpret_cast<const uint4*>(V + ((size_t)h * n + j) * D) : nullptr;
    };
    {
        // the first tile: keys first (the landmark loop needs them), values behind them
        const uint4 *kp, *vp;
        row_ptrs(w, kp, vp);
        if (kp) {
#pragma unroll
            for (int c8 = 0; c8 < D8; ++c8) kr[c8] = kp[c8];
#pragma unroll
            for (int c8 = 0; c8 < D8; ++c8) vr[c8] = vp[c8];
        }
    }
    // Each wave walks the landmark rows from its own starting pair, so that the waves sharing
    // a CU (and its scalar cache) fetch different rows of the table at first instead of all
    // waiting on the same row.  The order only decides which row of the B tile is written
    // when, not the result.
    const int npairs = (m + 1) >> 1;
    const int rot = ((__builtin_amdgcn_readfirstlane(w) + 4 * (int)(blockIdx.x & 1)) * npairs) >> 3;
    for (int step = 0; step < nsteps; ++step) {
        const int tile = 4 * step + w;
        if (tile < ntiles) {
            // keys past the end of the chunk have zero rows; their kernel values are masked to 0
            const uint32_t vmask = j_begin + tile * 64 + l < j_end ? 0xffffffffu : 0u;
            uint32_t kf[D2];
#pragma unroll
            for (int c8 = 0; c8 < D8; ++c8) {
                kf[4 * c8 + 0] = fix2_bf16(kr[c8].x, inv2R);
                kf[4 * c8 + 1] = fix2_bf16(kr[c8].y, inv2R);
                kf[4 * c8 + 2] = fix2_bf16(kr[c8].z, inv2R);
                kf[4 * c8 + 3] = fix2_bf16(kr[c8].w, inv2R);
            }
            // keys past the end of the chunk: exponent bias -inf, kernel values exactly 0 (their
            // value registers hold finite values of this head, so the products stay 0)
            float kbias = vmask ? ebias : -__builtin_inff();
            if (clamped) {
                // a head with tokens beyond the range: the key's excess enters the exponent
                float ex = 0.f;
#pragma unroll
                for (int c8 = 0; c8 < D8; ++c8) {
                    const uint32_t wd[4] = {kr[c8].x, kr[c8].y, kr[c8].z, kr[c8].w};
#pragma unroll
                    for (int t = 0; t < 4; ++t)
                        ex += fmaxf(fabsf(bf16_lo(wd[t])), R) + fmaxf(fabsf(bf16_hi(wd[t])), R);
                }
                kbias = vmask ? fmaf(ex - (float)D * R, xsc, ebias) : -__builtin_inff();
            }
            // The next tile's keys are fetched in D/8 column groups spread over the landmark
            // loop, so that the key stream reaches memory as a steady flow rather than one
            // burst per tile from every wave at once; its values follow after this tile's
            // values have been moved to LDS.
            const uint4 *kp, *vp;
            row_ptrs(tile + 4, kp, vp);
            // landmark pairs (2p, 2p+1): rows 2p, 2p+1 of the [a][j] tile; table rows >= m are
            // zero codes, so the value of a landmark m (odd m) is finite, and row m of U is
            // dropped by the zero column m of X_T
            uint16_t* brow = reinterpret_cast<uint16_t*>(sB) + l;
            uint32_t ta[D2], tb[D2];
            load_row<D2>(ta, tab + (2 * rot) * D2);
            int p = rot;
#pragma unroll
            for (int c8 = 0; c8 < D8; ++c8) {
                if (kp) kr[c8] = kp[c8];
#pragma unroll 1
                for (int i = c8 * npairs / D8; i < (c8 + 1) * npairs / D8; ++i) {
                    const int pn = p + 1 < npairs ? p + 1 : 0;
                    const float b0 = lap_row<D2>(kf, ta, tb, tab + (2 * p + 1) * D2, esc, kbias);
                    const float b1 = lap_row<D2>(kf, tb, ta, tab + (2 * pn) * D2, esc, kbias);
                    const uint32_t v = pk_f16(b0, b1);
                    uint16_t* r2 = brow + (2 * p) * kLP;
                    r2[0] = (uint16_t)(v & 0xffffu);
                    r2[kLP] = (uint16_t)(v >> 16);
                    p = pn;
                }
            }
            // this tile's values to fp16 (times the value prescale), transposed into LDS
#pragma unroll
            for (int c8 = 0; c8 < D8; ++c8) {
                const uint32_t yw[4] = {vr[c8].x, vr[c8].y, vr[c8].z, vr[c8].w};
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    const uint32_t pv = pk_f16(bf16_lo(yw[t]) * vsc, bf16_hi(yw[t]) * vsc);
                    reinterpret_cast<uint16_t*>(sV)[(8 * c8 + 2 * t) * kLP + l] = (uint16_t)(pv & 0xffffu);
                    reinterpret_cast<uint16_t*>(sV)[(8 * c8 + 2 * t + 1) * kLP + l] = (uint16_t)(pv >> 16);
                }
            }
            if (vp) {
#pragma unroll
                for (int c8 = 0; c8 < D8; ++c8) vr[c8] = vp[c8];
            }
        }
        __syncthreads();   // the step's tiles are complete
        // U rows [16w, 16w + 16) over the step's tiles, 32 keys per product: A = B[a][j]
        // (A[l%16][8(l/16) + i]), B = V[j][c] through the transposed tile ([c][j]).
        const int live = min(4, ntiles - 4 * step);
        if (rows_live) {
            const int ao = (16 * w + (l & 15)) * kLP + 8 * (l >> 4);
            const int bo = (l & 15) * kLP + 8 * (l >> 4);
            for (int t = 0; t < live; ++t) {
                const _Float16* tB = tiles + t * (2 * 64 * kLP);
                const _Float16* tV = tB + 64 * kLP;
#pragma unroll
                for (int half = 0; half < 2; ++half) {
                    const h8_t A = *reinterpret_cast<const h8_t*>(tB + ao + 32 * half);
#pragma unroll
                    for (int cc = 0; cc < C16; ++cc) {
                        const h8_t Bv = *reinterpret_cast<const h8_t*>(tV + 16 * cc * kLP + bo + 32 * half);
                        acc[cc] = __builtin_amdgcn_mfma_f32_16x16x32_f16(A, Bv, acc[cc], 0, 0, 0);
                    }
                    acc[C16] = __builtin_amdgcn_mfma_f32_16x16x32_f16(A, ones, acc[C16], 0, 0, 0);
                }
            }
        }
        __syncthreads();   // the tiles are rewritten by the next step
    }
    // rows a = 16w + 4(l/16) + r, column 16cc + l%16 (the value columns were formed from
    // V * vscale); the ones column from column 0 of its block
    const float inv_vsc = 1.f / vsc;
    float* dst = Upart + ((size_t)h * nkb + kb) * (D + 1) * 64;
#pragma unroll
    for (int cc = 0; cc < C16; ++cc)
#pragma unroll
        for (int r = 0; r < 4; ++r) dst[(16 * cc + (l & 15)) * 64 + 16 * w + 4 * (l >> 4) + r] = acc[cc][r] * inv_vsc;
    if ((l & 15) == 0) {
#pragma unroll
        for (int r = 0; r < 4; ++r) dst[D * 64 + 16 * w + 4 * (l >> 4) + r] = acc[C16][r];
    }
}

// ------------------------------------------------------------------------------------------
// Key-side partial sums: blocks [0, BH*nkb), one key chunk each.
constexpr int kKeyLds = kKeyTileLds;

template <int D>
__global__ __launch_bounds__(256, 2) void key_kernel(const uint16_t* __restrict__ K, const uint16_t* __restrict__ V,
                                                     const uint32_t* __restrict__ qfix,
                                                     const float* __restrict__ frame, float* __restrict__ Upart,
                                                     int BH, int n, int m, int kpb, int nkb) {
    __shared__ __attribute__((aligned(16))) char lds[kKeyLds];
    const int b = blockIdx.x, nkey = BH * nkb;
    int kbb = xcd_rank(b, nkey, 0);
    if ((nkey & 255) == 0) {
        // When the key blocks fill whole rounds of the 8 x 32 CUs, the blocks of one XCD that
        // would share a CU (its 32 CUs take local blocks i, i + 32, ...) get adjacent key
        // chunks of one head, so a CU's scalar cache holds one landmark table.
        const int per = nkey >> 3, R = nkey >> 8, i = kbb % per;
        kbb = kbb - i + (i & 31) * R + (i >> 5);
    }
    key_role<D>(kbb / nkb, kbb % nkb, lds, K, V, qfix, frame, Upart, n, m, kpb, nkb);
}

// ------------------------------------------------------------------------------------------
// Newton-Schulz of one head by the four waves of a key2_kernel block (m > 48), so that the solve
// runs beside the key side instead of before it: the same computation as frame_ns_kernel's
// solve (W from the landmark code tables, c, X0 = W^T / c, the T updates in product form,
// fp16-pair MFMA 32x32x16, ns_iterate_split), with each wave owning the 32 x 32 block
// (rb, cb) = (w / 2, w % 2) of both chains, and the transposed copies of Z and E in one buffer
// each (a second barrier per step instead of a second buffer) to fit the key blocks' LDS:
// kNsRoleLds bytes.
constexpr int kNsRoleLds = kNsSplitLds + 2 * 4 * 64 * 4 + 64 * 4;

template <int D>
__device__ void ns_role(int h, char* lds, const uint32_t* __restrict__ qfix, const uint32_t* __restrict__ kfix,
                        float* __restrict__ frame, float* __restrict__ XT, float* __restrict__ cinfo,
                        uint32_t* __restrict__ kcen, int m, int T, float eps) {
    constexpr int NW = 4;
    constexpr int D2 = D / 2;
    constexpr int BPW = 64 / NW;   // columns b of W per wave
    constexpr int WP = kWP;        // fp32 pitch of the set-up copy of W
    constexpr int TB = 64 * kLP;
    // lds: the iteration's Z^T and E^T (kNsSplitLds bytes), then the partial sums
    _Float16* const ETh = reinterpret_cast<_Float16*>(lds) + 2 * TB;
    float* const part = reinterpret_cast<float*>(lds + kNsSplitLds);   // 2 x NW x 64
    float* const sred = part + 2 * NW * 64;                        // 64
    // set-up aliases in the E^T region, each dead before its successor is written: the code
    // tables, then W in fp32 (read until the barrier that precedes the first store of E^T)
    uint32_t* const sQ = reinterpret_cast<uint32_t*>(ETh);
    uint32_t* const sK = sQ + 64 * D2;
    float* const sWf = reinterpret_cast<float*>(ETh);
    static_assert(2 * 64 * D2 * 4 <= 2 * TB * 2 && 64 * WP * 4 <= 2 * TB * 2, "set-up copies exceed E^T");
    const int tid = threadIdx.x, w = tid >> 6, l = tid & 63;
    const float esc = frame[h * 8 + 2];
    const float ebias = -kTwo23 * esc;
    {
        constexpr int NE = 64 * D2 / 256;
        uint32_t a[NE], b[NE];   // every load issued before the first LDS write
#pragma unroll
        for (int r = 0; r < NE; ++r) {
            a[r] = qfix[(size_t)h * 64 * D2 + tid + 256 * r];
            b[r] = kfix[(size_t)h * 64 * D2 + tid + 256 * r];
        }
#pragma unroll
        for (int r = 0; r < NE; ++r) {
            sQ[tid + 256 * r] = a[r];
            sK[tid + 256 * r] = b[r];
        }
    }
    __syncthreads();
    // ---- the query side's row bound from the key-landmark codes (rows >= m of the table are
    // zero): kcen[h][c/2] = their centre (per coordinate, the rounded mean over the m landmarks)
    // and frame[h][6] = rho = max_l sum_c |u(kt_{l,c}) - centre_c| (code units); by the triangle
    // inequality every query's code distance to landmark l is at least its distance to the
    // centre minus rho.
    uint32_t* const scen = reinterpret_cast<uint32_t*>(part);   // D2 words, dead before the norms
    if (tid < D2) {
        uint32_t slo = 0, shi = 0;
#pragma unroll 16
        for (int a = 0; a < 64; ++a) {
            const uint32_t u = sK[a * D2 + tid];
            slo += u & 0xffffu;
            shi += u >> 16;
        }
        const uint32_t cen = ((slo + m / 2) / m) | (((shi + m / 2) / m) << 16);
        scen[tid] = cen;
        kcen[(size_t)h * D2 + tid] = cen;
    }
    __syncthreads();
    if (w == 0) {
        uint32_t dist = 0;
        if (l < m) {
#pragma unroll
            for (int c2 = 0; c2 < D2; ++c2) dist = __builtin_amdgcn_sad_u16(sK[l * D2 + c2], scen[c2], dist);
        }
        const float rho = (float)__float_as_uint(wave_max_dpp(__uint_as_float(dist)));
        if (l == 0) frame[h * 8 + 6] = rho;
    }
    // ---- W[a][b] = k(qt_a, kt_b) (+ eps on the diagonal): lane a, columns b = BPW w..+BPW
    uint32_t qa[D2];
#pragma unroll
    for (int c4 = 0; c4 < D2 / 4; ++c4) {
        const uint4 x = reinterpret_cast<const uint4*>(sQ + l * D2)[c4];
        qa[4 * c4] = x.x; qa[4 * c4 + 1] = x.y; qa[4 * c4 + 2] = x.z; qa[4 * c4 + 3] = x.w;
    }
    float wv[BPW];
    const uint4* krow = reinterpret_cast<const uint4*>(sK + BPW * w * D2);
#pragma unroll
    for (int bb = 0; bb < BPW; bb += 2) {
        uint4 t0[D2 / 4], t1[D2 / 4];
#pragma unroll
        for (int c4 = 0; c4 < D2 / 4; ++c4) {
            t0[c4] = krow[bb * (D2 / 4) + c4];
            t1[c4] = krow[(bb + 1) * (D2 / 4) + c4];
        }
        uint32_t u0 = 0x4B000000u, u1 = 0u, v0 = 0x4B000000u, v1 = 0u;
#pragma unroll
        for (int c4 = 0; c4 < D2 / 4; ++c4) {
            u0 = __builtin_amdgcn_sad_u16(qa[4 * c4 + 0], t0[c4].x, u0);
            u1 = __builtin_amdgcn_sad_u16(qa[4 * c4 + 1], t0[c4].y, u1);
            v0 = __builtin_amdgcn_sad_u16(qa[4 * c4 + 0], t1[c4].x, v0);
            v1 = __builtin_amdgcn_sad_u16(qa[4 * c4 + 1], t1[c4].y, v1);
            u0 = __builtin_amdgcn_sad_u16(qa[4 * c4 + 2], t0[c4].z, u0);
            u1 = __builtin_amdgcn_sad_u16(qa[4 * c4 + 3], t0[c4].w, u1);
            v0 = __builtin_amdgcn_sad_u16(qa[4 * c4 + 2], t1[c4].z, v0);
            v1 = __builtin_amdgcn_sad_u16(qa[4 * c4 + 3], t1[c4].w, v1);
        }
        wv[bb] = __builtin_amdgcn_exp2f(fmaf(__uint_as_float(u0 + u1), esc, ebias));
        wv[bb + 1] = __builtin_amdgcn_exp2f(fmaf(__uint_as_float(v0 + v1), esc, ebias));
    }
#pragma unroll
    for (int bb = 0; bb < BPW; ++bb) {
        const int b = BPW * w + bb;
        if (l == b) wv[bb] += eps;
        wv[bb] = (l < m && b < m) ? wv[bb] : 0.f;
    }
    float rsum = 0.f, wmax = 0.f;
#pragma unroll
    for (int bb = 0; bb < BPW; ++bb) {
        rsum += fabsf(wv[bb]);
        wmax = fmaxf(wmax, fabsf(wv[bb]));
    }
    wmax = wave_max_dpp(wmax);
    __syncthreads();   // every wave is done with the code tables, which W replaces
#pragma unroll
    for (int q = 0; q < BPW / 4; ++q)
        *reinterpret_cast<float4*>(sWf + l * WP + BPW * w + 4 * q) =
            make_float4(wv[4 * q], wv[4 * q + 1], wv[4 * q + 2], wv[4 * q + 3]);
    if (l == 0) sred[16 + w] = wmax;
    __syncthreads();
    {
        float csum = 0.f;   // column l, rows BPW w..+BPW
#pragma unroll
        for (int i = 0; i < BPW; ++i) csum += fabsf(sWf[(BPW * w + i) * WP + l]);
        part[w * 64 + l] = csum;
        part[NW * 64 + w * 64 + l] = rsum;   // row l, columns BPW w..+BPW
    }
    __syncthreads();
    if (w == 0) {
        // column and row sums in a fixed order, then the first maximising column / row
        float n1 = 0.f, ninf = 0.f, mx = 0.f;
#pragma unroll
        for (int g = 0; g < NW; ++g) {
            n1 += part[g * 64 + l];
            ninf += part[NW * 64 + g * 64 + l];
            mx = fmaxf(mx, sred[16 + g]);
        }
        int bs, as;
        wave_argmax_dpp(n1, bs);
        wave_argmax_dpp(ninf, as);
        if (l == 0) {
            const float c = n1 * ninf;
            sred[2] = c;
            sred[3] = mx;
            cinfo[h * 4 + 0] = c;
            cinfo[h * 4 + 1] = n1;
            cinfo[h * 4 + 2] = ninf;
            cinfo[h * 4 + 3] = (float)(as * 256 + bs);
        }
    }
    __syncthreads();
    const float c = sred[2];
    const float inv_c = c > 0.f ? 1.f / c : 0.f;
    // the iteration (product form, ns_split.hpp); W lies in the E^T region
    float* const XTh = XT + (size_t)h * 4096;
    ns_iterate_split<false, true>(sWf, inv_c, sred[3], lds, sred + 32, T,
                                  [&](int, const f32x16_t& z, int rb, int cb) {
#pragma unroll
                                      for (int r = 0; r < 16; ++r)
                                          XTh[(32 * rb + c_row(r, l)) * 64 + 32 * cb + (l & 31)] = z[r];
                                  });
}

// ------------------------------------------------------------------------------------------
// Key-side partial sums with the landmarks split over the waves (m > 48).  A landmark row in
// scalar registers feeds one VALU instruction per lane and coordinate pair; in key_kernel each
// row serves the 64 keys of one wave, and the scalar cache that delivers the rows, not the VALU,
// sets the pace.  Here a block takes tiles of 128 keys; every wave takes all of them (two per
// lane: keys l and 64 + l) against its own 16 landmarks 16w..16w+15, so each row serves 128
// keys, and contracts its rows of U over the tile on fp16 MFMA 16x16x32.  Per tile:
//   staging: wave w converts its quarter of each key row (coordinates 16w'.. of the codes, u as
//     in key_kernel) and its quarter of the value columns (fp16 times the value prescale,
//     transposed to [c][j]) into LDS; one block barrier;
//   each lane reads its two keys' codes back (rows of pitch D/2 + 4 words: conflict-free
//   16-byte reads), forms the 2 x 16 kernel values and writes them to the wave's rows of the
//   [a][j] tile;
//   MFMA: U[16w + r][c] += sum_j B[16w + r][j] V[j][c] (and the ones column) over the 4 steps
//   of 32 keys; one block barrier before the next tile's staging.
// The raw rows of the next tile (each wave its quarters) are loaded behind the landmark loop.
// Block (h, kb) takes tiles [kb T / nkb, (kb + 1) T / nkb) of the head's T = ceil(n / 128).
// Writes Upart[h][kb][c][a] as key_kernel does.
// The first nns blocks of the launch solve Newton-Schulz for heads 0 .. nns - 1 (ns_role) while
// the key blocks run: mfinal_kernel, the next launch, is the first to need X_T.
typedef unsigned short u16x2_t __attribute__((ext_vector_type(2)));
constexpr int kK2Keys = 128;
constexpr int kK2VP = kK2Keys + 8;   // pitch (halves) of the [c][j] value and [a][j] kernel-value tiles

template <int D>
struct K2Lds {
    static constexpr int CP = D / 2 + 4;   // code row pitch (words)
    static constexpr int C_BYTES = kK2Keys * CP * 4;
    static constexpr int V_BYTES = D * kK2VP * 2;
    static constexpr int B_BYTES = 4 * 16 * kK2VP * 2;
    static constexpr int KEY = C_BYTES + V_BYTES + B_BYTES;   // then the four quarters' exponents (16 bytes)
    static constexpr int BYTES = KEY + 16 > kNsRoleLds ? KEY + 16 : kNsRoleLds;
};

template <int D>
__global__ __launch_bounds__(256, D == 32 ? 4 : 3) void key2_kernel(const uint16_t* __restrict__ K,
                                                                    const uint16_t* __restrict__ V,
                                                                    const uint32_t* __restrict__ qfix,
                                                                    const uint32_t* __restrict__ kfix,
                                                                    float* __restrict__ frame,
                                                                    float* __restrict__ Upart,
                                                                    float* __restrict__ vpart, float* __restrict__ XT,
                                                                    float* __restrict__ cinfo,
                                                                    uint32_t* __restrict__ kcen, int BH, int n, int m,
                                                                    int ntile, int nkb, int T, float eps, int nns) {
    constexpr int D2 = D / 2;
    constexpr int D8 = D / 8;
    constexpr int C16 = D / 16;
    constexpr int CP = K2Lds<D>::CP;
    constexpr int QW = D8 / 4;      // 16-byte chunks of a row per wave (a quarter)
    constexpr int VP = kK2VP;
    __shared__ __attribute__((aligned(16))) char lds[K2Lds<D>::BYTES];
    if ((int)blockIdx.x < nns) {
        ns_role<D>(blockIdx.x, lds, qfix, kfix, frame, XT, cinfo, kcen, m, T, eps);
        return;
    }
    uint32_t* const sC = reinterpret_cast<uint32_t*>(lds);
    _Float16* const sV = reinterpret_cast<_Float16*>(lds + K2Lds<D>::C_BYTES);
    _Float16* const sBt = reinterpret_cast<_Float16*>(lds + K2Lds<D>::C_BYTES + K2Lds<D>::V_BYTES);
    const int nblk = BH * nkb;
    const int kbb = xcd_rank((int)blockIdx.x - nns, nblk, nns);
    const int h = kbb / nkb, kb = kbb % nkb;
    const int tid = threadIdx.x, w = tid >> 6, l = tid & 63;
    const float inv2R = frame[h * 8 + 1], esc = frame[h * 8 + 2];
    const float R = frame[h * 8 + 0], xsc = frame[h * 8 + 4];
    const bool clamped = __float_as_uint(frame[h * 8 + 5]) != 0u;   // integer test: a scalar branch
    const float ebias = -kTwo23 * esc;
    const uint32_t* tabw = qfix + ((size_t)h * 64 + 16 * __builtin_amdgcn_readfirstlane(w)) * D2;
    const int t0 = (int)((long long)kb * ntile / nkb), t1 = (int)((long long)(kb + 1) * ntile / nkb);
    _Float16* const brow = sBt + w * 16 * VP;
    f32x4_t acc[C16 + 1];
#pragma unroll
    for (int cc = 0; cc <= C16; ++cc) acc[cc] = (f32x4_t){0.f, 0.f, 0.f, 0.f};
    h8_t ones;   // B operand of the ones column: 1 in column 0
#pragma unroll
    for (int i = 0; i < 8; ++i) ones[i] = (l & 15) == 0 ? (_Float16)1.f : (_Float16)0.f;
    // Value statistics.  The fp16 copies of wave q's quarter of the value columns carry a
    // power-of-two scale 2^sig[q], the running minimum over the tiles so far of the exponent that
    // puts the tile quarter's largest |v| in [2^13, 2^14) (so no copy overflows and a quarter's
    // large values keep fp16's precision); acc of a column is rescaled exactly when its quarter's
    // exponent drops.  Wave w < C16 also sums the value columns 16w .. 16w + 15 over the keys
    // (a row of ones as the A operand against the staged values), for vbar.
    constexpr int QC = D / 4;   // value columns per quarter
    int sig[4] = {100, 100, 100, 100};   // running exponents of the four quarters (wave-uniform)
    int sigw = 100;                      // this wave's quarter's
    int* const ssig = reinterpret_cast<int*>(lds + K2Lds<D>::KEY);
    float vsum = 0.f;   // wave w < C16, lane l < 16: the sum of value column 16w + l so far
    const int wu = __builtin_amdgcn_readfirstlane(w);

    // raw quarters of the lane's two key and value rows (keys past n keep the last key rows
    // loaded, finite values of this head whose kernel values are exactly 0; their value rows are
    // zero, for the value sums)
    uint4 kq[2][QW] = {}, vq[2][QW] = {};
    // the head's rows from wave-uniform bases and a 32-bit lane offset (no 64-bit address per
    // lane to keep live through the loop)
    const uint4* const kh4 = reinterpret_cast<const uint4*>(K + (size_t)h * n * D);
    const uint4* const vh4 = reinterpret_cast<const uint4*>(V + (size_t)h * n * D);
    auto fetch = [&](int tile) {
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2) {
            const int j = tile * kK2Keys + 64 * s2 + l;
            if (j < n) {
                const uint32_t o = (uint32_t)j * (uint32_t)D8 + (uint32_t)(QW * w);
#pragma unroll
                for (int i = 0; i < QW; ++i) kq[s2][i] = kh4[o + i];
#pragma unroll
                for (int i = 0; i < QW; ++i) vq[s2][i] = vh4[o + i];
            } else {
#pragma unroll
                for (int i = 0; i < QW; ++i) vq[s2][i] = make_uint4(0u, 0u, 0u, 0u);
            }
        }
    };
    if (t0 < t1) fetch(t0);
    for (int tile = t0; tile < t1; ++tile) {
        // this wave's quarter: the largest exponent field of its values in the tile, its running
        // exponent, shared with the other waves through LDS
        {
            // |v| of a bf16 value orders as its low 15 bits: a packed 16-bit maximum of the
            // magnitudes, one instruction per two values
            u16x2_t e2 = {0, 0};
#pragma unroll
            for (int s2 = 0; s2 < 2; ++s2)
#pragma unroll
                for (int i = 0; i < QW; ++i) {
                    const uint32_t wd[4] = {vq[s2][i].x, vq[s2][i].y, vq[s2][i].z, vq[s2][i].w};
#pragma unroll
                    for (int t = 0; t < 4; ++t)
                        e2 = __builtin_elementwise_max(e2, __builtin_bit_cast(u16x2_t, wd[t] & 0x7fff7fffu));
                }
            // the wave's maximum by DPP (integer compares of the bits, wave_max_dpp)
            const int em = __float_as_int(wave_max_dpp(__int_as_float((int)max((uint32_t)e2[0], (uint32_t)e2[1]))));
            const int E = em >> 7;   // biased exponent of the largest |v| (0: zero or subnormal)
            const int st = E == 0 ? 100 : max(140 - E, -115);
            sigw = min(sigw, st);
            if (l == 0) ssig[w] = sigw;
        }
        const float vsc = __uint_as_float((uint32_t)(127 + sigw) << 23);
        // staging: this wave's quarter of the codes and of the value columns of the 128 keys
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2) {
            const int r = 64 * s2 + l;   // key row in the tile
#pragma unroll
            for (int i = 0; i < QW; ++i) {
                const uint4 x = kq[s2][i];
                *reinterpret_cast<uint4*>(sC + r * CP + 4 * (QW * w + i)) =
                    make_uint4(fix2_bf16(x.x, inv2R), fix2_bf16(x.y, inv2R), fix2_bf16(x.z, inv2R),
                               fix2_bf16(x.w, inv2R));
                const uint4 y = vq[s2][i];
                const uint32_t yw[4] = {y.x, y.y, y.z, y.w};
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    const int c = 8 * (QW * w + i) + 2 * t;
                    const uint32_t pv = pk_f16(bf16_lo(yw[t]) * vsc, bf16_hi(yw[t]) * vsc);
                    reinterpret_cast<uint16_t*>(sV)[c * VP + r] = (uint16_t)(pv & 0xffffu);
                    reinterpret_cast<uint16_t*>(sV)[(c + 1) * VP + r] = (uint16_t)(pv >> 16);
                }
            }
        }
        __syncthreads();   // the tile's codes and values are complete
        if (tile + 1 < t1) fetch(tile + 1);
        // the lane's two keys: codes, and the exponent bias (-inf past n: kernel values 0)
        uint32_t kf0[D2], kf1[D2];
#pragma unroll
        for (int c4 = 0; c4 < D2 / 4; ++c4) {
            const uint4 a0 = *reinterpret_cast<const uint4*>(sC + l * CP + 4 * c4);
            const uint4 a1 = *reinterpret_cast<const uint4*>(sC + (64 + l) * CP + 4 * c4);
            kf0[4 * c4] = a0.x; kf0[4 * c4 + 1] = a0.y; kf0[4 * c4 + 2] = a0.z; kf0[4 * c4 + 3] = a0.w;
            kf1[4 * c4] = a1.x; kf1[4 * c4 + 1] = a1.y; kf1[4 * c4 + 2] = a1.z; kf1[4 * c4 + 3] = a1.w;
        }
        const int j0 = tile * kK2Keys + l, j1 = j0 + 64;
        float kb0 = j0 < n ? ebias : -__builtin_inff(), kb1 = j1 < n ? ebias : -__builtin_inff();
        if (clamped) {
            // a head with tokens beyond the range: each key's excess enters its exponent (the
            // whole rows read again, from cache)
#pragma unroll
            for (int s2 = 0; s2 < 2; ++s2) {
                const int j = s2 ? j1 : j0;
                if (j < n) {
                    const uint4* kp = reinterpret_cast<const uint4*>(K + ((size_t)h * n + j) * D);
                    float ex = 0.f;
#pragma unroll
                    for (int c8 = 0; c8 < D8; ++c8) {
                        const uint4 r4 = kp[c8];
                        const uint32_t wd[4] = {r4.x, r4.y, r4.z, r4.w};
#pragma unroll
                        for (int t = 0; t < 4; ++t)
                            ex += fmaxf(fabsf(bf16_lo(wd[t])), R) + fmaxf(fabsf(bf16_hi(wd[t])), R);
                    }
                    const float bias = fmaf(ex - (float)D * R, xsc, ebias);
                    if (s2) kb1 = bias;
                    else kb0 = bias;
                }
            }
        }
        // kernel values of the wave's 16 landmarks (table rows past m are zero codes: finite
        // values, in rows of U that the zero columns of X_T drop) for both keys, into the
        // wave's rows of the [a][j] tile
        {
            uint16_t* bw = reinterpret_cast<uint16_t*>(brow);
            // the rows are the same every tile: an opaque copy of the table pointer keeps the
            // compiler from hoisting all 16 rows' loads out of the tile loop (they would not fit
            // the scalar registers)
            const uint32_t* tabt = tabw;
            asm volatile("" : "+s"(tabt));
            uint32_t ta[D2], tb[D2];
            load_row<D2>(ta, tabt);
#pragma unroll
            for (int p = 0; p < 8; ++p) {
                float x0, y0, x1, y1;   // x: key l, y: key 64 + l; landmarks 16w + 2p, 16w + 2p + 1
                lap_arg2<D2>(kf0, kf1, ta, tb, tabt + (2 * p + 1) * D2, esc, kb0, kb1, x0, y0);
                lap_arg2<D2>(kf0, kf1, tb, ta, tabt + (p < 7 ? 2 * p + 2 : 15) * D2, esc, kb0, kb1, x1, y1);
                const uint32_t v0 = pk_f16(__builtin_amdgcn_exp2f(x0), __builtin_amdgcn_exp2f(y0));
                const uint32_t v1 = pk_f16(__builtin_amdgcn_exp2f(x1), __builtin_amdgcn_exp2f(y1));
                bw[(2 * p) * VP + l] = (uint16_t)(v0 & 0xffffu);
                bw[(2 * p) * VP + 64 + l] = (uint16_t)(v0 >> 16);
                bw[(2 * p + 1) * VP + l] = (uint16_t)(v1 & 0xffffu);
                bw[(2 * p + 1) * VP + 64 + l] = (uint16_t)(v1 >> 16);
            }
        }
        {
            // quarters whose exponent dropped (scalar branches, rare after a block's first tile):
            // their accumulated columns to the new scale (exact); the first tile starts from zero
            int sn[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) sn[q] = __builtin_amdgcn_readfirstlane(ssig[q]);
            if (tile > t0) {
#pragma unroll
                for (int cc = 0; cc < C16; ++cc) {
                    const int qa = (16 * cc) / QC, qb = (16 * cc + 15) / QC;   // the column tile's quarters
                    const int sa = qa == 0 ? sig[0] : qa == 1 ? sig[1] : qa == 2 ? sig[2] : sig[3];
                    const int sb = qb == 0 ? sig[0] : qb == 1 ? sig[1] : qb == 2 ? sig[2] : sig[3];
                    const int na = qa == 0 ? sn[0] : qa == 1 ? sn[1] : qa == 2 ? sn[2] : sn[3];
                    const int nb = qb == 0 ? sn[0] : qb == 1 ? sn[1] : qb == 2 ? sn[2] : sn[3];
                    if (na != sa || nb != sb) {
                        const float f = ldexpf(1.f, ((16 * cc + (l & 15)) / QC == qa) ? na - sa : nb - sb);
                        acc[cc] *= f;
                        if (cc == wu) vsum *= f;
                    }
                }
            }
#pragma unroll
            for (int q = 0; q < 4; ++q) sig[q] = sn[q];
        }
        // the wave's LDS requests complete in order; the barrier keeps the compiler from moving
        // the reads of other lanes' values above the writes
        __builtin_amdgcn_wave_barrier();
        {
            const int ao = (l & 15) * VP + 8 * (l >> 4);
            f32x4_t accv = (f32x4_t){0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int s4 = 0; s4 < 4; ++s4) {
                const h8_t A = *reinterpret_cast<const h8_t*>(brow + ao + 32 * s4);
#pragma unroll
                for (int cc = 0; cc < C16; ++cc) {
                    const h8_t Bv = *reinterpret_cast<const h8_t*>(sV + 16 * cc * VP + ao + 32 * s4);
                    acc[cc] = __builtin_amdgcn_mfma_f32_16x16x32_f16(A, Bv, acc[cc], 0, 0, 0);
                    // the value sums of column tile w: `ones` as the A operand is a row 0 of ones
                    // (held by the lanes with l % 16 = 0), so row 0 of the product sums the tile's
                    // keys.  A scalar branch: a matrix instruction under a zero lane mask would
                    // still write accv.
                    if (cc == wu) accv = __builtin_amdgcn_mfma_f32_16x16x32_f16(ones, Bv, accv, 0, 0, 0);
                }
                acc[C16] = __builtin_amdgcn_mfma_f32_16x16x32_f16(A, ones, acc[C16], 0, 0, 0);
            }
            vsum += accv[0];   // row 0 (lanes l < 16: column 16w + l)
        }
        __syncthreads();   // every wave is done with the codes and values before the next staging
    }
    // rows a = 16w + 4(l/16) + r, column 16cc + l%16 (the value columns were formed from
    // V 2^sig of their quarter); the ones column from column 0 of its block; the value sums of
    // wave w < C16 from row 0 (lanes l < 16, column 16w + l)
    float* dst = Upart + ((size_t)h * nkb + kb) * (D + 1) * 64;
#pragma unroll
    for (int cc = 0; cc < C16; ++cc) {
        const int q = (16 * cc + (l & 15)) / QC;
        const int sq = q == 0 ? sig[0] : q == 1 ? sig[1] : q == 2 ? sig[2] : sig[3];
        const float inv = ldexpf(1.f, -sq);
#pragma unroll
        for (int r = 0; r < 4; ++r) dst[(16 * cc + (l & 15)) * 64 + 16 * w + 4 * (l >> 4) + r] = acc[cc][r] * inv;
        if (cc == wu && l < 16) vpart[((size_t)h * nkb + kb) * D + 16 * cc + l] = vsum * inv;
    }
    if ((l & 15) == 0) {
#pragma unroll
        for (int r = 0; r < 4; ++r) dst[D * 64 + 16 * w + 4 * (l >> 4) + r] = acc[C16][r];
    }
}

// ------------------------------------------------------------------------------------------
// U = sum over key chunks, M = X_T U, and the query side's copy of M, by column groups:
// grid (NG, BH) with NG = D/8 + 1, 576 threads (nine waves).  Group g < D/8 holds value columns
// 8g..8g+7, group D/8 the ones column D.  M = X_T U is separable by columns, so each block sums
// only its columns of the chunk partials (Upart[h][kb][c][a], four quarters of the chunks
// combined in a fixed order) and forms only its columns of M.  With `center` (the inline
// normalisation) a value group also sums the ones column and forms its operand columns as
// M'[a][c] = sum_b X_T[a][b] (U[b][c] - U[b][D] vbar[c]) = M[a][c] - M[a][D] vbar[c] in fp32:
// Y'_i = sum_l a_il M'_l = Y_i[:d] - s_i vbar, and the output Y'_i + vbar no longer takes the
// difference of Y_i[:d] and s_i vbar after the fp16 rounding of M (terms that grow with n when
// the kernel values are flat).
// Value columns: fp16 MFMA operand tiles Mt[h][s][cb][lane][i] = M[16s + 8(lane/32) + i]
// [32cb + lane%32] * 2^-e_g with mscale[h][g] = 2^e_g putting the group's largest magnitude in
// [2^14, 2^15).  Ones column: Mones[h][a] = M[a][D] in fp32.
// With vpart given (m > 48: the key blocks' value sums, [h][kb][d]), each value group forms vbar
// for its columns (the sums over the key blocks in order, in fp64, over n) and writes it for the
// query side; a non-finite sum (a NaN or infinite value) makes vbar and the frame's R NaN, so that
// every output of the head is NaN.  Otherwise vbar is read.
// With kfix given (m <= 48; for m > 48 the solve blocks of key2_kernel form it), the ones group
// also forms the query side's row bound from the key-landmark codes kfix[h]:
// kcen[h][c/2] = their centre (per coordinate, the rounded mean over the m landmarks) and
// frame[h][6] = rho = max_l sum_c |u(kt_{l,c}) - centre_c| (code units); by the triangle
// inequality every query's code distance to landmark l is at least its distance to the centre
// minus rho.
constexpr int kMfinalThreads = 576;

template <int D>
__global__ __launch_bounds__(kMfinalThreads) void mfinal_kernel(const float* __restrict__ Upart,
                                                                const float* __restrict__ XT,
                                                                _Float16* __restrict__ Mt, float* __restrict__ mscale,
                                                                float* __restrict__ Mones, float* __restrict__ Mout,
                                                                int m, int nkb, const float* __restrict__ whiten,
                                                                int mspace, int H, float* __restrict__ mvec,
                                                                float* __restrict__ vbar,
                                                                const float* __restrict__ vpart, int n, int center,
                                                                const uint32_t* __restrict__ kfix,
                                                                uint32_t* __restrict__ kcen,
                                                                float* __restrict__ frame) {
    constexpr int D1 = D + 1;
    constexpr int D2 = D / 2;
    constexpr int CB = D / 32;
    constexpr int NG = D / 8 + 1;
    constexpr int NI = 9 * 16;   // float4 items per chunk: nine columns of 64 rows
    __shared__ float sX[64 * 65];
    __shared__ __attribute__((aligned(16))) float sU[9 * 64];   // [column][b]
    __shared__ __attribute__((aligned(16))) float sM[8 * 64];   // [c][a]
    __shared__ __attribute__((aligned(16))) float4 red[3 * NI];
    __shared__ uint32_t scen[D2];
    __shared__ float smx[8];
    __shared__ float svb[8];
    const int g = blockIdx.x, h = blockIdx.y, tid = threadIdx.x, w = tid / 64, l = tid & 63;
    const bool ones = g == NG - 1;
    const int c0 = 8 * g, nc = ones ? 1 : 8;   // operand columns of this group
    // X_T (written by the previous launch, possibly through another XCD's L2) into registers
    // first, every load in flight together; stored into LDS after the chunk sums
    constexpr int NX = (4096 + kMfinalThreads - 1) / kMfinalThreads;
    float xr[NX];
#pragma unroll
    for (int i = 0; i < NX; ++i) {
        const int e = tid + i * kMfinalThreads;
        xr[i] = e < 4096 ? XT[(size_t)h * 4096 + e] : 0.f;
    }
    if (!ones && w == 0) {
        // lane (column l % 8, part l / 8): the key blocks k = part, part + 8, ... (the first
        // eight loads issued together), then the eight parts by a butterfly (the same order in
        // every lane)
        if (vpart) {
            const int col = l & 7, part = l >> 3;
            const float* src = vpart + (size_t)h * nkb * D + c0 + col;
            double t = 0.0;
            float a[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) a[i] = part + 8 * i < nkb ? src[(size_t)(part + 8 * i) * D] : 0.f;
#pragma unroll
            for (int i = 0; i < 8; ++i) t += (double)a[i];
            for (int k = part + 64; k < nkb; k += 8) t += (double)src[(size_t)k * D];
            t += __shfl_xor(t, 8, 64);
            t += __shfl_xor(t, 16, 64);
            t += __shfl_xor(t, 32, 64);
            if (l < 8) {
                float vb = (float)(t / n);
                if (!isfinite(vb)) {   // a non-finite value: every output of the head NaN
                    vb = __builtin_nanf("");
                    frame[h * 8 + 0] = vb;   // R, read by the query side
                }
                vbar[(size_t)h * D + c0 + l] = vb;
                svb[l] = vb;
            }
        } else if (l < 8) {
            svb[l] = vbar[(size_t)h * D + c0 + l];
        }
    }
    const int ncol = ones ? 1 : (center ? 9 : 8);   // columns summed: the operand columns and column D
    // item f: local column f / 16 (column D for local column 8, and in the ones group), rows
    // 4 (f % 16) .. +3 of every chunk partial; the chunks in four quarters, eight loads in flight
    const int f = tid % NI, qq = tid / NI;
    const int cl = f >> 4;
    const int gc = (ones || cl == 8) ? D : c0 + cl;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    if (cl < ncol) {
        const float4* src = reinterpret_cast<const float4*>(Upart + ((size_t)h * nkb * D1 + gc) * 64) + (f & 15);
        const int k_lo = qq * nkb / 4, k_hi = (qq + 1) * nkb / 4;
        for (int k0 = k_lo; k0 < k_hi; k0 += 8) {
            float4 t[8];
#pragma unroll
            for (int kk = 0; kk < 8; ++kk)
                t[kk] = k0 + kk < k_hi ? src[(size_t)(k0 + kk) * D1 * 16] : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
            for (int kk = 0; kk < 8; ++kk) {
                acc.x += t[kk].x; acc.y += t[kk].y; acc.z += t[kk].z; acc.w += t[kk].w;
            }
        }
    }
#pragma unroll
    for (int i = 0; i < NX; ++i) {
        const int e = tid + i * kMfinalThreads;
        if (e < 4096) sX[(e >> 6) * 65 + (e & 63)] = xr[i];
    }
    if (qq > 0 && cl < ncol) red[(qq - 1) * NI + f] = acc;
    __syncthreads();
    if (qq == 0 && cl < ncol) {
        const float4 r1 = red[f], r2 = red[NI + f], r3 = red[2 * NI + f];
        reinterpret_cast<float4*>(sU)[f] = make_float4(((acc.x + r1.x) + r2.x) + r3.x, ((acc.y + r1.y) + r2.y) + r3.y,
                                                       ((acc.z + r1.z) + r2.z) + r3.z, ((acc.w + r1.w) + r2.w) + r3.w);
    }
    if (ones && w == 8 && kfix) {
        // centre of the key-landmark codes (rows >= m of the table are zero)
        const uint32_t* tab = kfix + (size_t)h * 64 * D2;
        if (l < D2) {
            uint32_t slo = 0, shi = 0;
#pragma unroll 16
            for (int a = 0; a < 64; ++a) {
                const uint32_t u = tab[a * D2 + l];
                slo += u & 0xffffu;
                shi += u >> 16;
            }
            const uint32_t cen = ((slo + m / 2) / m) | (((shi + m / 2) / m) << 16);
            scen[l] = cen;
            kcen[(size_t)h * D2 + l] = cen;
        }
    }
    __syncthreads();
    if (ones && w == 8 && kfix) {
        // rho: the largest code distance of a landmark from the centre
        const uint32_t* tab = kfix + (size_t)h * 64 * D2;
        uint32_t dist = 0;
        if (l < m) {
#pragma unroll
            for (int c2 = 0; c2 < D2; ++c2) dist = __builtin_amdgcn_sad_u16(tab[l * D2 + c2], scen[c2], dist);
        }
        const float rho = (float)__float_as_uint(wave_max_dpp(__uint_as_float(dist)));
        if (l == 0) frame[h * 8 + 6] = rho;
    }
    // M[a][col] = sum_b X_T[a][b] U[b][col]: thread (column w, a = l); with `center`, U's value
    // columns less U[b][D] vbar[col]
    float t = 0.f;
    if (w < nc) {
        if (center && !ones) {
            const float vb = svb[w];
#pragma unroll 16
            for (int b = 0; b < 64; ++b) t = fmaf(sX[l * 65 + b], fmaf(-sU[8 * 64 + b], vb, sU[w * 64 + b]), t);
        } else {
#pragma unroll 16
            for (int b = 0; b < 64; ++b) t = fmaf(sX[l * 65 + b], sU[w * 64 + b], t);
        }
    }
    // landmark-space normalisation: the operand rows are w_l M[l] (whitening w, ones when
    // whiten is NULL), and each value column also gives sum_l w_l M[l][c] and (1/m) sum_l M[l][c]
    float mv = 0.f;
    if (w < nc) {
        if (l < m && !(center && !ones)) Mout[((size_t)h * m + l) * D1 + c0 + w] = t;
        if (mspace && !ones) {
            const float tv = l < m ? t : 0.f;
            float tw = whiten && l < m ? whiten[(size_t)(h % H) * m + l] * tv : tv;
            sM[w * 64 + l] = tw;
            float s1 = tw, s0 = tv;
#pragma unroll
            for (int off = 32; off >= 1; off >>= 1) {
                s1 += __shfl_xor(s1, off, 64);
                s0 += __shfl_xor(s0, off, 64);
            }
            if (l == 0) {
                mvec[(size_t)h * 2 * D + c0 + w] = s1;
                mvec[(size_t)h * 2 * D + D + c0 + w] = s0 / (float)m;
            }
            t = tw;
        } else {
            sM[w * 64 + l] = t;
        }
        mv = fabsf(t);
    }
    if (w < 8) {
        mv = wave_max_dpp(mv);
        if (l == 0) smx[w] = mv;
    }
    __syncthreads();
    float mxg = smx[0];
#pragma unroll
    for (int i = 1; i < 8; ++i) mxg = fmaxf(mxg, smx[i]);
    const int e = pow2_exp(mxg);
    if (tid == 0) mscale[h * NG + g] = ldexpf(1.f, e);
    if (ones) {   // rows >= m are zero; the landmark-space form weights every landmark by 1/m
        if (tid < 64) Mones[(size_t)h * 64 + tid] = mspace ? (tid < m ? 1.f / (float)m : 0.f) : sM[tid];
        return;
    }
    // operand tiles: one 16-byte chunk (i = 0..7) per (column, s, lane half)
    if (tid < nc * 4 * 2) {
        const int cc = tid & 7, hl = (tid >> 3) & 1, s4 = tid >> 4;
        const int lane = ((c0 + cc) & 31) + 32 * hl, cb = (c0 + cc) >> 5;
        _Float16 v8[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) v8[i] = (_Float16)ldexpf(sM[cc * 64 + 16 * s4 + 8 * hl + i], -e);
        const size_t o = (((size_t)h * 4 + s4) * CB + cb) * 512 + lane * 8;
        *reinterpret_cast<uint4*>(Mt + o) = *reinterpret_cast<const uint4*>(v8);
    }
}

// ------------------------------------------------------------------------------------------
// Query side.  grid (ceil(n/256) * BH) (XCD-aware order), 256 threads, lane = query.  Per wave: u(q_i) in
// registers, the m kernel values a_il from v_sad_u16 against the landmark-key table
// (wave-uniform, scalar loads) packed as fp16 pairs, a permlane32 swap that turns "query per
// lane" into the 32x32x16 operand layout for both 32-query halves, then Y^T = M^T A^T on fp16
// MFMA (M's value columns as fp16 with a power-of-two scale per column group): the result
// holds, per lane, 16 output columns of one query, so the normalisation and the bf16 stores
// happen straight from registers.  The row sum s_i = sum_l a_il M[l][d] (the ones column) is
// accumulated in fp32 in the landmark loop from the unrounded kernel values where the
// normalisation needs it (row sums, landmark space); the inline form reads M centred by
// mfinal_kernel, out_i = Y'_i + vbar.
// DWC = 1: the 3 x 3 convolution branch of Eq. (7) is formed here from the value rows of the
// queries' map neighbours (V, bf16; filters dwc_w [H][d][3][3] and bias dwc_b [H][d] or NULL;
// map width gw) instead of being read from `extra`.  The wave's 64 rows are convolved in D/8
// passes between the landmark pairs, lane l taking channels 8 (l % (D/8)) .. +7 of one row, so
// that each neighbour load reads whole rows and its latency hides behind the kernel
// evaluations; the sums wait in LDS (fp32) for the epilogue, which adds the attention part there
// and converts the row once.
template <int D, int NORM, int DWC = 0>
__global__ __launch_bounds__(256) void query2_kernel(const uint16_t* __restrict__ Q, uint16_t* __restrict__ Out,
                                                     const uint32_t* __restrict__ kfix,
                                                     const uint32_t* __restrict__ kcen,
                                                     const float* __restrict__ frame, const _Float16* __restrict__ Mt,
                                                     const float* __restrict__ mscale,
                                                     const float* __restrict__ Mones, const float* __restrict__ vbar,
                                                     const float* __restrict__ extra,
                                                     const float* __restrict__ mvec, int n, int m, int nqb, int BH,
                                                     const uint16_t* __restrict__ V, const float* __restrict__ dwc_w,
                                                     const float* __restrict__ dwc_b, int gw, int H) {
    constexpr int D2 = D / 2;
    constexpr int D8 = D / 8;
    constexpr int CB = D / 32;
    __shared__ __attribute__((aligned(16))) _Float16 sM[4 * CB * 512];
    __shared__ __attribute__((aligned(16))) float sVb[D];
    __shared__ __attribute__((aligned(16))) float sMo[64];
    __shared__ __attribute__((aligned(16))) float sMb[NORM == NORM_MSPACE ? D : 4];
    // per wave: the bf16 output rows of one 32-query half, staged so that they leave as whole
    // rows (pitch D + 8 halves)
    constexpr int OP = D + 8;
    __shared__ __attribute__((aligned(16))) uint16_t sOut[DWC ? 8 : 4 * 32 * OP];
    // convolution branch: per wave, its 64 rows in fp32 (pitch D + 4 floats), first the
    // branch's sums and then the finished output rows
    constexpr int SP = D + 4;
    __shared__ __attribute__((aligned(16))) float sSt[DWC ? 4 * 64 * SP : 4];
    // without the branch: the odd landmark rows of the key-landmark table come from LDS
    constexpr bool HYB = DWC == 0;
    __shared__ __attribute__((aligned(16))) uint32_t sTab[HYB ? 64 * D2 : 4];
    const int lin = xcd_rank(blockIdx.x, nqb * BH, 0);
    const int h = lin / nqb, qblk = lin % nqb;
    const int tid = threadIdx.x, w = tid >> 6, l = tid & 63;
    {
        const uint4* src = reinterpret_cast<const uint4*>(Mt + (size_t)h * 4 * CB * 512);
        uint4* dst = reinterpret_cast<uint4*>(sM);
        for (int e = tid; e < 4 * CB * 64; e += 256) dst[e] = src[e];
        if (tid < D) {
            if (NORM == NORM_MSPACE) {
                sVb[tid] = mvec[(size_t)h * 2 * D + tid];
                sMb[tid] = mvec[(size_t)h * 2 * D + D + tid];
            } else {
                sVb[tid] = vbar[(size_t)h * D + tid];
            }
        }
        if (tid < 64) sMo[tid] = Mones[(size_t)h * 64 + tid];
        if (HYB) {
            const uint4* ts = reinterpret_cast<const uint4*>(kfix + (size_t)h * 64 * D2);
            for (int e = tid; e < 64 * D2 / 4; e += 256) reinterpret_cast<uint4*>(sTab)[e] = ts[e];
        }
    }
    const float R = frame[h * 8 + 0], inv2R = frame[h * 8 + 1], esc = frame[h * 8 + 2];
    const float xsc = frame[h * 8 + 4];
    const bool clamped = __float_as_uint(frame[h * 8 + 5]) != 0u;   // integer test: a scalar branch
    const float rho = frame[h * 8 + 6];
    const float ebias = -kTwo23 * esc;
    constexpr int NG = D / 8 + 1;
    float scv[D / 8];
#pragma unroll
    for (int g = 0; g < D / 8; ++g) scv[g] = mscale[h * NG + g];

    const uint32_t* tab = kfix + (size_t)h * 64 * D2;
    const int i0 = qblk * 256 + w * 64;
    const int i = i0 + l;
    uint32_t qf[D2];
    float qbias = ebias;   // with the query's excess beyond the range when the head has far tokens
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
    if (clamped) {
        // a head with tokens beyond the range: the query's excess enters the exponent (its row
        // read again, from cache, so that the raw words need not stay live above)
        if (i < n) {
            const uint4* qr = reinterpret_cast<const uint4*>(Q + ((size_t)h * n + i) * D);
            float ex = 0.f;
#pragma unroll
            for (int c8 = 0; c8 < D8; ++c8) {
                const uint4 r4 = qr[c8];
                const uint32_t wd[4] = {r4.x, r4.y, r4.z, r4.w};
#pragma unroll
                for (int t = 0; t < 4; ++t) ex += fmaxf(fabsf(bf16_lo(wd[t])), R) + fmaxf(fabsf(bf16_hi(wd[t])), R);
            }
            qbias = fmaf(ex - (float)D * R, xsc, ebias);
        }
    }
    // kernel values, two landmarks per fp16 pair register (landmarks >= m give 0); the
    // landmark rows come through scalar registers, the loads of each row issued right after
    // the first use of the previous one (the table has 64 rows, zero past m).
    // Row shift: with the exp2 argument g_c of the query's distance to the landmarks' centre,
    // every landmark's argument is at most g_c + rho |escale| (triangle inequality in code
    // space), so the values are formed as exp2(g_l - sh) with sh = min(g_c + rho |escale|, 0):
    // at most 1, and a far query's values stay in fp16's range instead of underflowing.  The
    // factor f = exp2(sh) of the row is applied in fp32 in the epilogue (it cancels under the
    // row-sum normalisation).
    // convolution passes: pass k covers rows k RPP + l / CPR of the wave, channels cw .. cw + 7
    constexpr int CPR = D / 8, RPP = 64 / CPR, NP = 64 / RPP, PI = 32 / NP;
    const int cw = (l % CPR) * 8;
    float dw[9][8], db[8];   // this lane's filter taps and bias
    uint4 nv[9];             // the pass's neighbour rows, loaded a pass ahead
    // V rows of this head through a raw buffer resource: a tap off the map reads at the
    // resource's end, where the load returns zeros (its product adds nothing)
    const uint32_t vbytes = (uint32_t)n * (uint32_t)(2 * D);   // < 2^32: B H n d < 2^31
    const uint64_t vbase = (uint64_t)(V + (size_t)h * n * D);   // the block's head: one value per block
    const uint64_t vbase_s = ((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(vbase >> 32)) << 32) |
                             (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)vbase);
    const __amdgpu_buffer_rsrc_t vres = __builtin_amdgcn_make_buffer_rsrc((void*)vbase_s, 0, (int)vbytes, kRawBufferWord3);
    // map position (xq, yq) of the lane's row in the next pass, advanced by RPP tokens a pass;
    // rows past n are not clamped: their loads stay range-checked and their sums are not stored
    const int gh = DWC ? n / gw : 1;
    const int qy = DWC ? RPP / gw : 0, rx = RPP - qy * gw;
    int yq = 0, xq = 0;
    if (DWC) {
        const int iq = i0 + l / CPR;
        yq = iq / gw;
        xq = iq - yq * gw;
    }
    const uint32_t oc0 = (uint32_t)((i0 + l / CPR) * D + cw) * 2u;
    auto dwc_issue = [&](int k) {
        const bool yu = yq > 0, yd = yq < gh - 1, xl = xq > 0, xr = xq < gw - 1;
#pragma unroll
        for (int tp = 0; tp < 9; ++tp) {
            const int dy = tp / 3 - 1, dx = tp % 3 - 1;
            const bool in = (dy < 0 ? yu : (dy > 0 ? yd : true)) & (dx < 0 ? xl : (dx > 0 ? xr : true));
            // in-map offsets are exact under the unsigned wrap
            const uint32_t o = in ? oc0 + (uint32_t)((k * RPP + dy * gw + dx) * 2 * D) : vbytes;
            nv[tp] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(vres, (int)o, 0, 0));
        }
        xq += rx;
        yq += qy;
        if (xq >= gw) {
            xq -= gw;
            ++yq;
        }
    };
    auto dwc_pass = [&](int k) {
        float a[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) a[e] = db[e];
#pragma unroll
        for (int tp = 0; tp < 9; ++tp) {
            const uint32_t wd[4] = {nv[tp].x, nv[tp].y, nv[tp].z, nv[tp].w};
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                a[2 * t] = fmaf(dw[tp][2 * t], __uint_as_float(wd[t] << 16), a[2 * t]);
                a[2 * t + 1] = fmaf(dw[tp][2 * t + 1], __uint_as_float(wd[t] & 0xffff0000u), a[2 * t + 1]);
            }
        }
        float* dst = sSt + (w * 64 + k * RPP + l / CPR) * SP + cw;
        *reinterpret_cast<float4*>(dst) = make_float4(a[0], a[1], a[2], a[3]);
        *reinterpret_cast<float4*>(dst + 4) = make_float4(a[4], a[5], a[6], a[7]);
    };
    if (DWC) {
        // filters [H][d][3][3]: the lane's eight channels are 72 consecutive floats
        const float4* fw = reinterpret_cast<const float4*>(dwc_w + ((size_t)(h % H) * D + cw) * 9);
        float f[72];
#pragma unroll
        for (int e = 0; e < 18; ++e) {
            const float4 v4 = fw[e];
            f[4 * e] = v4.x;
            f[4 * e + 1] = v4.y;
            f[4 * e + 2] = v4.z;
            f[4 * e + 3] = v4.w;
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) {
#pragma unroll
            for (int tp = 0; tp < 9; ++tp) dw[tp][e] = f[9 * e + tp];
            db[e] = dwc_b ? dwc_b[(size_t)(h % H) * D + cw + e] : 0.f;
        }
        dwc_issue(0);
    }
    uint32_t ah[32];
    float srow = 0.f;   // s_i of this lane's query (of the shifted values)
    float fsh;          // exp2(sh)
    __syncthreads();    // sM, sMo, sVb
    {
        uint32_t ta[D2], tb[D2];
        load_row<D2>(tb, kcen + (size_t)h * D2);
        const float gc = lap_arg<D2>(qf, tb, ta, tab, esc, qbias);   // issues landmark row 0 into ta
        const float sh = fminf(fmaf(-esc, rho, gc), 0.f);
        qbias -= sh;
        fsh = __builtin_amdgcn_exp2f(sh);
#pragma unroll
        for (int p = 0; p < 32; ++p) {
            if (2 * p < m) {
                float a0, a1;
                if (HYB) {   // row 2p in scalar registers, row 2p + 1 from LDS
                    a0 = __builtin_amdgcn_exp2f(lap_arg_lds<D2>(qf, ta, tb, sTab + (2 * p + 1) * D2, esc, qbias));
                    a1 = lap_row<D2>(qf, tb, ta, tab + (p < 31 ? 2 * p + 2 : 63) * D2, esc, qbias);
                } else {
                    a0 = lap_row<D2>(qf, ta, tb, tab + (2 * p + 1) * D2, esc, qbias);
                    a1 = lap_row<D2>(qf, tb, ta, tab + (p < 31 ? 2 * p + 2 : 63) * D2, esc, qbias);
                }
                if (2 * p + 1 >= m) a1 = 0.f;
                if (NORM == NORM_ROWSUM || NORM == NORM_MSPACE) {
                    const float2 mo = *reinterpret_cast<const float2*>(&sMo[2 * p]);
                    srow = fmaf(a1, mo.y, fmaf(a0, mo.x, srow));
                }
                ah[p] = pk_f16(a0, a1);
            } else {
                ah[p] = 0u;
            }
            if (DWC && p % PI == PI - 1) {
                dwc_pass(p / PI);
                if (p / PI + 1 < NP) dwc_issue(p / PI + 1);
            }
        }
    }
    if (DWC) __builtin_amdgcn_wave_barrier();   // the passes' rows are read by other lanes below
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
    const int NSTEP = (m + 15) / 16;
    // s_i for the two 32-query halves in the output layout (lane l: query 32 qb + l%32)
    const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(srow), __float_as_uint(srow), false, false);
    const auto sf = __builtin_amdgcn_permlane32_swap(__float_as_uint(fsh), __float_as_uint(fsh), false, false);
    const bool nan_head = !isfinite(R);
#pragma unroll
    for (int qb = 0; qb < 2; ++qb) {
        h8_t A[4];
#pragma unroll
        for (int s4 = 0; s4 < 4; ++s4)
            A[s4] = __builtin_bit_cast(h8_t, (uint4){ah[8 * s4 + 4 * qb], ah[8 * s4 + 4 * qb + 1],
                                                     ah[8 * s4 + 4 * qb + 2], ah[8 * s4 + 4 * qb + 3]});
        const float si = __uint_as_float(sw[qb]), fi = __uint_as_float(sf[qb]);
        float tmul, tadd;   // o = y * tmul * scv[group] + tadd * vbar (+ mb, landmark-space form)
        if (NORM == NORM_INLINE) { tmul = fi; tadd = 1.f; }   // M centred: y = Y[:d] - s vbar
        else if (NORM == NORM_ROWSUM) { tmul = 1.f / si; tadd = 0.f; }
        else if (NORM == NORM_MSPACE) { tmul = fi; tadd = -si * fi; }
        else { tmul = fi; tadd = 0.f; }
        if (nan_head) tmul = __builtin_nanf("");   // every output of the head NaN
        uint16_t* stage = sOut + w * 32 * OP + (l & 31) * OP;
#pragma unroll
        for (int cb = 0; cb < CB; ++cb) {
            f32x16_t y = {};
#pragma unroll
            for (int s4 = 0; s4 < 4; ++s4) {
                if (s4 < NSTEP) {
                    const _Float16* bt = sM + (s4 * CB + cb) * 512 + l * 8;
                    y = __builtin_amdgcn_mfma_f32_32x32x16_f16(*reinterpret_cast<const h8_t*>(bt), A[s4], y, 0, 0, 0);
                }
            }
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const int c0 = 32 * cb + 8 * g + 4 * (l >> 5);
                const float4 vb = *reinterpret_cast<const float4*>(&sVb[c0]);
                const float tm = tmul * scv[4 * cb + g];   // columns c0..c0+3 are in group 4cb + g
                float o0 = fmaf(y[4 * g + 0], tm, tadd * vb.x);
                float o1 = fmaf(y[4 * g + 1], tm, tadd * vb.y);
                float o2 = fmaf(y[4 * g + 2], tm, tadd * vb.z);
                float o3 = fmaf(y[4 * g + 3], tm, tadd * vb.w);
                if (NORM == NORM_MSPACE) {
                    const float4 mb = *reinterpret_cast<const float4*>(&sMb[c0]);
                    o0 += mb.x;
                    o1 += mb.y;
                    o2 += mb.z;
                    o3 += mb.w;
                }
                if (DWC) {
                    // the convolution branch of Eq. (7), summed by the passes above: the row
                    // finishes in fp32 where the sums were and is converted once, below
                    float* so = sSt + (w * 64 + 32 * qb + (l & 31)) * SP + c0;
                    const float4 cv = *reinterpret_cast<const float4*>(so);
                    o0 += cv.x;
                    o1 += cv.y;
                    o2 += cv.z;
                    o3 += cv.w;
                    *reinterpret_cast<float4*>(so) = make_float4(o0, o1, o2, o3);
                    continue;
                } else if (extra) {   // the convolution branch of Eq. (7); rows past n read row n - 1
                    const int iq = min(i0 + 32 * qb + (l & 31), n - 1);
                    const float4 ex = *reinterpret_cast<const float4*>(extra + ((size_t)h * n + iq) * D + c0);
                    o0 += ex.x;
                    o1 += ex.y;
                    o2 += ex.z;
                    o3 += ex.w;
                }
                typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
                const bf16x2_t p0 = {(__bf16)o0, (__bf16)o1}, p1 = {(__bf16)o2, (__bf16)o3};
                uint2 st;
                st.x = __builtin_bit_cast(uint32_t, p0);
                st.y = __builtin_bit_cast(uint32_t, p1);
                *reinterpret_cast<uint2*>(stage + c0) = st;
            }
        }
        // The wave's LDS requests complete in order; the barrier keeps the compiler from moving
        // the reads of other lanes' rows above the writes.  Rows leave as 16-byte chunks, D/8
        // lanes per row, with non-temporal stores (the output is not read again here).
        __builtin_amdgcn_wave_barrier();
#pragma unroll
        for (int r0 = 0; r0 < 32; r0 += RPP) {
            const int r = r0 + l / CPR, c = (l % CPR) * 8;
            uint4 v;
            if (DWC) {
                typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
                const float* src = sSt + (w * 64 + 32 * qb + r) * SP + c;
                const float4 u0 = *reinterpret_cast<const float4*>(src);
                const float4 u1 = *reinterpret_cast<const float4*>(src + 4);
                const bf16x2_t p0 = {(__bf16)u0.x, (__bf16)u0.y}, p1 = {(__bf16)u0.z, (__bf16)u0.w};
                const bf16x2_t p2 = {(__bf16)u1.x, (__bf16)u1.y}, p3 = {(__bf16)u1.z, (__bf16)u1.w};
                v = {__builtin_bit_cast(uint32_t, p0), __builtin_bit_cast(uint32_t, p1),
                     __builtin_bit_cast(uint32_t, p2), __builtin_bit_cast(uint32_t, p3)};
            } else {
                v = *reinterpret_cast<const uint4*>(sOut + (w * 32 + r) * OP + c);
            }
            const int iq = i0 + 32 * qb + r;
            if (iq < n)
                __builtin_nontemporal_store(__builtin_bit_cast(u32x4_t, v),
                                            reinterpret_cast<u32x4_t*>(Out + ((size_t)h * n + iq) * D + c));
        }
        __builtin_amdgcn_wave_barrier();   // the next half overwrites the rows after these reads
    }
}

// ------------------------------------------------------------------------------------------
// Launch wrappers.

hipError_t launch_fast_pool(const void* Q, const void* K, const void* V, float* qt, float* kt, double* vseg,
                            float* segmax, float* vsegmax, int BH, int n, int d, int m, LmPool pl, hipStream_t st) {
    dim3 grid(m, BH);
    // m > 48: the key side (key2_kernel) forms the value statistics, V is not read here
#define LAPATTN_P2(Dv, RVv)                                                                            \
    hipLaunchKernelGGL((pool2_kernel<Dv, RVv>), grid, dim3(256), 0, st, (const uint16_t*)Q, (const uint16_t*)K, \
                       (const uint16_t*)V, qt, kt, vseg, segmax, vsegmax, n, m, pl)
    if (d == 32 && m > 48) LAPATTN_P2(32, false);
    else if (d == 32) LAPATTN_P2(32, true);
    else if (m > 48) LAPATTN_P2(64, false);
    else LAPATTN_P2(64, true);
#undef LAPATTN_P2
    return hipGetLastError();
}

hipError_t launch_fast_frame_ns(const float* qt, const float* kt, const double* vseg, const float* segmax,
                                const float* vsegmax, float* frame, uint32_t* qfix, uint32_t* kfix, float* vbar,
                                float* XT, float* cinfo, int BH, int n, int d, int m, float lambda, int T, float eps,
                                hipStream_t st) {
    // m > 48: the frame alone; the solve runs in the key-side launch (key2_kernel)
    if (d == 32 && m > 48)
        hipLaunchKernelGGL((frame_ns_kernel<32, false>), dim3(BH), dim3(kSolveThreads), 0, st, qt, kt, vseg, segmax,
                           vsegmax, frame, qfix, kfix, vbar, XT, cinfo, n, m, lambda, T, eps);
    else if (m > 48)
        hipLaunchKernelGGL((frame_ns_kernel<64, false>), dim3(BH), dim3(kSolveThreads), 0, st, qt, kt, vseg, segmax,
                           vsegmax, frame, qfix, kfix, vbar, XT, cinfo, n, m, lambda, T, eps);
    else if (d == 32)
        hipLaunchKernelGGL((frame_ns_kernel<32, true>), dim3(BH), dim3(kSolveThreads), 0, st, qt, kt, vseg, segmax,
                           vsegmax, frame, qfix, kfix, vbar, XT, cinfo, n, m, lambda, T, eps);
    else
        hipLaunchKernelGGL((frame_ns_kernel<64, true>), dim3(BH), dim3(kSolveThreads), 0, st, qt, kt, vseg, segmax,
                           vsegmax, frame, qfix, kfix, vbar, XT, cinfo, n, m, lambda, T, eps);
    return hipGetLastError();
}

hipError_t launch_fast_key2(const void* K, const void* V, const uint32_t* qfix, const uint32_t* kfix,
                            float* frame, float* Upart, float* vpart, float* XT, float* cinfo, uint32_t* kcen, int BH,
                            int n, int d, int m, int ntile, int nkb, int T, float eps, hipStream_t st) {
    dim3 grid(BH + BH * nkb);   // BH solve blocks first, then the key blocks
    if (d == 32)
        hipLaunchKernelGGL(key2_kernel<32>, grid, dim3(256), 0, st, (const uint16_t*)K, (const uint16_t*)V, qfix, kfix,
                           frame, Upart, vpart, XT, cinfo, kcen, BH, n, m, ntile, nkb, T, eps, BH);
    else
        hipLaunchKernelGGL(key2_kernel<64>, grid, dim3(256), 0, st, (const uint16_t*)K, (const uint16_t*)V, qfix, kfix,
                           frame, Upart, vpart, XT, cinfo, kcen, BH, n, m, ntile, nkb, T, eps, BH);
    return hipGetLastError();
}

hipError_t launch_fast_key(const void* K, const void* V, const uint32_t* qfix, const float* frame, float* Upart,
                           int BH, int n, int d, int m, int kpb, int nkb, hipStream_t st) {
    dim3 grid(BH * nkb);
    if (d == 32)
        hipLaunchKernelGGL(key_kernel<32>, grid, dim3(256), 0, st, (const uint16_t*)K, (const uint16_t*)V, qfix,
                           frame, Upart, BH, n, m, kpb, nkb);
    else
        hipLaunchKernelGGL(key_kernel<64>, grid, dim3(256), 0, st, (const uint16_t*)K, (const uint16_t*)V, qfix,
                           frame, Upart, BH, n, m, kpb, nkb);
    return hipGetLastError();
}

hipError_t launch_fast_mfinal(const float* Upart, const float* XT, _Float16* Mt, float* mscale, float* Mones,
                              float* M, int BH, int d, int m, int nkb, const float* whiten, int mspace, int H,
                              float* mvec, float* vbar, const float* vpart, int n, int center, const uint32_t* kfix,
                              uint32_t* kcen, float* frame, hipStream_t st) {
    if (d == 32)
        hipLaunchKernelGGL(mfinal_kernel<32>, dim3(32 / 8 + 1, BH), dim3(kMfinalThreads), 0, st, Upart, XT, Mt, mscale,
                           Mones, M, m, nkb, whiten, mspace, H, mvec, vbar, vpart, n, center, kfix, kcen, frame);
    else
        hipLaunchKernelGGL(mfinal_kernel<64>, dim3(64 / 8 + 1, BH), dim3(kMfinalThreads), 0, st, Upart, XT, Mt, mscale,
                           Mones, M, m, nkb, whiten, mspace, H, mvec, vbar, vpart, n, center, kfix, kcen, frame);
    return hipGetLastError();
}

hipError_t launch_fast_query(int norm, const void* Q, void* Out, const uint32_t* kfix, const uint32_t* kcen,
                             const float* frame,
                             const _Float16* Mt, const float* mscale, const float* Mones, const float* vbar,
                             const float* extra, const float* mvec, int BH, int n, int d, int m, const void* V,
                             const float* dwc_w, const float* dwc_b, int gw, int H, hipStream_t st) {
    const int nqb = (n + 255) / 256;
    dim3 grid(nqb * BH);
    const bool fused = dwc_w != nullptr;   // the 3 x 3 branch in the epilogue
#define LAPATTN_Q2(Dv, Nv, Fv)                                                                                        \
    hipLaunchKernelGGL((query2_kernel<Dv, Nv, Fv>), grid, dim3(256), 0, st, (const uint16_t*)Q, (uint16_t*)Out, kfix, \
                       kcen, frame, Mt, mscale, Mones, vbar, extra, mvec, n, m, nqb, BH, (const uint16_t*)V, dwc_w,   \
                       dwc_b, gw, H)
#define LAPATTN_Q2N(Dv, Fv)                                              \
    do {                                                                 \
        if (norm == NORM_INLINE) LAPATTN_Q2(Dv, NORM_INLINE, Fv);        \
        else if (norm == NORM_ROWSUM) LAPATTN_Q2(Dv, NORM_ROWSUM, Fv);   \
        else if (norm == NORM_MSPACE) LAPATTN_Q2(Dv, NORM_MSPACE, Fv);   \
        else LAPATTN_Q2(Dv, NORM_NONE, Fv);                              \
    } while (0)
    if (d == 32) {
        if (fused) LAPATTN_Q2N(32, 1);
        else LAPATTN_Q2N(32, 0);
    } else {
        if (fused) LAPATTN_Q2N(64, 1);
        else LAPATTN_Q2N(64, 0);
    }
#undef LAPATTN_Q2N
#undef LAPATTN_Q2
    return hipGetLastError();
}

}  // namespace lapattn
