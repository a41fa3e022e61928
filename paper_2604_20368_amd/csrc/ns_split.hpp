// ns_split.hpp -- Newton-Schulz (Algorithm 2) on 64 x 64 matrices in product form on the fp16
// matrix cores, with every factor an fp16 pair (hi + lo, about 22 significant bits), for one
// workgroup of four waves: the solve of the bf16-input path (fast.hip), whose tolerance the
// 22-bit products meet.  (The fp32-input path keeps fp32 products: in product form the rounding
// of E_0 is never corrected, and where K_LL is ill-conditioned -- m = n, T = 50 -- 22 bits gave
// 2e-4 against the 1e-4 fp32 tolerance.)
//
// Product form.  With X0 = W^T / c and E = I - W X0, the updates X_{t+1} = X_t (2I - W X_t)
// satisfy I - W X_t = E^(2^t), hence
//   X_T = X0 (I + E_0)(I + E_1) ... (I + E_{T-1}),  E_0 = E,  E_{k+1} = E_k E_k,
// and Z_k = X0 (I + E_0) ... (I + E_{k-1}) equals X_k in exact arithmetic.  The two products of a
// step (Z_{k+1} = Z_k + Z_k E_k, E_{k+1} = E_k E_k) are independent.  Wave w owns the 32 x 32
// block (rb, cb) = (w / 2, w % 2) of both; only transposed copies are stored (Z^T, E^T as fp16
// pairs, pitch kLP), and the A operands come through transposing LDS reads.
// Scales: ||E_k||_2 <= 1 (E's spectrum lies in [0, 1)), so E is stored unscaled.  Z carries a
// power-of-two scale: Z_0's from its exact maximum (largest entry in [2^14, 2^15)), Z_{k+1}'s
// from the maximum of Z_k, placing that maximum in [2^7, 2^8); ||I + E_k||_2 <= 2 bounds the
// growth of the largest entry by 2 * 64 = 2^7 per step, so stored values stay below 2^15.
// Z itself is accumulated in fp32 registers.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace lapattn {

typedef _Float16 h8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));
typedef short s4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s4_t lds_s4_t;

constexpr int kLP = 72;   // LDS row pitch (halves) of the 64 x 64 fp16 tiles
constexpr int kWP = 68;   // LDS row pitch (floats) of W in fp32

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

// Two floats to a packed fp16 pair, round to nearest even (v_cvt_pk_f16_f32).
__device__ __forceinline__ uint32_t pk_f16(float a, float b) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){a, b}, f16x2_t));
}

// Row of result register r of a 32x32 MFMA block at lane l (within the block).
__device__ __forceinline__ int c_row(int r, int l) { return 8 * (r >> 2) + 4 * (l >> 5) + (r & 3); }

// Power-of-two exponent that brings a maximum magnitude into [2^14, 2^15) (0 when mx is 0).
__device__ __forceinline__ int pow2_exp(float mx) { return (mx > 0.f && isfinite(mx)) ? ilogbf(mx) - 14 : 0; }

// The A operand of MFMA 32x32x16 (8 halves: row 32 rb + l%32, k = k0 + 8(l/32)..+8) of a
// matrix held transposed in LDS (Mt[k][row], pitch kLP), via two ds_read_b64_tr_b16.  Within a
// 16-lane group that instruction gives lane i element i%4 of the 4-element reads of lanes
// 4q + i/4 (q = 0..3): when lane j of the group points at Mt[k1 + j/4][r0 + 4(j%4)], lane i
// receives Mt[k1 + q][r0 + i], q = 0..3 -- row r0 + i of M over 4 consecutive k.
__device__ __forceinline__ h8_t a_from_transposed(const _Float16* Mt, int rb, int k0) {
    const int l = threadIdx.x & 63, g = l >> 4, i = l & 15;
    const _Float16* p = Mt + (k0 + 8 * (g >> 1) + (i >> 2)) * kLP + 32 * rb + 16 * (g & 1) + 4 * (i & 3);
    const s4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4_t*)p);
    const s4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s4_t*)(p + 4 * kLP));
    typedef short s8_t __attribute__((ext_vector_type(8)));
    return __builtin_bit_cast(h8_t, (s8_t)__builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

// One wave's 32 x 32 block of a 64 x 64 product, both factors fp16 pairs, B read from its
// transposed copy (BT[col][k]); the A operands of the four k steps are given (hi, lo).
// Result register r holds row 32 rb + c_row(r, l), column 32 cb + l%32.
__device__ __forceinline__ f32x16_t mm32_split(const h8_t (&ah)[4], const h8_t (&al)[4],
                                               const _Float16* __restrict__ BTh, const _Float16* __restrict__ BTl,
                                               int cb) {
    const int l = threadIdx.x & 63;
    const int bo = (32 * cb + (l & 31)) * kLP + 8 * (l >> 5);
    f32x16_t hh = {}, hl = {}, lh = {};
#pragma unroll
    for (int s4 = 0; s4 < 4; ++s4) {
        const h8_t bh = *reinterpret_cast<const h8_t*>(BTh + bo + 16 * s4);
        const h8_t bl = *reinterpret_cast<const h8_t*>(BTl + bo + 16 * s4);
        hh = __builtin_amdgcn_mfma_f32_32x32x16_f16(ah[s4], bh, hh, 0, 0, 0);
        hl = __builtin_amdgcn_mfma_f32_32x32x16_f16(ah[s4], bl, hl, 0, 0, 0);
        lh = __builtin_amdgcn_mfma_f32_32x32x16_f16(al[s4], bh, lh, 0, 0, 0);
    }
    return hh + (hl + lh);
}

// Two floats as packed fp16 pairs: hi = rn(x), lo = rn(x - hi) (each one v_cvt_pk_f16_f32).
__device__ __forceinline__ void split_pk(float x0, float x1, uint32_t& hi, uint32_t& lo) {
    const f16x2_t h = __builtin_convertvector((f32x2_t){x0, x1}, f16x2_t);
    const f32x2_t back = __builtin_convertvector(h, f32x2_t);
    hi = __builtin_bit_cast(uint32_t, h);
    lo = pk_f16(x0 - back[0], x1 - back[1]);
}

// Store a wave's 32 x 32 block (times `scale`) transposed as an fp16 pair: four consecutive
// rows of one column per 8-byte write.
__device__ __forceinline__ void store32_t(const f32x16_t& v, float scale, int rb, int cb, _Float16* MTh,
                                          _Float16* MTl) {
    const int l = threadIdx.x & 63;
    const int col = 32 * cb + (l & 31);
#pragma unroll
    for (int g = 0; g < 4; ++g) {
        uint32_t h0, l0, h1, l1;
        split_pk(v[4 * g] * scale, v[4 * g + 1] * scale, h0, l0);
        split_pk(v[4 * g + 2] * scale, v[4 * g + 3] * scale, h1, l1);
        const int o = col * kLP + 32 * rb + 8 * g + 4 * (l >> 5);
        *reinterpret_cast<uint2*>(MTh + o) = make_uint2(h0, h1);
        *reinterpret_cast<uint2*>(MTl + o) = make_uint2(l0, l1);
    }
}

// LDS the iteration needs: Z^T and E^T as fp16 pairs.
constexpr int kNsSplitLds = 4 * 64 * kLP * 2;

// The T updates of Algorithm 2 in product form, by the four waves of a workgroup (256 threads),
// for W (64 x 64, zero outside m x m) held in fp32 in LDS (sWf, pitch kWP), with inv_c = 1 / c
// (0 when c = 0: X = 0) and wmax = max |W_ab|.  buf is kNsSplitLds bytes of LDS, free on entry;
// W_IN_ET: sWf lies in buf's E^T half (it is read until E_0 replaces it), else it must not alias
// buf.  sred is 4 floats of LDS.  Every wave must call it; it begins and ends with a barrier.
// emit(k, z, rb, cb) receives each wave's 32 x 32 block of X_k (fp32; result register r is row
// 32 rb + c_row(r, l), column 32 cb + l % 32) for k = 0 .. T when all_iterates, else for k = T
// only.
template <bool all_iterates, bool W_IN_ET, class Emit>
__device__ __forceinline__ void ns_iterate_split(const float* sWf, float inv_c, float wmax, char* buf, float* sred,
                                                 int T, Emit&& emit) {
    constexpr int TB = 64 * kLP;
    _Float16* const ZTh = reinterpret_cast<_Float16*>(buf);
    _Float16* const ZTl = ZTh + TB;
    _Float16* const ETh = ZTh + 2 * TB;
    _Float16* const ETl = ZTh + 3 * TB;
    const int tid = threadIdx.x, w = tid >> 6, l = tid & 63;
    const int rb = w >> 1, cb = w & 1;
    float mx = wmax * inv_c;                // max |X0| = max |Z_0|
    float zs = ldexpf(1.f, pow2_exp(mx));   // Z_true = Z_stored * zs
    __syncthreads();   // W complete; buf free
    {
        // Z_0^T = X0^T = W / c: row a, columns 8 j .. 8 j + 7 per thread and pass
        const float x0s = inv_c / zs;
#pragma unroll
        for (int p = 0; p < 2; ++p) {
            const int e = tid + 256 * p, a = e >> 3, b0 = 8 * (e & 7);
            const float4 u = *reinterpret_cast<const float4*>(sWf + a * kWP + b0);
            const float4 v = *reinterpret_cast<const float4*>(sWf + a * kWP + b0 + 4);
            uint32_t h[4], lo[4];
            split_pk(u.x * x0s, u.y * x0s, h[0], lo[0]);
            split_pk(u.z * x0s, u.w * x0s, h[1], lo[1]);
            split_pk(v.x * x0s, v.y * x0s, h[2], lo[2]);
            split_pk(v.z * x0s, v.w * x0s, h[3], lo[3]);
            *reinterpret_cast<uint4*>(ZTh + a * kLP + b0) = make_uint4(h[0], h[1], h[2], h[3]);
            *reinterpret_cast<uint4*>(ZTl + a * kLP + b0) = make_uint4(lo[0], lo[1], lo[2], lo[3]);
        }
    }
    // Z_0 = X0 (this wave's block, fp32): X0[row][col] = W[col][row] / c
    f32x16_t zreg;
#pragma unroll
    for (int r = 0; r < 16; ++r) zreg[r] = sWf[(32 * cb + (l & 31)) * kWP + 32 * rb + c_row(r, l)] * inv_c;
    if (all_iterates || T == 0) emit(0, zreg, rb, cb);
    __syncthreads();   // Z_0^T complete
    if (T == 0) return;
    // E_0 = I - W X0 (A = W split from the fp32 copy, B = X0 through Z^T)
    {
        h8_t wah[4], wal[4];
#pragma unroll
        for (int s4 = 0; s4 < 4; ++s4) {
            const float* src = sWf + (32 * rb + (l & 31)) * kWP + 16 * s4 + 8 * (l >> 5);
            uint32_t hq[4], lq[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) split_pk(src[2 * q], src[2 * q + 1], hq[q], lq[q]);
            wah[s4] = __builtin_bit_cast(h8_t, make_uint4(hq[0], hq[1], hq[2], hq[3]));
            wal[s4] = __builtin_bit_cast(h8_t, make_uint4(lq[0], lq[1], lq[2], lq[3]));
        }
        f32x16_t e0 = mm32_split(wah, wal, ZTh, ZTl, cb);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int row = 32 * rb + c_row(r, l), col = 32 * cb + (l & 31);
            e0[r] = (row == col ? 1.f : 0.f) - e0[r] * zs;
        }
        if (W_IN_ET) __syncthreads();   // every wave has read W before E_0 takes its place
        store32_t(e0, 1.f, rb, cb, ETh, ETl);
    }
    __syncthreads();
    for (int k = 0; k < T; ++k) {
        // Z_{k+1} = Z_k + Z_k E_k and, but for the last step, E_{k+1} = E_k E_k
        h8_t ah[4], al[4];
#pragma unroll
        for (int s4 = 0; s4 < 4; ++s4) {
            ah[s4] = a_from_transposed(ZTh, rb, 16 * s4);
            al[s4] = a_from_transposed(ZTl, rb, 16 * s4);
        }
        const f32x16_t dz = mm32_split(ah, al, ETh, ETl, cb);
#pragma unroll
        for (int r = 0; r < 16; ++r) zreg[r] = fmaf(dz[r], zs, zreg[r]);
        if (all_iterates || k + 1 == T) emit(k + 1, zreg, rb, cb);
        if (k + 1 < T) {
#pragma unroll
            for (int s4 = 0; s4 < 4; ++s4) {
                ah[s4] = a_from_transposed(ETh, rb, 16 * s4);
                al[s4] = a_from_transposed(ETl, rb, 16 * s4);
            }
            const f32x16_t e = mm32_split(ah, al, ETh, ETl, cb);
            // scale of Z_{k+1} from the maximum of Z_k (mx)
            zs = ldexpf(1.f, (mx > 0.f && isfinite(mx)) ? ilogbf(mx) - 7 : 0);
            float lm = 0.f;
#pragma unroll
            for (int r = 0; r < 16; ++r) lm = fmaxf(lm, fabsf(zreg[r]));
            lm = wave_max_dpp(lm);
            __syncthreads();   // every wave's reads of step k are done
            store32_t(zreg, 1.f / zs, rb, cb, ZTh, ZTl);
            store32_t(e, 1.f, rb, cb, ETh, ETl);
            if (l == 0) sred[w] = lm;
            __syncthreads();
            mx = fmaxf(fmaxf(sred[0], sred[1]), fmaxf(sred[2], sred[3]));
        }
    }
    __syncthreads();   // buf and sred free for the caller
}

}  // namespace lapattn
