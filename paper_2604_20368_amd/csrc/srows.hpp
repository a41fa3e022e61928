// srows.hpp -- wave-uniform rows through scalar registers, shared by the fp32 kernels.
//
// A table row that every lane of a wave reads at the same address (a landmark row) is loaded
// with scalar loads, 32 floats at a time, and used as the scalar operand of the VALU.  Loops
// over rows keep two 32-float buffers and issue the loads of the next unit right after the
// first use of the current one (which is where the wave waits for it), so that one unit is in
// flight while the other is consumed.
#pragma once

#include <hip/hip_runtime.h>

namespace lapattn {

// 32 consecutive floats of a wave-uniform row (scalar loads).  The row is read through the
// constant address space: the tables are written by earlier launches and never within the
// reading kernel, and this is what lets the loads be scalar (s_load) wherever the kernel also
// stores to memory before them.
typedef const __attribute__((address_space(4))) float cfloat_t;

__device__ __forceinline__ void srow32(float (&t)[32], const float* __restrict__ p) {
    cfloat_t* q = (cfloat_t*)p;
#pragma unroll
    for (int c = 0; c < 32; ++c) t[c] = q[c];
}

// acc + sum_c |t_c - x_c| over 32 coordinates (t in scalar registers); the loads of the next
// unit into `nt` are issued after the first use of `t`.
__device__ __forceinline__ float l1_unit(const float* x, const float (&t)[32], float (&nt)[32],
                                         const float* __restrict__ next, float acc) {
    float a0 = acc + fabsf(t[0] - x[0]);
    __builtin_amdgcn_sched_barrier(0);
    srow32(nt, next);
    __builtin_amdgcn_sched_barrier(0);
    float a1 = fabsf(t[1] - x[1]);
#pragma unroll
    for (int c = 2; c < 32; c += 2) {
        a0 += fabsf(t[c] - x[c]);
        a1 += fabsf(t[c + 1] - x[c + 1]);
    }
    return a0 + a1;
}

// dq_c += dd * sign(q_c - t_c) over 32 coordinates (t in scalar registers), sign(0) = 0, as
// (dd 2^64) * med3(q_c - t_c, -2^-64, 2^-64): the clamp is exactly +-2^-64 for every difference
// of magnitude at least 2^-64 (smaller nonzero differences give a fraction of dd), and both
// scalings by powers of two are exact.  The next unit's loads go into `nt` after the first use
// of `t`.
__device__ __forceinline__ float sgn_term(float x, float t) { return __builtin_amdgcn_fmed3f(x - t, -0x1p-64f, 0x1p-64f); }

__device__ __forceinline__ void sgn_unit(float* dq, const float* q, const float (&t)[32], float (&nt)[32],
                                         const float* __restrict__ next, float dd) {
    const float dds = dd * 0x1p64f;
    dq[0] = fmaf(dds, sgn_term(q[0], t[0]), dq[0]);
    __builtin_amdgcn_sched_barrier(0);
    srow32(nt, next);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int c = 1; c < 32; ++c) dq[c] = fmaf(dds, sgn_term(q[c], t[c]), dq[c]);
}

// The same without a prefetch (the row was loaded for an earlier unit and is still live).
__device__ __forceinline__ void sgn_unit_nopf(float* dq, const float* q, const float (&t)[32], float dd) {
    const float dds = dd * 0x1p64f;
#pragma unroll
    for (int c = 0; c < 32; ++c) dq[c] = fmaf(dds, sgn_term(q[c], t[c]), dq[c]);
}

}  // namespace lapattn
