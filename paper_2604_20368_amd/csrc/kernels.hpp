// kernels.hpp -- launch wrappers of the lapattn HIP kernels (internal to the library).
//
// Workspace arrays are described in host.cpp; every pointer here is device memory.
// All wrappers enqueue on `st` and return the launch status.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "common.hpp"

namespace lapattn {

// Forward ---------------------------------------------------------------------

// Landmark means qt, kt [BH][m][d] (fp32; V is not read: the key side forms its sums); pl
// selects segments or r x r windows (common.hpp).  When m BH is small each landmark's tokens
// are split over pool_split(BH, n, m) blocks whose fp64 sums go to part ([BH][m][S][2][d]) and
// are added in order by a second launch.
int pool_split(int BH, int n, int m);
hipError_t launch_pool(int dt, const void* Q, const void* K, float* qt, float* kt, double* part,
                       int BH, int n, int d, int m, LmPool pl, hipStream_t st);

// Key-side summary: per key chunk, Upart[h][chunk][a][c] = sum_j k(qt_a, k_j) [v_j | 1]_c and the
// value sums vpart[h][chunk][c] = sum_j v_jc (for vbar); with Bsave, also the rows
// B[j][a] = k(qt_a, k_j) for the backward, group-major ([BH][G][n][64] for the G = ceil(m / 64)
// landmark groups, zeros past m).
hipError_t launch_key_summary(int dt, const void* K, const void* V, const float* qt, float* Upart, float* vpart,
                              float* Bsave, int BH, int n, int d, int m, float lambda, int chunk_keys, int nkc,
                              hipStream_t st);

// Newton-Schulz on K_LL and the solved matrix M = X_T U, m <= 64.
//   Xs:    [BH][store_all ? T+2 : 1][MP][MP] fp64 iterates (padded to MP), then W
//   cinfo: [BH][4] fp64: scale c, ||W||_1, ||W||_inf, (a* * 256 + b*)
//   U, M:  [BH][m][d+1] fp32;  Mc: [BH][m][d] fp32, M[:, :d] - M[:, d] vbar^T;  vbar: [BH][d] fp32
//   (vbar from the key chunks' value sums vpart)
hipError_t launch_ns_solve(const float* qt, const float* kt, const float* Upart, const float* vpart,
                           double* Xs, double* cinfo, float* U, float* M, float* Mc, float* vbar,
                           int BH, int n, int d, int m, int T, double lambda, double eps, int nkc,
                           int store_all, int MP, hipStream_t st);

// Query side: Out_i = normalise(sum_l k(q_i, kt_l) M_l) (+ extra_i when extra, [BH][n][d], is given);
// the inline form reads Mc (launch_ns_solve).
// The landmark-space normalisation takes the whitening [H][m] (NULL: ones) and mvec below.
// With Asave, also the rows A[i][l] = k(q_i, kt_l) for the backward, group-major ([BH][G][n][64],
// columns below m).
hipError_t launch_query_out(int dt, int norm, const void* Q, void* Out, const float* kt, const float* M,
                            const float* Mc, const float* vbar, const float* extra, const float* whiten, const float* mvec,
                            float* Asave, int BH, int H, int n, int d, int m, float lambda, hipStream_t st);

// Small heads (fp32, n <= 256, m <= 32, d 32 or 64; norm inline, row sums or none): the whole
// forward of a head in one workgroup, Out [BH][n][d]; no workspace.
hipError_t launch_small_forward(int norm, const float* Q, const float* K, const float* V, float* Out, int BH, int n,
                                int d, int m, float lambda, int T, float eps, LmPool pl, hipStream_t st);

// The same for 64 < m <= 128 (nsbig.hip), products spread over many workgroups:
//   Xs:    [BH][T+2][128][128] fp64: X_0 .. X_T, then W (always all of them)
//   Ebuf:  [BH][2][128][128] fp64 scratch;  Ud: [BH][m][d+1] fp64 scratch
struct NsbJob {   // Out = alpha op(A) op(B) + beta1 C1 + beta2 C2 + gamma I (diagonal below idm)
    const double *A, *B, *C1, *C2;
    double* Out;
    long long sA, sB, sC1, sC2, sOut;   // per-head strides (doubles)
    int pa, pb, pc1, pc2, pout;          // row pitches (doubles)
    int ta, tb;                          // op(X) = X^T
    int M, N, K, idm;                    // Out is M x N; K <= 128
    double alpha, beta1, beta2, gamma;
};
struct NsbJobs {
    NsbJob j[3];
};
NsbJob nsb_job(const double* A, long long sA, int pa, bool ta, const double* B, long long sB, int pb, bool tb,
               double* Out, long long sOut, int pout, int M, int N, int K, double alpha);
hipError_t launch_nsb_mm(const NsbJobs& js, int njobs, int BH, hipStream_t st);
hipError_t launch_nsb_forward(const float* qt, const float* kt, const float* Upart, const float* vpart, double* Xs,
                              double* Ebuf, double* Ud, double* cinfo, float* U, float* M, float* Mc, float* vbar,
                              int BH, int n, int d, int m, int T, double lambda, double eps, int nkc, hipStream_t st);
// Scratch doubles of launch_nsb_backward.
inline size_t nsb_backward_scratch(int BH, int d) {
    return (size_t)BH * (7 * 128 * 128 + 3 * 128 * (size_t)(d + 1) + 2 * (size_t)d);
}

// Landmark-space normalisation: mvec[BH][2][d] = {sum_l w_l M_l[:d], (1/m) sum_l M_l[:d]}.
hipError_t launch_mspace_vec(const float* M, const float* whiten, float* mvec, int BH, int H, int d, int m,
                             hipStream_t st);

// Backward (fp32 inputs) --------------------------------------------------------

// Query-major pass: writes the direct dQ term, the kernel values Aq (read instead when saved: the
// forward's launch_query_out left them there) and dDq = -A dA / lambda
// ([BH][G][n][64], group-major for the G = ceil(m / 64) landmark groups), per-query dY scale rs and last column dYd ([BH][n]), and per-block
// partial sums of dvbar ([BH][nqb][d]; for the landmark-space normalisation also the sums of
// dO into p0_part, with the whitening and mvec of the forward).
hipError_t launch_bwd_query(int norm, const float* Q, const float* dO, float* dQ,
                            const float* kt, const float* M, const float* vbar,
                            float* Aq, float* dDq, float* rs, float* dYd, float* dvbar_part,
                            float* p0_part, const float* whiten, const float* mvec, int saved,
                            int BH, int H, int n, int d, int m, float lambda, int nqb, hipStream_t st);

// Landmark-major pass over queries: partial dM [BH][nlc][m][d+1] and dkt [BH][nlc][m][d].
hipError_t launch_bwd_query_lm(const float* Q, const float* dO, const float* kt,
                               const float* Aq, const float* dDq, const float* rs, const float* dYd,
                               float* dM_part, float* dkt_part,
                               int BH, int n, int d, int m, int chunk, int nlc, hipStream_t st);

// Newton-Schulz backward: dU [BH][m][d+1], dvbar [BH][d], the K_LL gradient mapped to the
// query landmarks, dqtW [BH][m][d], and the whole key-landmark gradient over each landmark's
// token count, dkpool [BH][m][d] = (K_LL term + the query-side partials dkt_part) / |S_l|;
// dDW [BH][MP][MP] fp32 is scratch (the gradient of the kernel distances, between the solve's
// backward and launch_kll_backward).
hipError_t launch_bwd_ns(const float* qt, const float* kt, const double* Xs, const double* cinfo,
                         const float* U, const float* dM_part, const float* dvbar_part,
                         float* dU, float* dvbar, float* dqtW, float* dkpool, const float* dkt_part, LmPool pl,
                         const float* p0_part, const float* whiten, int mspace, float* dDW,
                         int BH, int H, int n, int d, int m, int T, double lambda, double eps,
                         int nlc, int nqb, int MP, hipStream_t st);
// K_LL backward from dDW [BH][MPW][MPW] (zero past m): dqtW and dkpool as above (nsbig.hip).
hipError_t launch_kll_backward(const float* qt, const float* kt, const float* dDW, float* dqtW, float* dkpool,
                               const float* dkt_part, LmPool pl, int BH, int n, int d, int m, int MPW, int nlc,
                               hipStream_t st);
// The same for 64 < m <= 128 (nsbig.hip), with nsb_backward_scratch(BH, d) doubles of scratch and
// dDW [BH][128][128] fp32; Xs as launch_nsb_forward left it.
hipError_t launch_nsb_backward(const float* qt, const float* kt, const double* Xs, const double* cinfo,
                               const float* U, const float* dM_part, const float* dvbar_part,
                               const float* p0_part, const float* whiten, int mspace, float* dU, float* dvbar,
                               float* dqtW, float* dkpool, const float* dkt_part, LmPool pl, double* scratch,
                               float* dDW, int BH, int H, int n, int d, int m, int T, double lambda, double eps,
                               int nlc, int nqb, hipStream_t st);

// Key-major pass: final dK (the direct term plus dkpool of the key's landmark), final dV, and
// dDk = -B dB / lambda ([BH][G][n][64], group-major).  saved: dDk holds B's rows from the forward on entry
// (launch_key_summary's Bsave) instead of being recomputed.
hipError_t launch_bwd_key(const float* K, const float* V, float* dK, float* dV,
                          const float* qt, const float* dU, const float* dvbar, float* dDk, const float* dkpool,
                          LmPool pl, int saved, int BH, int n, int d, int m, float lambda, hipStream_t st);

// Landmark-major pass over keys: partial dqt [BH][nlc][m][d].
hipError_t launch_bwd_key_lm(const float* K, const float* qt, const float* dDk, float* dqt_part,
                             int BH, int n, int d, int m, int chunk, int nlc, hipStream_t st);

// Landmark-mean backward of the queries: dQ_i += dqt_{l(i)} / |S_l| (dqt = dqtW + the key-side
// partials); the keys' share is added by launch_bwd_key.
hipError_t launch_bwd_pool(float* dQ, const float* dqtW, const float* dqt_part,
                           int BH, int n, int d, int m, int nlc, LmPool pl, hipStream_t st);

// bf16 backward: the four inputs widened to fp32 (exact), the three fp32 gradients rounded to
// bf16 (nearest even); count elements each, a multiple of 8, 16-byte aligned arrays.  With G
// NULL only Q, K, V are widened (the forward for m > 64); with gK NULL only gQ is rounded.
hipError_t launch_widen_bf16(const uint16_t* Q, const uint16_t* K, const uint16_t* V, const uint16_t* G, float* wQ,
                             float* wK, float* wV, float* wG, size_t count, hipStream_t st);
hipError_t launch_narrow_bf16(const float* gQ, const float* gK, const float* gV, uint16_t* dQ, uint16_t* dK,
                              uint16_t* dV, size_t count, hipStream_t st);

// bf16 fast forward path (fast.hip) -------------------------------------------------------

hipError_t launch_fast_pool(const void* Q, const void* K, const void* V, float* qt, float* kt, double* vseg,
                            float* segmax, float* vsegmax, int BH, int n, int d, int m, LmPool pl,
                            hipStream_t st);
hipError_t launch_fast_frame_ns(const float* qt, const float* kt, const double* vseg, const float* segmax,
                                const float* vsegmax, float* frame, uint32_t* qfix, uint32_t* kfix, float* vbar,
                                float* XT, float* cinfo, int BH, int n, int d, int m, float lambda, int T, float eps,
                                hipStream_t st);
// The same with the landmarks split over the waves (m > 48): blocks (h, kb) of the head's
// ntile = ceil(n / 128) tiles of 128 keys, tiles [kb ntile / nkb, (kb + 1) ntile / nkb); the
// launch also holds BH blocks that solve Newton-Schulz (T updates, eps) into XT and cinfo, from
// the code tables qfix, kfix (launch_fast_frame_ns writes only the frame when m > 48), and the
// query side's row bound: kcen [BH][d/2] (centre of the key-landmark codes) and frame[h][6] (its
// radius).
// The key blocks also form the value statistics (pool and frame leave them out for m > 48): the
// value sums per key block, vpart [BH][nkb][d], for launch_fast_mfinal's vbar.
hipError_t launch_fast_key2(const void* K, const void* V, const uint32_t* qfix, const uint32_t* kfix,
                            float* frame, float* Upart, float* vpart, float* XT, float* cinfo, uint32_t* kcen, int BH,
                            int n, int d, int m, int ntile, int nkb, int T, float eps, hipStream_t st);
hipError_t launch_fast_key(const void* K, const void* V, const uint32_t* qfix, const float* frame, float* Upart,
                           int BH, int n, int d, int m, int kpb, int nkb, hipStream_t st);
// mspace: the landmark-space normalisation (operand rows scaled by the whitening [H][m], NULL:
// ones; the ones column 1/m; mvec[BH][2][d] written as for launch_mspace_vec).  center (the
// inline normalisation): the operand columns are M[a][c] - M[a][d] vbar[c] (vbar [BH][d]), and M's
// value columns are not written.  With kfix (m <= 48) also the query side's row bound: kcen
// [BH][d/2] (centre of the key-landmark codes kfix) and frame[h][6] (its radius); NULL: formed by
// launch_fast_key2.  With vpart (m > 48), vbar is formed here from the key blocks' value sums
// (over n tokens) and written; otherwise it is read (launch_fast_frame_ns).
hipError_t launch_fast_mfinal(const float* Upart, const float* XT, _Float16* Mt, float* mscale, float* Mones,
                              float* M, int BH, int d, int m, int nkb, const float* whiten, int mspace, int H,
                              float* mvec, float* vbar, const float* vpart, int n, int center, const uint32_t* kfix,
                              uint32_t* kcen, float* frame, hipStream_t st);
// Query side: Out = normalise(K_QL M) (+ extra [BH][n][d] fp32 when given); with dwc_w, the 3 x 3
// convolution branch (filters [H][d][3][3], bias [H][d] or NULL, map width gw) formed from V in
// the epilogue instead.
hipError_t launch_fast_query(int norm, const void* Q, void* Out, const uint32_t* kfix, const uint32_t* kcen,
                             const float* frame, const _Float16* Mt, const float* mscale, const float* Mones,
                             const float* vbar, const float* extra, const float* mvec, int BH, int n, int d, int m,
                             const void* V, const float* dwc_w, const float* dwc_b, int gw, int H, hipStream_t st);

// Depth-wise convolution branch of Eq. (7) (dwc.hip) ------------------------------------------
// Filters W [H][d][k][k], bias [H][d] (may be NULL), over the row-major token map of width gw;
// k odd, at most 7.

// E = DWC(V) + bias, fp32 [BH][n][d]; V fp32 or bf16 (dt).
hipError_t launch_dwc_fwd(int dt, const void* V, const float* W, const float* bias, float* E, int BH, int H, int n,
                          int d, int gw, int k, hipStream_t st);
// dV += DWC^T(G), all fp32 [BH][n][d].
hipError_t launch_dwc_bwd_dv(const float* G, const float* W, float* dV, int BH, int H, int n, int d, int gw, int k,
                             hipStream_t st);
// dW [H][d][k][k] and db [H][d] (either may be NULL) of sum(DWC(V) * G), summed over the batch;
// part holds B*H*ceil(n/chunk)*d*(k*k+1) floats of per-chunk partial sums.
hipError_t launch_dwc_bwd_w(const float* G, const float* V, float* part, float* dW, float* db, int B, int H, int n,
                            int d, int gw, int k, int chunk, hipStream_t st);

}  // namespace lapattn
