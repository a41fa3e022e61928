/*
 * lapattn.h -- C ABI of the MI355X (gfx950) library for Nystrom-approximated
 * Laplacian-kernel attention (LaplacianFormer, arXiv 2604.20368).
 *
 * Per head (b, h), with q_i, k_j, v_j the rows of Q, K, V (n x d):
 *   k(x, y)   = exp(-||x - y||_1 / lambda)                 Sec. 1; Sec. 4.1; Eq. (8)
 *   landmarks qt_l, kt_l = means of the tokens of segment l,
 *             segment l = [floor(l n/m), floor((l+1) n/m))  Sec. 4.2, sampling (1-D reading)
 *   K_LL[a][b] = k(qt_a, kt_b)                              Algorithm 1, kernel on sampled points
 *   K_QL[i][l] = k(q_i, kt_l)                               Eq. (8), cross-kernel
 *   K_LK[a][j] = k(qt_a, k_j)
 *   X_T       = Newton-Schulz iterate of Algorithm 2 on W = K_LL + eps I:
 *               X_0 = W^T / (||W||_1 ||W||_inf),  X_{t+1} = X_t (2I - W X_t);
 *               X := 0 when the scale ||W||_1 ||W||_inf is 0
 *   G^        = K_QL X_T K_LK  (never formed: Y = K_QL (X_T (K_LK [V | 1])))
 *   s_i       = (G^ 1)_i,  vbar = mean_j v_j
 *   Out_i     = LAPATTN_NORM_INLINE:  (G^ V)_i + (1 - s_i) vbar
 *                 i.e. Z V with z_ij = g^_ij - s_i/n + 1/n, the injective centring
 *                 of Eq. (4) with the whitening taken as the identity
 *               LAPATTN_NORM_ROWSUM:  (G^ V)_i / s_i       (Eq. (3))
 *               LAPATTN_NORM_NONE:    (G^ V)_i
 *               LAPATTN_NORM_MSPACE:  sum_l z_il M[l][:d],  M = X_T (K_LK V),
 *                 z_il = w_l (a_il - mean_l' a_il') + 1/m with a_il = K_QL[i][l]: the
 *                 landmark-space normalised embedding of Appendix B, whose m x m diagonal
 *                 whitening w is given per head (lapattn_opts.whiten)
 * Optional depth-wise convolution branch of Eq. (7), off by default (lapattn_opts.dwc_k):
 *   Out_i += DWC(V)_i, each value channel of each head cross-correlated over the token map
 *   with its own k x k filter (stride 1, zero padding (k-1)/2) plus a per-channel bias.
 *
 * Layout: Q, K, V, Out, dOut, dQ, dK, dV are device pointers to contiguous
 * row-major [B][H][n][d] arrays of the element type `dtype` (fp32, or bf16 as
 * raw 16-bit patterns).  The value head dimension equals d.
 *
 * Ownership: the caller owns every buffer, including the workspace (device
 * memory of at least lapattn_workspace_size() bytes).  The library never
 * allocates or frees device memory and keeps no state between calls apart from
 * the optional timing switch below.  Outputs are overwritten, never accumulated.
 * Outputs must not alias inputs, each other, or the workspace.  Every tensor
 * pointer must be 16-byte aligned and the workspace 256-byte aligned (device
 * allocations are; offset views may not be).
 *
 * Asynchrony: every call validates its arguments on the host, enqueues its
 * kernels on `stream` (a hipStream_t; NULL = the default stream) and returns
 * without synchronising.  Results are valid once the stream has reached that
 * point.  Calls on different streams with different workspaces may run
 * concurrently; calls sharing a workspace must be ordered by the caller.
 * Results are bitwise deterministic for identical inputs (no float atomics).
 *
 * Errors: a nonzero return means nothing was enqueued and nothing was written,
 * except LAPATTN_ERR_HIP, which reports a failed kernel launch (work enqueued
 * before the failure may have run).  No C++ exception crosses this interface.
 */
#ifndef LAPATTN_H
#define LAPATTN_H

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ihipStream_t* lapattn_stream_t;   /* the same type as hipStream_t */

typedef enum { LAPATTN_FP32 = 0, LAPATTN_BF16 = 1 } lapattn_dtype;

typedef enum {
    LAPATTN_NORM_INLINE = 0,
    LAPATTN_NORM_ROWSUM = 1,
    LAPATTN_NORM_NONE = 2,
    LAPATTN_NORM_MSPACE = 3
} lapattn_norm;

enum {
    LAPATTN_OK = 0,
    LAPATTN_ERR_NULL = 1,         /* a required pointer is NULL */
    LAPATTN_ERR_SHAPE = 2,        /* B, H, n < 1, m < 1, m > n, B*H*n*d >= 2^31, n not a
                                     multiple of grid_w, or landmark windows that do not tile
                                     the token map (lapattn_opts) */
    LAPATTN_ERR_PARAM = 3,        /* lambda not finite or <= 0, ns_iters outside [0, 64],
                                     eps not finite or < 0, unknown norm or dtype,
                                     window options negative or pool_r without grid_w,
                                     dwc_k not 0, 1, 3, 5 or 7, or dwc_k without grid_w */
    LAPATTN_ERR_UNSUPPORTED = 4,  /* d not in {32, 64} or m > 128 */
    LAPATTN_ERR_WORKSPACE = 5,    /* workspace NULL or smaller than lapattn_workspace_size() */
    LAPATTN_ERR_HIP = 6,          /* a HIP launch failed */
    LAPATTN_ERR_ALIGN = 7,        /* a tensor pointer is not 16-byte aligned, or the
                                     workspace is not 256-byte aligned */
    LAPATTN_ERR_SCRATCH = 8       /* lapattn_forward_noalloc: the call needs more workspace
                                     than the library's static scratch array holds (32 MiB) */
};

/* Options; a NULL pointer means all fields zero: {LAPATTN_NORM_INLINE, 0.0f, 0, 0, 0, NULL, ...}.
 * eps is the diagonal perturbation W <- W + eps I of Algorithm 2 (>= 0).
 * Token map: with grid_w > 0 the n tokens form a row-major H' x W' map (W' = grid_w,
 * H' = n / W'; n must be a multiple of W', LAPATTN_ERR_SHAPE otherwise).
 * Landmarks (Sec. 4.2, sampling): with pool_r = 0 they are the means of m balanced
 * segments of consecutive tokens, [floor(l n/m), floor((l+1) n/m)).  With pool_r = r > 0
 * they are the means of the map's r x r windows (average pooling with kernel and stride r),
 * landmark l = Y (W'/r) + X for the window at rows Y r.., columns X r..; this needs
 * grid_w > 0 (LAPATTN_ERR_PARAM), r dividing H' and W', and m = (H'/r)(W'/r)
 * (LAPATTN_ERR_SHAPE).  Negative values are LAPATTN_ERR_PARAM.
 * Convolution branch (Eq. (7)): dwc_k = k in {1, 3, 5, 7} adds DWC(V) to Out:
 *   Out[b][h][y W' + x][c] += dwc_b[h][c]
 *       + sum_{u,t < k} dwc_w[h][c][u][t] V[b][h][(y+u-p) W' + x+t-p][c],  p = (k-1)/2,
 * terms outside the map dropped; it needs grid_w > 0 (LAPATTN_ERR_PARAM) and dwc_w
 * (LAPATTN_ERR_NULL), and the workspace sized with LAPATTN_WS_DWC.  dwc_w is a device array
 * [H][d][k][k] of fp32 and dwc_b [H][d] fp32 or NULL (no bias), shared by the batch, for
 * either dtype.  lapattn_backward adds the branch's part to dV and, when the pointers are
 * not NULL, writes the filter gradient dwc_dw [H][d][k][k] and the bias gradient dwc_db [H][d]
 * (fp32, summed over the batch, overwritten); lapattn_forward ignores those two.
 * whiten: with LAPATTN_NORM_MSPACE, the diagonal whitening w as a device array [H][m] of fp32
 * shared by the batch (NULL: all ones); ignored by the other normalisations.
 * save (fp32 inputs; ignored for bf16): lapattn_forward keeps the landmark means, the key-side
 * summary, every Newton-Schulz iterate and the n x m kernel values of both sides (K_QL and
 * K_LK^T, 64 floats per token for each group of 64 landmarks) in the workspace, which must
 * then be sized with LAPATTN_WS_BACKWARD; a following lapattn_backward with save set and the same inputs, sizes,
 * options and workspace (the caller orders the two calls) reuses them instead of recomputing
 * them.  Results are bitwise those of the calls without save. */
typedef struct {
    int norm;            /* lapattn_norm */
    float eps;
    int grid_w;          /* token-map width W', or 0: no map */
    int pool_r;          /* landmark window side r, or 0 for segments */
    int dwc_k;           /* convolution filter side k, or 0: no convolution branch */
    const float* dwc_w;  /* device [H][d][k][k] filters */
    const float* dwc_b;  /* device [H][d] bias, or NULL */
    float* dwc_dw;       /* backward: device [H][d][k][k] filter gradient, or NULL */
    float* dwc_db;       /* backward: device [H][d] bias gradient, or NULL */
    const float* whiten; /* LAPATTN_NORM_MSPACE: device [H][m] diagonal whitening, or NULL */
    int save;            /* 1: forward leaves its internals for the backward (see above) */
} lapattn_opts;

/* Workspace flags. */
enum { LAPATTN_WS_BACKWARD = 1, LAPATTN_WS_DWC = 2 };

/* Bytes of device workspace that lapattn_forward (flags without LAPATTN_WS_BACKWARD) or
 * lapattn_backward (with it) needs for these sizes, with LAPATTN_WS_DWC when the call uses
 * the convolution branch; 0 if the sizes or flags are invalid.  Pure host function, callable
 * without a GPU. */
size_t lapattn_workspace_size(int B, int H, int n, int d, int m, int ns_iters,
                              int dtype, int flags);

/* Forward pass (Algorithm 1 with Algorithm 2 as the pseudoinverse, the
 * key-summary reordering of Sec. 3.2, and the normalisation chosen in opts).
 * lambda > 0 is the kernel scale, m the number of landmarks (1 <= m <= min(n, 128)),
 * ns_iters the number T of Newton-Schulz updates (T = 0 uses X_0).  dtype = LAPATTN_BF16
 * computes from the bf16 inputs directly for m <= 64 (fixed-point L1 distances, fp16 matrix
 * cores, fp32 accumulation); for m > 64 it runs the fp32 computation on the exactly widened
 * inputs and rounds the output to bf16 (nearest even).  fp32 heads with n <= 256, m <= 32 and
 * no convolution branch, saved state or landmark-space form run in one workgroup per head,
 * with the L1 distances in 32-bit fixed point on one grid per head (grid step at most
 * 2^-21 max|Q, K|).  On these two paths (bf16, and the fp32 small heads) a NaN or infinity in
 * Q or K makes every output of its head NaN. */
int lapattn_forward(const void* Q, const void* K, const void* V, void* Out,
                    int B, int H, int n, int d, int m, float lambda, int ns_iters,
                    int dtype, const lapattn_opts* opts,
                    void* workspace, size_t workspace_bytes, lapattn_stream_t stream);

/* Backward pass: dQ, dK, dV = gradients of sum(Out * dOut) with respect to
 * Q, K, V, through the landmark means, the three kernel blocks and every
 * Newton-Schulz update including the scale of X_0 (kernel gradient of App. A,
 * with sign(0) = 0 and each sign decided on the landmark means as held in fp32;
 * ties in the norm maxima go to the lowest index).  Without opts->save the
 * forward internals are recomputed here; with it (fp32 inputs) they are read from
 * the workspace left by a lapattn_forward call with save set (see lapattn_opts).
 * dtype = LAPATTN_BF16 runs the fp32 computation on the exactly widened bf16
 * inputs (held in the workspace, which is correspondingly larger) and rounds the
 * three gradients to bf16 (nearest even); dQ, dK, dV are in the input dtype. */
int lapattn_backward(const void* Q, const void* K, const void* V, const void* dOut,
                     void* dQ, void* dK, void* dV,
                     int B, int H, int n, int d, int m, float lambda, int ns_iters,
                     int dtype, const lapattn_opts* opts,
                     void* workspace, size_t workspace_bytes, lapattn_stream_t stream);

/* Forward pass without a caller workspace, for callers that cannot allocate device memory:
 * code under HIP graph capture, tight serving loops, harnesses that forbid hipMalloc.
 * Arguments, results and errors as lapattn_forward, whose kernels it runs on a static device
 * array of the library (32 MiB per GPU, held by every GPU the library runs on until the process
 * ends) in place of the workspace; it calls no allocating routine.  A call whose
 * lapattn_workspace_size (with LAPATTN_WS_DWC when opts->dwc_k is set) exceeds 32 MiB returns
 * LAPATTN_ERR_SCRATCH, and opts->save returns LAPATTN_ERR_PARAM (the saved state would sit in
 * the shared array), both before anything is enqueued.  All calls on one GPU share its array:
 * calls that overlap on one GPU (other streams, other threads) race and must be ordered by the
 * caller.  The first call on each device looks up that device's array (with the device
 * current). */
int lapattn_forward_noalloc(const void* Q, const void* K, const void* V, void* Out,
                            int B, int H, int n, int d, int m, float lambda, int ns_iters,
                            int dtype, const lapattn_opts* opts, lapattn_stream_t stream);

/* Human-readable name of a status code (static storage). */
const char* lapattn_status_str(int status);

/* Kernel timing (a measurement aid).  lapattn_timing_enable(1) clears the record
 * and makes every following forward/backward call record a HIP event pair around
 * each kernel it launches, on the caller's stream; lapattn_timing_enable(0) stops
 * recording (the record is kept).  lapattn_timing_read() waits for the recorded
 * events, writes up to `cap` per-launch durations in milliseconds (launch order,
 * over all calls since timing was enabled) into ms, and returns the number of
 * recorded launches (-1 on a HIP error).  lapattn_timing_name(i) names launch i
 * (static storage; "" when out of range).  Timing is process-wide state guarded
 * by a mutex and adds two event records per kernel: keep it off outside
 * measurement.  Returns of lapattn_timing_enable: the previous setting. */
int lapattn_timing_enable(int enable);
int lapattn_timing_read(float* ms, int cap);
const char* lapattn_timing_name(int index);

#ifdef __cplusplus
}
#endif
#endif /* LAPATTN_H */
