/*
 * lapattn_oracle.h -- fp64 CPU oracle for Nystrom-approximated Laplacian-kernel
 * attention (LaplacianFormer, arXiv 2604.20368).
 *
 * TEST INFRASTRUCTURE ONLY.  This library exists so that tests, the smoke check
 * and the CPU-baseline leg of the benchmark can check the HIP path against a
 * plain, slow, obviously correct implementation.  Nothing in the product path
 * may link, load or call it.  It shares no code, header, table or constant with
 * the HIP library.
 *
 * Every array is fp64, contiguous, row-major.  Q, K, V, dOut and the gradients
 * are [B][H][n][d].  "BH" below means B*H independent heads.
 *
 * Readings of the paper this oracle takes (each is listed, with its reason, in
 * the design notes of the repository):
 *   R1  factor orientation  G^ = K_QL * NS(K_LL) * K_LK with
 *       K_QL[i][l] = k(q_i, kt_l), K_LL[a][b] = k(qt_a, kt_b), K_LK[a][j] = k(qt_a, k_j)
 *   R2  NS start X0 = K_LL^T / (||K_LL||_1 * ||K_LL||_inf), per head
 *   R3  perturbation eps of Algorithm 2 is an argument (0 by default)
 *   R4  row normalisation = the injective centring of Eq. (4) with Sigma^{-1/2} = I
 *   R5  landmarks = means of m balanced segments of consecutive tokens, or (when a
 *       token-map width is given) of the r x r windows of the H' x W' map
 *   R8  sign(0) = 0; argmax ties -> lowest index; gradient flows through X0's scale
 *   R9  T counts NS updates; T = 0 returns X0
 *   R10 if the X0 scale is 0, X_t := 0 for every t
 *   R14 the depth-wise convolution branch of Eq. (7): k x k filters, stride 1, zero padding
 *   R15 ORACLE_NORM_MSPACE: the landmark-space normalised embedding of Appendix B with its
 *       diagonal whitening w (per head, given; NULL = ones) in place of the query's landmark
 *       kernel vector: z_il = w_l (a_il - mean_l' a_il') + 1/m, Out_i = sum_l z_il M[l][:d]
 *   R16 the backward decides each sign(x - y) of the kernel gradient with the landmark mean
 *       y rounded to fp32 (the precision the GPU kernels hold landmarks in); the rest stays fp64
 */
#ifndef LAPATTN_ORACLE_H
#define LAPATTN_ORACLE_H

#ifdef __cplusplus
extern "C" {
#endif

enum { ORACLE_NORM_INLINE = 0, ORACLE_NORM_ROWSUM = 1, ORACLE_NORM_NONE = 2, ORACLE_NORM_MSPACE = 3 };

/* Laplacian kernel k(x, y) = exp(-||x - y||_1 / lambda)  (Sec. 1; Sec. 4.1). */
double lapattn_oracle_kernel(const double* x, const double* y, int d, double lambda);

/* Segment boundaries (R5): starts[l] = floor(l*n/m), l = 0..m (starts[m] = n). */
int lapattn_oracle_segments(int n, int m, int* starts);

/* Landmark membership: landmark l averages tokens members[starts[l] .. starts[l+1]).
 * grid_w = r = 0: the balanced segments of lapattn_oracle_segments (members[i] = i).
 * Otherwise the tokens form an H' x W' map in row-major order (W' = grid_w, H' = n / W')
 * and landmark l = Y (W'/r) + X averages the r x r window at rows Y r.., columns X r..
 * (Sec. 4.2, average pooling with kernel and stride r); r must divide H' and W' and
 * m must equal (H'/r)(W'/r).  starts has m + 1 entries, members n.  Returns nonzero
 * on invalid arguments. */
int lapattn_oracle_windows(int n, int m, int grid_w, int r, int* starts, int* members);

/* Newton-Schulz iteration of Algorithm 2 on one m x m matrix W (R2, R3, R9, R10).
 * Xs receives X_0 .. X_T, (T+1)*m*m doubles.  Returns the X0 scale c. */
double lapattn_oracle_ns(const double* W, int m, int T, double eps, double* Xs);

/* Forward pass.  Out is [B][H][n][d].  Every pointer after Out may be NULL;
 * when given they receive the per-head intermediates:
 *   Qt, Kt  [BH][m][d]     landmark means
 *   Wk      [BH][m][m]     K_LL (with eps on the diagonal)
 *   Xs      [BH][T+1][m][m] NS iterates X_0..X_T
 *   U       [BH][m][d+1]   K_LK * [V | 1]
 *   M       [BH][m][d+1]   X_T * U
 *   Y       [BH][n][d+1]   K_QL * M   (column d is the row sum s_i of G^)
 *   vbar    [BH][d]        mean of the values
 * grid_w, r select the landmark windows (lapattn_oracle_windows; 0, 0 = segments).
 * whiten [H][m] is the diagonal of ORACLE_NORM_MSPACE (NULL: ones; ignored by the other
 * normalisations).  Returns 0 on success, nonzero on a bad argument. */
int lapattn_oracle_forward(const double* Q, const double* K, const double* V, double* Out,
                           int B, int H, int n, int d, int m, double lambda, int T,
                           int norm, double eps, int grid_w, int r,
                           double* Qt, double* Kt, double* Wk, double* Xs,
                           double* U, double* M, double* Y, double* vbar, const double* whiten);

/* Backward pass: gradients of sum(Out * dOut) with respect to Q, K, V.
 * dQ, dK, dV are [B][H][n][d] and are overwritten.  Returns 0 on success. */
int lapattn_oracle_backward(const double* Q, const double* K, const double* V,
                            const double* dOut, double* dQ, double* dK, double* dV,
                            int B, int H, int n, int d, int m, double lambda, int T,
                            int norm, double eps, int grid_w, int r, const double* whiten);

/* Depth-wise convolution branch of Eq. (7), DWC(V) (reading R14): the n tokens of each head
 * form an H' x W' map in row-major order (W' = grid_w, H' = n / W'), and each value channel c
 * of head h is cross-correlated with its own k x k filter Wt[h][c] (k odd, stride 1, zero
 * padding (k-1)/2, so the output has the map's size), plus bias[h][c] (bias may be NULL):
 *   E[b][h][y W' + x][c] = bias[h][c] + sum_{u,t < k} Wt[h][c][u][t] V[b][h][(y+u-p) W' + x+t-p][c]
 * with p = (k-1)/2 and terms outside the map dropped.  Wt is [H][d][k][k], bias [H][d], V and
 * E [B][H][n][d]; E is overwritten.  Returns nonzero on invalid arguments. */
int lapattn_oracle_dwc(const double* V, const double* Wt, const double* bias, double* E,
                       int B, int H, int n, int d, int grid_w, int k);

/* Gradients of sum(E * dE) for E = DWC(V) above: dV (the convolution's part only,
 * [B][H][n][d]), dWt [H][d][k][k] and dbias [H][d] (summed over the batch), all overwritten. */
int lapattn_oracle_dwc_backward(const double* V, const double* Wt, const double* dE,
                                double* dV, double* dWt, double* dbias,
                                int B, int H, int n, int d, int grid_w, int k);

/* Number of OpenMP threads the oracle's parallel loops use. */
int lapattn_oracle_threads(void);

#ifdef __cplusplus
}
#endif
#endif
