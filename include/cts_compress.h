/*
 * cts_compress.h -- C ABI of the offline compressor of "Compress then Serve"
 * (arXiv 2407.00066): joint diagonalization of a LoRA collection (Sec. 3.1,
 * App. A.1 case 1, App. A.2) and its clustering (Sec. 3.2, App. A.3), on the
 * GPU.  It turns LoRAs (A_i, B_i) into the shared bases U_k, V_k, the cores
 * Sigma_i and the cluster map that cts_apply (cts.h) serves.
 *
 * Layouts (row-major, fp32, device memory owned by the caller, 16-byte
 * aligned; id arrays int32, 4-byte aligned):
 *   A      [n][r_lora][d_in]      B      [n][d_out][r_lora]   (update B_i A_i)
 *   U      [d_out][r]             Vt     [r][d_in]            (V transposed)
 *   Sigma  [n][r][r]              Sigma_i = U^T B_i A_i V (eq. sigmastar)
 * With K clusters the bases are U [K][d_out][r] and Vt [K][r][d_in], the
 * layouts cts_apply takes (after conversion to its element type).
 *
 * Arithmetic is fp32: the large products run on fp32 matrix cores with fp32
 * accumulation; sums over the collection are split in a fixed order, so
 * results are bitwise reproducible on one GPU.
 *
 * Errors: every argument error is detected on the host before any launch
 * (CTS_ERR_INVALID_ARG / CTS_ERR_UNSUPPORTED / CTS_ERR_WORKSPACE of cts.h);
 * a failed launch or copy is CTS_ERR_HIP.  The compressor calls are offline
 * work: they may wait for the stream (stated per call); they never allocate.
 * Inputs with fewer than r independent directions (n * r_lora < r, or
 * degenerate LoRAs) make the orthogonalization divide by zero: results are
 * then NaN.
 *
 * Profiling: while the stage events of cts_set_stage_events (cts.h) are on,
 * every iteration of the JD records [1] before and [2] after its projection
 * kernels (P_i = A_i V, Q_i = B_i^T U, then the per-LoRA products) and [3]
 * after its expansion kernel (the sums over the collection); the last
 * iteration's records are the ones left.  cts_jd_diag records the same
 * three events around its U step's projection (C_i = P_i S_i; P_i = A_i V
 * comes from the preceding diagonal step unless the normalization rescaled
 * V since) and expansion kernel (sum_i B_i C_i, before the sum of its
 * pieces).
 */
#ifndef CTS_COMPRESS_H
#define CTS_COMPRESS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Limits (else CTS_ERR_UNSUPPORTED): 1 <= n <= 65536; r_lora in {4, 8, 16,
 * 32, 64}; r in {16, 32, 48, 64, 96, 128} with r <= n * r_lora; d_in and
 * d_out multiples of 4 in [r, 65536]; every array below 2^31 elements. */
typedef struct {
    int32_t n;        /* LoRAs in the collection */
    int32_t d_out;    /* rows of B_i (output features of the layer) */
    int32_t d_in;     /* columns of A_i (input features) */
    int32_t r_lora;   /* rank of the LoRAs */
    int32_t r;        /* rank of the joint diagonalization */
} cts_jd_problem;

/* Bytes of device workspace cts_jd_full needs (0 if p is invalid). */
size_t cts_jd_workspace_size(const cts_jd_problem* p);

/* Bytes of device workspace cts_jd_cluster needs for K clusters. */
size_t cts_jd_cluster_workspace_size(const cts_jd_problem* p, int32_t K);

/* ||B_i A_i||_F^2 for every LoRA (via the r_lora x r_lora Gram matrices
 * B_i^T B_i and A_i A_i^T): norms2 [n], device.  Does not wait. */
int cts_lora_norms2(const cts_jd_problem* p, const float* A, const float* B, float* norms2,
                    void* workspace, size_t workspace_bytes, void* stream);

/* JD-Full by the eigenvalue iteration of App. A.2: from the orthonormal pair
 * (U0, Vt0), each iteration forms
 *     U' = sum_i B_i (A_i V)(V^T A_i^T)(B_i^T U),
 *     V' = sum_i A_i^T (B_i^T U)(U^T B_i)(A_i V)
 * from the previous pair and orthogonalizes both (Q of the QR factorization
 * with positive diag(R), by CholeskyQR2).  crit [iters] (device) receives the
 * convergence measure of App. H (convergence) after each iteration:
 *     max over X in {U, V} of ||X_t+1 - X_t X_t^T X_t+1||_F / ||X_t+1||_F.
 * tau > 0 stops after the first iteration whose measure is below tau (the
 * call then waits for the stream after every iteration); tau <= 0 runs all
 * `iters` iterations without waiting.  normalize != 0 applies the Frobenius
 * normalization of Sec. 6.1 (every B_i A_i weighted to unit norm inside the
 * iteration) and restores the norms in Sigma.  Outputs: U, Vt, Sigma = U^T
 * B_i A_i V for every LoRA; *iters_done (host, may be NULL) the number of
 * iterations run.  U0/Vt0 may alias U/Vt.  iters >= 1. */
int cts_jd_full(const cts_jd_problem* p, const float* A, const float* B, const float* U0,
                const float* Vt0, int32_t iters, float tau, int32_t normalize, float* U, float* Vt,
                float* Sigma, float* crit, int32_t* iters_done, void* workspace,
                size_t workspace_bytes, void* stream);

/* JD-Diag by the alternating least squares of App. A.1 case 2: unconstrained
 * U, V (r columns) and diagonal cores.  From (U0, Vt0) the diagonals are solved
 * first, sigma_i = (U^T U o V^T V)^-1 (U^T B_i o V^T A_i^T) 1; then each of
 * `sweeps` sweeps solves U = (sum_i B_i A_i V S_i)(sum_i S_i V^T V S_i)^-1,
 * then V likewise with the new U, then the diagonals again (S_i =
 * diag(sigma_i)).  normalize != 0 then rescales the diagonals to
 * sum_i ||sigma_i||^2 = 1 and multiplies U and V by the square root of the
 * removed factor (every U diag(sigma_i) V^T unchanged).  The r x r systems
 * are solved by Cholesky (columns equilibrated).  Outputs U [d_out][r], Vt
 * [r][d_in], sigma [n][r] (the cores cts_apply_diag serves).  Same workspace
 * as cts_jd_full.  Does not wait.  sweeps >= 0. */
int cts_jd_diag(const cts_jd_problem* p, const float* A, const float* B, const float* U0,
                const float* Vt0, int32_t sweeps, int32_t normalize, float* U, float* Vt,
                float* sigma, void* workspace, size_t workspace_bytes, void* stream);

/* Cores for given orthonormal bases (eq. sigmastar): Sigma_i = U^T B_i A_i V
 * for every LoRA.  Same workspace as cts_jd_full.  Does not wait. */
int cts_jd_sigma(const cts_jd_problem* p, const float* A, const float* B, const float* U,
                 const float* Vt, float* Sigma, void* workspace, size_t workspace_bytes,
                 void* stream);

/* Clustering of App. A.3.  A single-basis JD-Full (jd_iters iterations from
 * U0, Vt0), k-means on vec(Sigma_i) from the centroids of the LoRAs
 * init_idx[K] (host array; Lloyd iterations until no label changes, at most
 * 100), then rounds of per-cluster JD-Full (each from Uc0[k], Vtc0[k]) and
 * reassignment of every LoRA to the cluster maximizing ||U_k^T B_i A_i V_k||_F
 * (= minimizing min_S ||B_i A_i - U_k S V_k^T||_F), until no LoRA moves or
 * after max_rounds rounds.  Ties go to the lowest index; an empty cluster
 * keeps its centroid and bases.  A cluster whose m members supply fewer than
 * r directions (m * r_lora < r) gets, in place of the per-cluster JD, the
 * positive-diagonal QR factors of [B_{i_1} ... B_{i_m} | Uc0[k][:, :q]] and
 * [A_{i_1}^T ... A_{i_m}^T | Vc0[k][:, :q]] (members in increasing id order,
 * q = r - m r_lora): bases that contain every member's columns and so
 * reconstruct the members exactly (Prop. 1), a minimizer of Step 1.
 * Outputs: cluster_of [n] (device int32), U [K][d_out][r], Vt [K][r][d_in],
 * Sigma [n][r][r] (each LoRA's core in its own cluster's bases), *rounds
 * (host, may be NULL).  normalize as in cts_jd_full.  Waits for the stream
 * (the control flow depends on results).  Uc0, Vtc0: [K][d_out][r],
 * [K][r][d_in]; 1 <= K <= n. */
int cts_jd_cluster(const cts_jd_problem* p, int32_t K, const float* A, const float* B,
                   const float* U0, const float* Vt0, const float* Uc0, const float* Vtc0,
                   const int32_t* init_idx, int32_t jd_iters, int32_t max_rounds,
                   int32_t normalize, int32_t* cluster_of, float* U, float* Vt, float* Sigma,
                   int32_t* rounds, void* workspace, size_t workspace_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* CTS_COMPRESS_H */
