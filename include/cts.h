/*
 * cts.h -- C ABI of the MI355X library for the batched multi-adapter linear
 * layer of "Compress then Serve: Serving Thousands of LoRA Adapters with
 * Little Overhead" (arXiv 2407.00066).
 *
 * The layer.  A batch holds T tokens; token t carries its own LoRA id
 * i(t) = adapter_id[t] (App. D: each request names the LoRA it wants).  The
 * n LoRAs were compressed offline into K clusters (Sec. 3.2); LoRA i belongs
 * to cluster k(i) = cluster_of[i], whose shared bases U_k, V_k are resident
 * on the GPU while Sigma_i is the LoRA's own r x r core (Sec. 3.1).  Then
 *
 *     y_t = W x_t + U_k Sigma_{i(t)} V_k^T x_t,        k = cluster_of[i(t)]
 *
 * i.e. (W_0 + Delta_i) x_t with Delta_i = U_k Sigma_i V_k^T (Sec. 3 and
 * Sec. 3.1 objective; the base term is computed once for the batch and the
 * adapter term per token, App. D).  The comparison path computes the same
 * layer with the uncompressed LoRAs, y_t = W x_t + B_i A_i x_t (Sec. 3).
 *
 * Layouts (row-major, element type given by cts_problem.dtype):
 *   x      [T][d_in]              W      [d_out][d_in]
 *   U      [K][d_out][r]          Vt     [K][r][d_in]   (V_k transposed)
 *   Sigma  [n][r][r]              applied as z' = Sigma_i z
 *   A      [n][r_lora][d_in]      B      [n][d_out][r_lora]
 *   y      [T][d_out]             element type cts_problem.out_dtype
 *   adapter_id int32 [T], cluster_of int32 [n]
 * There is no scale argument: a LoRA scale such as alpha/r is folded into
 * Sigma_i (or B_i) by the caller.
 *
 * Memory and ownership.  Every array pointer is DEVICE memory owned by the
 * caller; `p` is HOST memory, read during the call only.  Float arrays and
 * the workspace must be 16-byte aligned, id arrays 4-byte aligned (device
 * allocations are); a misaligned pointer is CTS_ERR_INVALID_ARG.  The library never
 * allocates, frees or synchronises in these calls: the caller provides a
 * device workspace of at least cts_workspace_size(p) (resp.
 * cts_workspace_size_uncompressed(p)) bytes, which may be reused between
 * calls on the same stream.  `stream` is a hipStream_t (NULL = the null
 * stream); calls only enqueue work on it and return.  Results are valid once
 * the stream has reached that point.  Concurrent calls need distinct
 * workspaces and outputs.
 *
 * Errors.  Every argument error is detected on the host before any HIP call
 * and reported by the return code; nothing is launched then.  T == 0 is a
 * valid no-op.  Device launch failures give CTS_ERR_HIP.  Ids are a
 * precondition like pointer validity in BLAS: 0 <= adapter_id[t] < n and
 * 0 <= cluster_of[i] < K.  The kernels clamp out-of-range ids so that they
 * never access memory outside the arrays, but the output rows of such tokens
 * are unspecified; cts_validate_ids checks the ids (synchronously).
 * A token that should see only the base layer can use an adapter whose
 * Sigma_i is zero: U_k * 0 adds exactly nothing.
 */
#ifndef CTS_H
#define CTS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    CTS_OK = 0,
    CTS_ERR_INVALID_ARG = 1,   /* null pointer, non-positive size, overlap */
    CTS_ERR_UNSUPPORTED = 2,   /* valid but outside this library's limits */
    CTS_ERR_WORKSPACE = 3,     /* workspace smaller than required */
    CTS_ERR_HIP = 4,           /* a HIP call or kernel launch failed */
    CTS_ERR_BAD_IDS = 5        /* cts_validate_ids found an id out of range */
} cts_status;

typedef enum { CTS_F32 = 0, CTS_BF16 = 1 } cts_dtype;

/* Problem description (host memory).  Limits (else CTS_ERR_UNSUPPORTED):
 *   T >= 0, d_in and d_out multiples of 8,
 *   r: multiple of 8 in [8, 128]; r_lora: multiple of 4 (f32) or 8 (bf16)
 *   in [4, 128]; 1 <= n_adapters <= 65536; 1 <= n_clusters <= 65536;
 *   dtype F32 with out_dtype F32, or dtype BF16 with out_dtype BF16 or F32.
 * Arithmetic: fp32 inputs are multiplied in fp32; bf16 inputs are multiplied
 * on bf16 matrix cores with fp32 accumulation; V^T x is kept in fp32, Sigma
 * is applied in fp32, and the result is rounded to the input type before the
 * U (or B) product.  Fields a call does not use are ignored (r, n_clusters
 * for the uncompressed path; r_lora for the compressed one).
 * Batches of more than 8192 tokens (the bucketing sorts at most 8192 tokens
 * in one workgroup) run as ceil(T / 8192) consecutive pieces of near-equal
 * size, the larger ones first, each a complete layer call on its rows of x,
 * adapter_id and y: every output row depends on its own token alone, so
 * the result is the whole batch's.  The workspace sizes cover the largest
 * piece; the bucketing read-back, cts_sort_by_cluster and
 * cts_apply_multi_sorted take at most 8192 tokens. */
typedef struct {
    int32_t T;            /* tokens in the batch */
    int32_t d_in;         /* input features of the layer */
    int32_t d_out;        /* output features of the layer */
    int32_t r;            /* rank of the shared bases U_k, V_k */
    int32_t n_adapters;   /* n: LoRAs in the collection */
    int32_t n_clusters;   /* K: clusters */
    int32_t r_lora;       /* rank of the uncompressed LoRAs (B_i, A_i) */
    int32_t dtype;        /* cts_dtype of x, W, U, Vt, Sigma, A, B */
    int32_t out_dtype;    /* cts_dtype of y */
} cts_problem;

/* Human-readable name of a status code (static storage, never NULL). */
const char* cts_status_string(int status);

/* Bytes of device workspace cts_apply needs for `p` (0 if p is invalid). */
size_t cts_workspace_size(const cts_problem* p);

/* Bytes of device workspace cts_apply_uncompressed needs for `p`. */
size_t cts_workspace_size_uncompressed(const cts_problem* p);

/* Debugging aid: where the bucketing of a call lies in its workspace.  Once
 * a cts_apply, cts_apply_diag, cts_apply_ranked or cts_apply_multi call
 * (compressed != 0; for cts_apply_multi, p with module 0's d_out) or a
 * cts_apply_uncompressed(_ranked) call (compressed == 0) for problem `p` has
 * completed, its workspace holds, at these byte offsets, the bucketing that
 * call used (the same as cts_sort_by_cluster's order):
 *   offsets[0]  int32 perm[T]     token of the j-th sorted position
 *   offsets[1]  int32 seg[T]      its cluster (uncompressed path: its adapter)
 *   offsets[2]  int32 aid[T]      its adapter
 *   offsets[3]  int32 items[c+1]  core-product items: the sorted positions
 *                                 where a run of one adapter starts or crosses
 *                                 a multiple of 16, ascending, then items[c] = T
 *   offsets[4]  int32 c           the number of items
 * `offsets` is a host array of 5 entries.  Returns CTS_ERR_INVALID_ARG or
 * CTS_ERR_UNSUPPORTED for a problem the call would refuse, and
 * CTS_ERR_UNSUPPORTED for T > 8192 (each piece of such a call overwrites
 * the bucketing of the one before). */
int cts_workspace_bucketing(const cts_problem* p, int32_t compressed, size_t* offsets);

/* Token bucketing (the grouping of tokens by cluster that makes the shared-
 * basis products contiguous GEMMs; Sec. 3.2 gives every LoRA of a cluster the
 * same U_k, V_k).  Sorts the tokens by the key (cluster_of[adapter_id[t]],
 * adapter_id[t], t), which is unique, so the result is exact and unique:
 *   perm[j]            = token with the j-th smallest key        (int32 [T])
 *   cluster_offsets[k] = number of tokens whose cluster is < k   (int32 [K+1])
 * cluster_of == NULL means every adapter is its own cluster (then K == n).
 * workspace: NULL, or device memory of at least cts_bucketing_size(T, n, K)
 * bytes (16-byte aligned), which then receives the rest of the bucketing the
 * layer uses (each sorted position's cluster and adapter, the runs of one
 * adapter and of one cluster): with perm, it is the `bucketing` argument of
 * cts_apply_multi_sorted, so that the modules of a whole model share one sort
 * per batch.  All arrays are device memory; T == 0 writes only
 * cluster_offsets (zeros).  Limits: T <= 8192, n and K <= 65536. */
size_t cts_bucketing_size(int32_t T, int32_t n, int32_t K);
int cts_sort_by_cluster(const int32_t* adapter_id, const int32_t* cluster_of,
                        int32_t T, int32_t n, int32_t K,
                        int32_t* perm, int32_t* cluster_offsets,
                        void* workspace, size_t workspace_bytes, void* stream);

/* Compressed multi-adapter layer: overwrites y[t] with
 * W x_t + U_k Sigma_i V_k^T x_t for every token (Sec. 3.1, 3.2, App. D).
 * y must not overlap any input or the workspace. */
int cts_apply(const cts_problem* p, const void* x, const int32_t* adapter_id,
              const int32_t* cluster_of, const void* W, const void* U,
              const void* Vt, const void* Sigma, void* y,
              void* workspace, size_t workspace_bytes, void* stream);

/* Diagonal-Sigma variant (Sec. 3.1, eq. JD-Diag; App. F): overwrites y[t]
 * with W x_t + U_k diag(sigma_i) V_k^T x_t.  Same arguments, layouts, limits,
 * workspace (cts_workspace_size) and errors as cts_apply, except that `sigma`
 * holds the diagonals only: sigma[n][r] in p->dtype (16-byte aligned), and
 * the core product is the elementwise scale z'_q = sigma_i[q] z_q (fp32,
 * rounded to the input type before the U_k product). */
int cts_apply_diag(const cts_problem* p, const void* x, const int32_t* adapter_id,
                   const int32_t* cluster_of, const void* W, const void* U,
                   const void* Vt, const void* sigma, void* y,
                   void* workspace, size_t workspace_bytes, void* stream);

/* Mixed ranks (Sec. 3.2: each cluster is given its own rank).  As cts_apply,
 * with U, Vt and Sigma stored at the largest rank p->r, and rank_of_cluster
 * (device int32 [K], 4-byte aligned) giving r_k: the layer uses
 * U_k[:, :r_k] Sigma_i[:r_k, :r_k] V_k^T[:r_k, :], and the stored entries past
 * r_k are never read into the result (they may hold anything, NaN included).
 * Each r_k must be a multiple of 8 in [0, p->r]; a value outside is clamped
 * into [0, p->r] and rounded down to a multiple of 8 (device contents are not
 * checked on the host).  Same workspace as cts_apply. */
int cts_apply_ranked(const cts_problem* p, const void* x, const int32_t* adapter_id,
                     const int32_t* cluster_of, const void* W, const void* U,
                     const void* Vt, const void* Sigma, const int32_t* rank_of_cluster,
                     void* y, void* workspace, size_t workspace_bytes, void* stream);

/* Uncompressed comparison path: overwrites y[t] with W x_t + B_i A_i x_t
 * (Sec. 3, first paragraph), i = adapter_id[t], rank p->r_lora. */
int cts_apply_uncompressed(const cts_problem* p, const void* x, const int32_t* adapter_id,
                           const void* W, const void* A, const void* B, void* y,
                           void* workspace, size_t workspace_bytes, void* stream);

/* Uncompressed LoRAs of different ranks (App. H): as cts_apply_uncompressed,
 * with A, B stored at the largest rank p->r_lora and rank_of_adapter (device
 * int32 [n], 4-byte aligned) giving r_i: the layer uses B_i[:, :r_i]
 * A_i[:r_i, :]; entries past r_i are never read into the result.  Each r_i
 * must be a multiple of 8 in [0, p->r_lora] (else clamped and rounded down,
 * as in cts_apply_ranked).  Same workspace as cts_apply_uncompressed. */
int cts_apply_uncompressed_ranked(const cts_problem* p, const void* x, const int32_t* adapter_id,
                                  const void* W, const void* A, const void* B,
                                  const int32_t* rank_of_adapter, void* y,
                                  void* workspace, size_t workspace_bytes, void* stream);

/* Multi-module batching: M projections of one layer that read the same x
 * (q, k and v, or gate and up) with the same LoRA per token and the same
 * cluster map.  Module m has its own W_m [d_out[m]][d_in], U_m
 * [K][d_out[m]][r] and Sigma_m [n][r][r]; the V_k^T of the modules come
 * stacked along r in one array Vt [K][M r][d_in] (rows m r .. m r + r - 1 of
 * cluster k are module m's V_k^T).  Then for every module
 *     y_m[t] = W_m x_t + U_k^(m) Sigma_i^(m) V_k^(m)T x_t
 * exactly as cts_apply with that module's arrays (Sec. 3.1, 3.2).  The
 * bucketing and the shrink run once for all modules (one GEMM over the M r
 * stacked rows, x read once), the core product and the fused GEMM once per
 * module.  d_out is a host array of M sizes; W, U, Sigma and y are host
 * arrays of M device pointers.  p->d_out is ignored; every other field of p
 * applies to all modules, and the limits of cts_apply hold per module, with
 * 1 <= M <= CTS_MAX_MODULES.  Outputs must not overlap each other, an input
 * or the workspace (cts_workspace_size_multi bytes). */
#define CTS_MAX_MODULES 8
size_t cts_workspace_size_multi(const cts_problem* p, int32_t M, const int32_t* d_out);
int cts_apply_multi(const cts_problem* p, int32_t M, const int32_t* d_out, const void* x,
                    const int32_t* adapter_id, const int32_t* cluster_of, const void* const* W,
                    const void* const* U, const void* Vt, const void* const* Sigma, void* const* y,
                    void* workspace, size_t workspace_bytes, void* stream);

/* cts_apply without a workspace argument, for callers that cannot allocate
 * device memory: code under HIP graph capture, tight serving loops and
 * harnesses that forbid allocation.  Same arguments (minus the workspace),
 * layouts, limits, results and errors as cts_apply; the call computes
 * exactly what cts_apply computes, with the same kernels.
 * Its scratch memory is one static device array of
 * CTS_NOALLOC_SCRATCH_BYTES bytes inside the library: every GPU the library
 * runs on holds its own copy of it until the process ends.  A problem whose
 * cts_workspace_size(p) exceeds that size is refused with
 * CTS_ERR_UNSUPPORTED before anything is launched.  The call allocates
 * nothing (no hipMalloc, hipFree or allocating library routine); its first
 * call on a device looks up that device's copy of the array (with the
 * stream's device current, as for every call).  All calls on one GPU share
 * that GPU's array: calls that overlap in time on one GPU (different
 * streams, or different host threads) race and give undefined results. */
#define CTS_NOALLOC_SCRATCH_BYTES (48u << 20)
int cts_apply_noalloc(const cts_problem* p, const void* x, const int32_t* adapter_id,
                      const int32_t* cluster_of, const void* W, const void* U,
                      const void* Vt, const void* Sigma, void* y, void* stream);

/* cts_apply_multi with a bucketing computed once for the batch by
 * cts_sort_by_cluster (perm and its workspace `bucketing`, bucketing_bytes
 * >= cts_bucketing_size(T, n, K)) instead of sorting the ids again: every
 * module of every layer of a model whose LoRAs share one cluster map
 * (Sec. 3.2) can take the same bucketing.  The sort must have been made with
 * p->T tokens, n = p->n_adapters and K = p->n_clusters and a cluster map
 * (not NULL), and have completed on `stream` (or a stream ordered before
 * it); the ids themselves are not arguments.  M = 1 is cts_apply's layer.
 * Same limits (and T <= 8192, the sort's), layouts, results and errors as
 * cts_apply_multi, and the same workspace (cts_workspace_size_multi bytes);
 * outputs must not overlap perm or the bucketing either. */
int cts_apply_multi_sorted(const cts_problem* p, int32_t M, const int32_t* d_out,
                           const int32_t* perm, const void* bucketing, size_t bucketing_bytes,
                           const void* x, const void* const* W, const void* const* U,
                           const void* Vt, const void* const* Sigma, void* const* y,
                           void* workspace, size_t workspace_bytes, void* stream);

/* cts_apply_multi (ids) or cts_apply_multi_sorted (a bucketing) writing one
 * packed output: the serving engine's fused projection output, into which
 * each module adds its slice (App. F's add_lora_slice_with_sigma writes the
 * columns [y_offset, y_offset + y_slice_size) of one y).  Module m writes
 * the columns [c_m, c_m + d_out[m]) of every row of y, c_m = d_out[0] + ... +
 * d_out[m-1]; the rows are ldy elements apart (ldy >= the sum of d_out, a
 * multiple of 8; y 16-byte aligned), and columns past the sum are left
 * untouched.  Exactly one of the pairs (adapter_id, cluster_of) and (perm,
 * bucketing) is given (the other NULL).  Same problem limits, workspace
 * (cts_workspace_size_multi), results and errors as the two calls it merges;
 * the packed range y[0 .. (T-1) ldy + sum of d_out) must not overlap an
 * input or the workspace. */
int cts_apply_multi_packed(const cts_problem* p, int32_t M, const int32_t* d_out,
                           const int32_t* adapter_id, const int32_t* cluster_of,
                           const int32_t* perm, const void* bucketing, size_t bucketing_bytes,
                           const void* x, const void* const* W, const void* const* U,
                           const void* Vt, const void* const* Sigma, void* y, int32_t ldy,
                           void* workspace, size_t workspace_bytes, void* stream);

/* Synchronous id check for tests and debugging: copies the ids to the host
 * (waiting for `stream`) and returns CTS_ERR_BAD_IDS if any adapter_id is
 * outside [0, n) or any cluster_of outside [0, K) (cluster_of may be NULL). */
int cts_validate_ids(const cts_problem* p, const int32_t* adapter_id,
                     const int32_t* cluster_of, void* stream);

/* Profiling aid; correct use of the library never needs it.
 * events == NULL turns it off.  Otherwise `events` is a host array of
 * CTS_N_STAGE_EVENTS hipEvent_t handles owned by the caller (a NULL entry is
 * skipped); the handles are copied, and every later cts_apply /
 * cts_apply_uncompressed call records them on its stream at the stage
 * boundaries of the layer:
 *   [0] before the bucketing          [1] before the shrink V_k^T X
 *   [2] before the core product       [3] before the fused W X + U_k Z' GEMM
 *   [4] after the fused GEMM          [5] after the split-K reduction
 *                                         (right after [4] when there is none)
 * The setting is process-wide; changing it while another thread is inside a
 * cts_apply call is a race. */
#define CTS_N_STAGE_EVENTS 6
int cts_set_stage_events(void* const* events);

#ifdef __cplusplus
}
#endif

#endif /* CTS_H */
