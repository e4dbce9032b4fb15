/*
 * cts_oracle.c -- plain, slow, fp64 CPU oracle for the batched multi-adapter
 * linear layer of "Compress then Serve" (arXiv 2407.00066).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the CPU
 * baseline leg of the benchmark may load this library.  It shares no code,
 * header or constant with the HIP library: it includes only the C standard
 * library and OpenMP.
 *
 * What it computes is the plain definition, not the fast factored route:
 *
 *   Sec. 3, first paragraph: a LoRA-updated layer maps x to (W_0 + B A) x.
 *   Sec. 3.1 (JD): the product B_i A_i is replaced by U Sigma_i V^T with U, V
 *     shared and Sigma_i an r x r matrix owned by LoRA i.
 *   Sec. 3.2 (clustering): LoRA i in cluster C_j uses that cluster's U_j, V_j.
 *   App. D: the base term W_0 x is computed once and the adapter term per
 *     request; the factored order V^T x -> Sigma(.) -> U(.) is only a cheaper
 *     route to the same value.
 *
 * So, per token t with adapter i = adapter_id[t] and cluster k = cluster_of[i]:
 *     Delta_i = U_k Sigma_i V_k^T            (formed explicitly, d_out x d_in)
 *     y_t     = (W + Delta_i) x_t
 * and, for the uncompressed comparison path, Delta_i = B_i A_i.
 * Sec. 3.1, the diagonal variant (eq. JD-Diag): Sigma_i is diagonal, given as
 * its r diagonal entries sigma_i, and Delta_i = U_k diag(sigma_i) V_k^T.
 * Mixed ranks (Sec. 3.2: each cluster is given its own rank; App. H: LoRAs of
 * different ranks): arrays are stored at the largest rank, cluster k uses its
 * first r_k columns of U_k, rows of V_k^T and the leading r_k x r_k block of
 * Sigma_i, and uncompressed adapter i its first r_i columns of B_i and rows
 * of A_i; the stored entries past those ranks are never read.
 *
 * Array layouts (row-major, all host memory, all double):
 *   x      [T][d_in]            W      [d_out][d_in]
 *   U      [K][d_out][r]        Vt     [K][r][d_in]   (V_k^T, same as a LoRA A)
 *   Sigma  [n][r][r]            (applied as z' = Sigma_i z)
 *   sigma  [n][r]               (diagonal variant: z'_q = sigma_i[q] z_q)
 *   A      [n][r_l][d_in]       B      [n][d_out][r_l]
 *   y      [n_tok][d_out]       rows follow the order of `tokens`
 *
 * Every sum is accumulated in double in ascending index order.  No blocking,
 * no reordering beyond "adapters ascending, then their tokens ascending",
 * which only decides when a Delta_i is (re)formed, never how a value is summed.
 *
 * Error behaviour: every function returns 0 on success and a negative code on
 * a bad argument (-1) or an id out of range (-2); it never aborts.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

int cts_oracle_num_threads(void) {
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* ------------------------------------------------------------------------ */
/* Bucketing.  The paper has no sort: grouping requests by adapter is prior
 * art it cites (Punica's segmented gather, Sec. 2) and grouping by cluster is
 * its proposed scheduling direction (Sec. 7).  The key used here is the
 * lexicographic triple (cluster_of[adapter_id[t]], adapter_id[t], t); the
 * token index makes every key distinct, so exactly one order is correct.   */

typedef struct { int64_t c, a, t; } sort_key;

static int key_cmp(const void* pa, const void* pb) {
    const sort_key* p = (const sort_key*)pa;
    const sort_key* q = (const sort_key*)pb;
    if (p->c != q->c) return p->c < q->c ? -1 : 1;
    if (p->a != q->a) return p->a < q->a ? -1 : 1;
    if (p->t != q->t) return p->t < q->t ? -1 : 1;
    return 0;
}

/* perm[j] = token with the j-th smallest key; offsets[k] = number of tokens
 * whose cluster is < k, for k = 0..K (so offsets[K] == T).
 * cluster_of == NULL means "every adapter is its own cluster" (K must be n). */
int cts_oracle_sort_by_cluster(const int32_t* adapter_id, int64_t T,
                               const int32_t* cluster_of, int64_t n, int64_t K,
                               int32_t* perm, int32_t* offsets) {
    if (T < 0 || n < 1 || K < 1) return -1;
    if (cluster_of == NULL && K != n) return -1;
    sort_key* keys = (sort_key*)malloc(sizeof(sort_key) * (size_t)(T > 0 ? T : 1));
    if (!keys) return -1;
    for (int64_t t = 0; t < T; ++t) {
        int64_t a = adapter_id[t];
        if (a < 0 || a >= n) { free(keys); return -2; }
        int64_t c = cluster_of ? cluster_of[a] : a;
        if (c < 0 || c >= K) { free(keys); return -2; }
        keys[t].c = c; keys[t].a = a; keys[t].t = t;
    }
    qsort(keys, (size_t)T, sizeof(sort_key), key_cmp);
    for (int64_t j = 0; j < T; ++j) perm[j] = (int32_t)keys[j].t;
    for (int64_t k = 0; k <= K; ++k) {
        int64_t cnt = 0;
        for (int64_t t = 0; t < T; ++t) cnt += (keys[t].c < k);
        offsets[k] = (int32_t)cnt;
    }
    free(keys);
    return 0;
}

/* ------------------------------------------------------------------------ */
/* Dense helpers: C[m][p] = sum_q A[m][q] * B[q][p], ascending q.            */

static void matmul(const double* A, const double* B, double* C,
                   int64_t m, int64_t q, int64_t p) {
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < m; ++i) {
        double* ci = C + i * p;
        for (int64_t c = 0; c < p; ++c) ci[c] = 0.0;
        for (int64_t s = 0; s < q; ++s) {
            const double a = A[i * q + s];
            const double* bs = B + s * p;
            for (int64_t c = 0; c < p; ++c) ci[c] += a * bs[c];
        }
    }
}

/* y_row[o] = sum_c (W[o][c] + D[o][c]) * x[c], ascending c. */
static void apply_rows(const double* W, const double* D, const double* x,
                       double* y_row, int64_t d_out, int64_t d_in) {
    #pragma omp parallel for schedule(static)
    for (int64_t o = 0; o < d_out; ++o) {
        const double* w = W + o * d_in;
        const double* d = D + o * d_in;
        double acc = 0.0;
        for (int64_t c = 0; c < d_in; ++c) acc += (w[c] + d[c]) * x[c];
        y_row[o] = acc;
    }
}

/* Order in which the requested tokens are visited: adapter ascending, then
 * position in `tokens` ascending.  Returns a malloc'd index list. */
static int64_t* visit_order(const int32_t* adapter_id, const int64_t* tokens,
                            int64_t n_tok, int64_t n) {
    int64_t* order = (int64_t*)malloc(sizeof(int64_t) * (size_t)(n_tok > 0 ? n_tok : 1));
    if (!order) return NULL;
    int64_t w = 0;
    for (int64_t a = 0; a < n; ++a)
        for (int64_t s = 0; s < n_tok; ++s)
            if (adapter_id[tokens[s]] == a) order[w++] = s;
    return order;
}

static int check_tokens(const int32_t* adapter_id, int64_t T, const int64_t* tokens,
                        int64_t n_tok, int64_t n) {
    for (int64_t s = 0; s < n_tok; ++s) {
        if (tokens[s] < 0 || tokens[s] >= T) return -1;
        int32_t a = adapter_id[tokens[s]];
        if (a < 0 || a >= n) return -2;
    }
    return 0;
}

/* Compressed path: Delta_i = U_k (Sigma_i V_k^T), k = cluster_of[i]
 * (Sec. 3.1 objective and Sec. 3.2 clustered objective). */
int cts_oracle_apply(int64_t T, int64_t d_in, int64_t d_out, int64_t r,
                     int64_t n, int64_t K,
                     const double* x, const int32_t* adapter_id,
                     const int32_t* cluster_of, const double* W,
                     const double* U, const double* Vt, const double* Sigma,
                     const int64_t* tokens, int64_t n_tok, double* y) {
    if (T < 0 || d_in < 1 || d_out < 1 || r < 1 || n < 1 || K < 1 || n_tok < 0) return -1;
    int rc = check_tokens(adapter_id, T, tokens, n_tok, n);
    if (rc) return rc;
    for (int64_t i = 0; i < n; ++i)
        if (cluster_of[i] < 0 || cluster_of[i] >= K) return -2;
    if (n_tok == 0) return 0;

    double* M = (double*)malloc(sizeof(double) * (size_t)(r * d_in));
    double* D = (double*)malloc(sizeof(double) * (size_t)(d_out * d_in));
    int64_t* order = visit_order(adapter_id, tokens, n_tok, n);
    if (!M || !D || !order) { free(M); free(D); free(order); return -1; }

    int64_t cur = -1;
    for (int64_t v = 0; v < n_tok; ++v) {
        const int64_t s = order[v];
        const int64_t t = tokens[s];
        const int64_t a = adapter_id[t];
        if (a != cur) {
            const int64_t k = cluster_of[a];
            /* M = Sigma_a V_k^T  (r x d_in) */
            matmul(Sigma + a * r * r, Vt + k * r * d_in, M, r, r, d_in);
            /* D = U_k M  (d_out x d_in) */
            matmul(U + k * d_out * r, M, D, d_out, r, d_in);
            cur = a;
        }
        apply_rows(W, D, x + t * d_in, y + s * d_out, d_out, d_in);
    }
    free(M); free(D); free(order);
    return 0;
}

/* Diagonal variant (Sec. 3.1, eq. JD-Diag): Delta_i = U_k diag(sigma_i) V_k^T,
 * with diag(sigma_i) V_k^T formed as V_k^T with row q scaled by sigma_i[q]. */
int cts_oracle_apply_diag(int64_t T, int64_t d_in, int64_t d_out, int64_t r,
                          int64_t n, int64_t K,
                          const double* x, const int32_t* adapter_id,
                          const int32_t* cluster_of, const double* W,
                          const double* U, const double* Vt, const double* sigma,
                          const int64_t* tokens, int64_t n_tok, double* y) {
    if (T < 0 || d_in < 1 || d_out < 1 || r < 1 || n < 1 || K < 1 || n_tok < 0) return -1;
    int rc = check_tokens(adapter_id, T, tokens, n_tok, n);
    if (rc) return rc;
    for (int64_t i = 0; i < n; ++i)
        if (cluster_of[i] < 0 || cluster_of[i] >= K) return -2;
    if (n_tok == 0) return 0;

    double* M = (double*)malloc(sizeof(double) * (size_t)(r * d_in));
    double* D = (double*)malloc(sizeof(double) * (size_t)(d_out * d_in));
    int64_t* order = visit_order(adapter_id, tokens, n_tok, n);
    if (!M || !D || !order) { free(M); free(D); free(order); return -1; }

    int64_t cur = -1;
    for (int64_t v = 0; v < n_tok; ++v) {
        const int64_t s = order[v];
        const int64_t t = tokens[s];
        const int64_t a = adapter_id[t];
        if (a != cur) {
            const int64_t k = cluster_of[a];
            /* M = diag(sigma_a) V_k^T  (r x d_in) */
            for (int64_t q = 0; q < r; ++q)
                for (int64_t c = 0; c < d_in; ++c)
                    M[q * d_in + c] = sigma[a * r + q] * Vt[k * r * d_in + q * d_in + c];
            /* D = U_k M  (d_out x d_in) */
            matmul(U + k * d_out * r, M, D, d_out, r, d_in);
            cur = a;
        }
        apply_rows(W, D, x + t * d_in, y + s * d_out, d_out, d_in);
    }
    free(M); free(D); free(order);
    return 0;
}

/* Mixed ranks, compressed path: Delta_i = U_k[:, :r_k] Sigma_i[:r_k, :r_k]
 * V_k^T[:r_k, :] with r_k = rank_of_cluster[k] (0 <= r_k <= r). */
int cts_oracle_apply_ranked(int64_t T, int64_t d_in, int64_t d_out, int64_t r,
                            int64_t n, int64_t K,
                            const double* x, const int32_t* adapter_id,
                            const int32_t* cluster_of, const double* W,
                            const double* U, const double* Vt, const double* Sigma,
                            const int32_t* rank_of_cluster,
                            const int64_t* tokens, int64_t n_tok, double* y) {
    if (T < 0 || d_in < 1 || d_out < 1 || r < 1 || n < 1 || K < 1 || n_tok < 0) return -1;
    int rc = check_tokens(adapter_id, T, tokens, n_tok, n);
    if (rc) return rc;
    for (int64_t i = 0; i < n; ++i)
        if (cluster_of[i] < 0 || cluster_of[i] >= K) return -2;
    for (int64_t k = 0; k < K; ++k)
        if (rank_of_cluster[k] < 0 || rank_of_cluster[k] > r) return -3;
    if (n_tok == 0) return 0;

    double* M = (double*)malloc(sizeof(double) * (size_t)(r * d_in));
    double* D = (double*)malloc(sizeof(double) * (size_t)(d_out * d_in));
    int64_t* order = visit_order(adapter_id, tokens, n_tok, n);
    if (!M || !D || !order) { free(M); free(D); free(order); return -1; }

    int64_t cur = -1;
    for (int64_t v = 0; v < n_tok; ++v) {
        const int64_t s = order[v];
        const int64_t t = tokens[s];
        const int64_t a = adapter_id[t];
        if (a != cur) {
            const int64_t k = cluster_of[a];
            const int64_t rk = rank_of_cluster[k];
            const double* Sa = Sigma + a * r * r;
            const double* Vk = Vt + k * r * d_in;
            const double* Uk = U + k * d_out * r;
            /* M = Sigma_a[:rk, :rk] V_k^T[:rk, :]  (rk x d_in) */
            #pragma omp parallel for schedule(static)
            for (int64_t q = 0; q < rk; ++q)
                for (int64_t c = 0; c < d_in; ++c) {
                    double acc = 0.0;
                    for (int64_t p = 0; p < rk; ++p) acc += Sa[q * r + p] * Vk[p * d_in + c];
                    M[q * d_in + c] = acc;
                }
            /* D = U_k[:, :rk] M  (d_out x d_in) */
            #pragma omp parallel for schedule(static)
            for (int64_t o = 0; o < d_out; ++o)
                for (int64_t c = 0; c < d_in; ++c) {
                    double acc = 0.0;
                    for (int64_t q = 0; q < rk; ++q) acc += Uk[o * r + q] * M[q * d_in + c];
                    D[o * d_in + c] = acc;
                }
            cur = a;
        }
        apply_rows(W, D, x + t * d_in, y + s * d_out, d_out, d_in);
    }
    free(M); free(D); free(order);
    return 0;
}

/* Mixed ranks, uncompressed path: Delta_i = B_i[:, :r_i] A_i[:r_i, :] with
 * r_i = rank_of_adapter[i] (0 <= r_i <= r_l). */
int cts_oracle_apply_uncompressed_ranked(int64_t T, int64_t d_in, int64_t d_out, int64_t r_l,
                                         int64_t n, const double* x, const int32_t* adapter_id,
                                         const double* W, const double* A, const double* B,
                                         const int32_t* rank_of_adapter,
                                         const int64_t* tokens, int64_t n_tok, double* y) {
    if (T < 0 || d_in < 1 || d_out < 1 || r_l < 1 || n < 1 || n_tok < 0) return -1;
    int rc = check_tokens(adapter_id, T, tokens, n_tok, n);
    if (rc) return rc;
    for (int64_t i = 0; i < n; ++i)
        if (rank_of_adapter[i] < 0 || rank_of_adapter[i] > r_l) return -3;
    if (n_tok == 0) return 0;

    double* D = (double*)malloc(sizeof(double) * (size_t)(d_out * d_in));
    int64_t* order = visit_order(adapter_id, tokens, n_tok, n);
    if (!D || !order) { free(D); free(order); return -1; }

    int64_t cur = -1;
    for (int64_t v = 0; v < n_tok; ++v) {
        const int64_t s = order[v];
        const int64_t t = tokens[s];
        const int64_t a = adapter_id[t];
        if (a != cur) {
            const int64_t ra = rank_of_adapter[a];
            const double* Ba = B + a * d_out * r_l;
            const double* Aa = A + a * r_l * d_in;
            #pragma omp parallel for schedule(static)
            for (int64_t o = 0; o < d_out; ++o)
                for (int64_t c = 0; c < d_in; ++c) {
                    double acc = 0.0;
                    for (int64_t q = 0; q < ra; ++q) acc += Ba[o * r_l + q] * Aa[q * d_in + c];
                    D[o * d_in + c] = acc;
                }
            cur = a;
        }
        apply_rows(W, D, x + t * d_in, y + s * d_out, d_out, d_in);
    }
    free(D); free(order);
    return 0;
}

/* Uncompressed comparison path: Delta_i = B_i A_i (Sec. 3, first paragraph). */
int cts_oracle_apply_uncompressed(int64_t T, int64_t d_in, int64_t d_out, int64_t r_l,
                                  int64_t n, const double* x, const int32_t* adapter_id,
                                  const double* W, const double* A, const double* B,
                                  const int64_t* tokens, int64_t n_tok, double* y) {
    if (T < 0 || d_in < 1 || d_out < 1 || r_l < 1 || n < 1 || n_tok < 0) return -1;
    int rc = check_tokens(adapter_id, T, tokens, n_tok, n);
    if (rc) return rc;
    if (n_tok == 0) return 0;

    double* D = (double*)malloc(sizeof(double) * (size_t)(d_out * d_in));
    int64_t* order = visit_order(adapter_id, tokens, n_tok, n);
    if (!D || !order) { free(D); free(order); return -1; }

    int64_t cur = -1;
    for (int64_t v = 0; v < n_tok; ++v) {
        const int64_t s = order[v];
        const int64_t t = tokens[s];
        const int64_t a = adapter_id[t];
        if (a != cur) {
            matmul(B + a * d_out * r_l, A + a * r_l * d_in, D, d_out, r_l, d_in);
            cur = a;
        }
        apply_rows(W, D, x + t * d_in, y + s * d_out, d_out, d_in);
    }
    free(D); free(order);
    return 0;
}
