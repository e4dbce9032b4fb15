"""Offline compression oracle: joint diagonalization of a LoRA collection and
its clustering (Sec. 3.1, 3.2, 4 and App. A), in float64 numpy.

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the benchmark's CPU
baseline leg are the only callers.  Nothing here is imported by the GPU
library, and nothing here imports it.

Every function follows the paper's definitions in its own order and notation,
with explicit products B_i A_i where the definition has them; only numpy's
matrix product, eigh, QR, solve and SVD are used as steps.

Conventions: A[n][r_l][d_in] and B[n][d_out][r_l] hold the LoRAs (the
layer's layout), so the i-th update is B_i A_i (d_out x d_in).  Bases are
U (d_out x r) and V (d_in x r); the layer takes U as is and V transposed.
Sigma[n][r][r] (JD-Full) or sigma[n][r] (JD-Diag diagonals).

Readings (where the paper leaves a choice open):
* Initial bases are inputs (the paper does not fix them); ``svd_of_sum_init``
  gives the top-r singular vectors of sum_i B_i A_i, the merged model of the
  lower bound of Thm. 1, from which the alternating solver never goes below
  that bound.
* The alternating solver updates U from the current V, then V from the new U
  (App. A.1 case 1).  The eigenvalue iteration updates both from the previous
  pair (App. A.2) and orthogonalizes with the Q of a QR factorization whose R
  has a positive diagonal (the unique one for full column rank).
* The convergence measure is the paper's criterion (App. H, convergence; tau = 1e-3):
  max over U, V of ||X_{t+1} - X_t X_t^T X_{t+1}||_F / ||X_{t+1}||_F.
* JD-Diag's optional normalization (App. A.1 case 2, step 4) rescales the
  diagonals to sum_i ||sigma_i||^2 = 1 and multiplies U and V by the square
  root of the removed factor, so that every U diag(sigma_i) V^T is unchanged.
* Frobenius normalization (Sec. 6.1) divides B_i by ||B_i A_i||_F; restoring
  the norms multiplies Sigma_i (sigma_i) by them.
* Clustering (App. A.3): k-means over vec(Sigma_i) of a single-basis JD-Full
  starts from the centroids Sigma_{i} of the given LoRA indices (ties and
  empty clusters: lowest index wins; an empty cluster keeps its centroid /
  bases); per-cluster JD-Full starts from the given per-cluster bases each
  round when its members supply at least r directions (members x r_l >= r).
  A non-empty cluster with fewer (members x r_l < r) takes ``span_bases``: by
  Prop. 1 any U_j holding every member's B_i columns and V_j holding every
  A_i^T column reconstructs the members exactly, so such a pair minimizes the
  cluster's objective of App. A.3 Step 1 (at zero); of these minimizers the
  one taken completes the members' columns with the leading columns of the
  given bases, orthogonalized in that order.  A LoRA moves to the cluster
  maximizing ||U_j^T B_i A_i V_j||_F^2,
  which for orthonormal U_j, V_j is the cluster minimizing
  min_Sigma ||B_i A_i - U_j Sigma V_j^T||_F^2.
"""
from __future__ import annotations

import numpy as np


# ------------------------------------------------------------------ basics
def products(A, B):
    """The LoRA updates B_i A_i (Sec. 3), each d_out x d_in."""
    A = np.asarray(A, np.float64)
    B = np.asarray(B, np.float64)
    return np.stack([B[i] @ A[i] for i in range(A.shape[0])])


def frob_normalize(A, B):
    """Sec. 6.1: every B_i A_i scaled to unit Frobenius norm (B_i divided by
    ||B_i A_i||_F).  Returns (A, B scaled, norms)."""
    A = np.asarray(A, np.float64)
    B = np.asarray(B, np.float64)
    norms = np.array([np.linalg.norm(B[i] @ A[i]) for i in range(A.shape[0])])
    return A, B / norms[:, None, None], norms


def sigma_star(U, V, A, B):
    """eq. sigmastar (App. A.1 case 1): the optimal core for orthonormal U, V,
    Sigma_i = U^T B_i A_i V."""
    return np.stack([U.T @ P @ V for P in products(A, B)])


def diag_sigma(U, V, A, B):
    """App. A.1 case 2: the optimal diagonals for fixed U, V,
    diag(Sigma_i) = (U^T U o V^T V)^{-1} (U^T B_i o V^T A_i^T) 1."""
    A = np.asarray(A, np.float64)
    B = np.asarray(B, np.float64)
    G = (U.T @ U) * (V.T @ V)
    out = []
    for i in range(A.shape[0]):
        w = ((U.T @ B[i]) * (V.T @ A[i].T)).sum(axis=1)
        out.append(np.linalg.solve(G, w))
    return np.stack(out)


def objective(U, V, S, A, B):
    """eq. jointsvd: sum_i ||B_i A_i - U Sigma_i V^T||_F^2; S is [n][r][r] or,
    for diagonal cores, [n][r]."""
    S = np.asarray(S, np.float64)
    tot = 0.0
    for i, P in enumerate(products(A, B)):
        Si = np.diag(S[i]) if S.ndim == 2 else S[i]
        tot += np.linalg.norm(P - U @ Si @ V.T) ** 2
    return tot


def recon_error(U, V, S, A, B):
    """Relative reconstruction error of Thm. 1:
    sum_i ||U Sigma_i V^T - B_i A_i||_F^2 / sum_i ||B_i A_i||_F^2."""
    return objective(U, V, S, A, B) / sum(np.linalg.norm(P) ** 2 for P in products(A, B))


def criterion(U, Un, V, Vn):
    """Convergence measure (App. H, convergence)."""
    cu = np.linalg.norm(Un - U @ (U.T @ Un)) / np.linalg.norm(Un)
    cv = np.linalg.norm(Vn - V @ (V.T @ Vn)) / np.linalg.norm(Vn)
    return max(cu, cv)


def orthogonalize(X):
    """Q of the reduced QR factorization X = QR with diag(R) > 0."""
    Q, R = np.linalg.qr(X)
    s = np.sign(np.diag(R))
    s[s == 0] = 1.0
    return Q * s


def random_orthonormal(rng, d, r):
    return orthogonalize(rng.standard_normal((d, r)))


def svd_of_sum_init(A, B, r):
    """Top-r left and right singular vectors of sum_i B_i A_i."""
    u, _, vt = np.linalg.svd(products(A, B).sum(axis=0))
    return u[:, :r], vt[:r].T


def _top_eigvecs(M, r):
    w, Q = np.linalg.eigh(M)
    return Q[:, np.argsort(w)[::-1][:r]]


# ----------------------------------------------------------------- JD-Full
def jd_full_alternating(A, B, r, U0, V0, iters=10, tau=None):
    """App. A.1 case 1: U <- top-r eigenvectors of M = sum_i B_i A_i V V^T
    A_i^T B_i^T, then V <- top-r eigenvectors of N = sum_i A_i^T B_i^T U U^T
    B_i A_i; Sigma_i from eq. sigmastar.  Stops after `iters` rounds or when
    the criterion drops below tau.  Returns U, V, Sigma and the per-round
    history [(objective after the U step, objective after the V step, crit)]."""
    Ps = products(A, B)
    U = np.asarray(U0, np.float64)
    V = np.asarray(V0, np.float64)
    hist = []
    for _ in range(iters):
        M = sum(P @ V @ V.T @ P.T for P in Ps)
        Un = _top_eigvecs(M, r)
        f_u = objective(Un, V, sigma_star(Un, V, A, B), A, B)
        N = sum(P.T @ Un @ Un.T @ P for P in Ps)
        Vn = _top_eigvecs(N, r)
        f_v = objective(Un, Vn, sigma_star(Un, Vn, A, B), A, B)
        c = criterion(U, Un, V, Vn)
        U, V = Un, Vn
        hist.append((f_u, f_v, c))
        if tau is not None and c < tau:
            break
    return U, V, sigma_star(U, V, A, B), hist


def eig_step(A, B, U, V):
    """One step of the App. A.2 eigenvalue iteration from the pair (U, V):
    U0' = sum_i B_i (A_i V)(V^T A_i^T)(B_i^T U),
    V0' = sum_i A_i^T (B_i^T U)(U^T B_i)(A_i V),
    returns orthogonalize(U0'), orthogonalize(V0')."""
    A = np.asarray(A, np.float64)
    B = np.asarray(B, np.float64)
    Un0 = sum(B[i] @ (A[i] @ V) @ (V.T @ A[i].T) @ (B[i].T @ U) for i in range(A.shape[0]))
    Vn0 = sum(A[i].T @ (B[i].T @ U) @ (U.T @ B[i]) @ (A[i] @ V) for i in range(A.shape[0]))
    return orthogonalize(Un0), orthogonalize(Vn0)


def jd_full_eig(A, B, r, U0, V0, iters=10, tau=None):
    """App. A.2 eigenvalue iteration: `iters` steps of eig_step (or until the
    criterion drops below tau).  Returns U, V, Sigma (eq. sigmastar) and the
    per-round criteria."""
    A = np.asarray(A, np.float64)
    B = np.asarray(B, np.float64)
    U = np.asarray(U0, np.float64)
    V = np.asarray(V0, np.float64)
    crits = []
    for _ in range(iters):
        Un, Vn = eig_step(A, B, U, V)
        c = criterion(U, Un, V, Vn)
        U, V = Un, Vn
        crits.append(c)
        if tau is not None and c < tau:
            break
    return U, V, sigma_star(U, V, A, B), crits


# ----------------------------------------------------------------- JD-Diag
def jd_diag_als(A, B, r, U0, V0, sweeps=10, normalize=False):
    """App. A.1 case 2, coordinate descent: the diagonals from (U0, V0), then
    per sweep U = (sum_i B_i A_i V S_i)(sum_i S_i V^T V S_i)^{-1},
    V = (sum_i A_i^T B_i^T U S_i)(sum_i S_i U^T U S_i)^{-1} (with the new U),
    the diagonals from the new pair, and optionally the normalization.
    Returns U, V, sigma[n][r] and the objective after each step
    [(after U, after V, after Sigma)]."""
    A = np.asarray(A, np.float64)
    B = np.asarray(B, np.float64)
    Ps = products(A, B)
    U = np.asarray(U0, np.float64).copy()
    V = np.asarray(V0, np.float64).copy()
    s = diag_sigma(U, V, A, B)
    hist = []
    for _ in range(sweeps):
        num = sum(Ps[i] @ V @ np.diag(s[i]) for i in range(len(Ps)))
        den = sum(np.diag(s[i]) @ V.T @ V @ np.diag(s[i]) for i in range(len(Ps)))
        U = num @ np.linalg.inv(den)
        f_u = objective(U, V, s, A, B)
        num = sum(Ps[i].T @ U @ np.diag(s[i]) for i in range(len(Ps)))
        den = sum(np.diag(s[i]) @ U.T @ U @ np.diag(s[i]) for i in range(len(Ps)))
        V = num @ np.linalg.inv(den)
        f_v = objective(U, V, s, A, B)
        s = diag_sigma(U, V, A, B)
        if normalize:
            nu = np.sqrt((s ** 2).sum())
            s = s / nu
            U = U * np.sqrt(nu)
            V = V * np.sqrt(nu)
        f_s = objective(U, V, s, A, B)
        hist.append((f_u, f_v, f_s))
    return U, V, s, hist


# -------------------------------------------------------------- clustering
def assign_scores(Us, Vs, A, B):
    """score[i][j] = ||U_j^T B_i A_i V_j||_F^2 (App. A.3 step 2, via eq.
    sigmastar: the best Sigma for cluster j leaves ||B_i A_i||^2 - score)."""
    Ps = products(A, B)
    return np.array([[np.linalg.norm(Us[j].T @ P @ Vs[j]) ** 2 for j in range(len(Us))] for P in Ps])


def kmeans(X, init_idx, max_iter=100):
    """Lloyd's k-means from the centroids X[init_idx]; stops when no label
    changes.  Ties and empty clusters: see the module readings."""
    X = np.asarray(X, np.float64)
    C = X[np.asarray(init_idx)].copy()
    labels = None
    for _ in range(max_iter):
        d = ((X[:, None, :] - C[None, :, :]) ** 2).sum(axis=2)
        new = np.argmin(d, axis=1)
        if labels is not None and np.array_equal(new, labels):
            break
        labels = new
        for j in range(C.shape[0]):
            if np.any(labels == j):
                C[j] = X[labels == j].mean(axis=0)
    return labels


def span_bases(A, B, r, Uc, Vc):
    """App. A.3 Step 1 for a cluster whose m members supply fewer than r
    directions (m r_l < r).  Every pair U, V with U containing the columns of
    all members' B_i and V those of all A_i^T gives U U^T B_i A_i V V^T =
    B_i A_i (Prop. 1), i.e. zero objective, the minimum.  Returned: the
    positive-diagonal QR factors of [B_1 ... B_m | Uc[:, :r - m r_l]] and
    [A_1^T ... A_m^T | Vc[:, :r - m r_l]] (members in increasing index
    order, the given bases' leading columns completing the rank)."""
    A = np.asarray(A, np.float64)
    B = np.asarray(B, np.float64)
    m, r_l = A.shape[0], A.shape[1]
    q = r - m * r_l
    if q <= 0:
        raise ValueError("span_bases needs fewer than r member directions")
    XU = np.concatenate([B[i] for i in range(m)] + [np.asarray(Uc, np.float64)[:, :q]], axis=1)
    XV = np.concatenate([A[i].T for i in range(m)] + [np.asarray(Vc, np.float64)[:, :q]], axis=1)
    return orthogonalize(XU), orthogonalize(XV)


def jd_cluster(A, B, k, r, U0, V0, Uc0, Vc0, init_idx, jd_iters=10, max_rounds=20, solver="eig"):
    """App. A.3: a single-basis JD-Full from (U0, V0), k-means on vec(Sigma_i)
    from the centroids of LoRAs init_idx, then rounds of per-cluster JD-Full
    (from the bases Uc0[j], Vc0[j]) and reassignment until no LoRA moves.
    Returns labels[n], Us[k], Vs[k], Sigma[n] (each from its own cluster's
    bases) and the number of rounds."""
    A = np.asarray(A, np.float64)
    B = np.asarray(B, np.float64)
    jd = jd_full_eig if solver == "eig" else jd_full_alternating
    _, _, S, _ = jd(A, B, r, U0, V0, jd_iters)
    labels = kmeans(S.reshape(A.shape[0], -1), init_idx)
    Us = [np.asarray(u, np.float64) for u in Uc0]
    Vs = [np.asarray(v, np.float64) for v in Vc0]
    rounds = 0
    for rounds in range(1, max_rounds + 1):
        for j in range(k):
            m = labels == j
            cnt = np.count_nonzero(m)
            if cnt * A.shape[1] >= r:
                Us[j], Vs[j], _, _ = jd(A[m], B[m], r, Uc0[j], Vc0[j], jd_iters)
            elif cnt > 0:
                Us[j], Vs[j] = span_bases(A[m], B[m], r, Uc0[j], Vc0[j])
        new = np.argmax(assign_scores(Us, Vs, A, B), axis=1)
        if np.array_equal(new, labels):
            break
        labels = new
    S = np.stack([Us[labels[i]].T @ (B[i] @ A[i]) @ Vs[labels[i]] for i in range(A.shape[0])])
    return labels, Us, Vs, S, rounds
