"""Pins of the compression oracle (oracle/compress.py) against what the paper
and the mathematics fix: Prop. 1 (lossless iff r >= r~), Thm. 1 and its
Corollary, monotone decrease of the alternating solvers (App. A.1), the k = n
case (eq. svd, Eckart-Young), brute-force least squares for the closed-form
cores (eq. sigmastar and the JD-Diag diagonals) and the JD-Diag U solve,
stationarity of the eigenvalue iteration (App. A.2), and the clustering of
App. A.3 on separable collections.  Planted mistakes show that the pins
catch a wrong transpose or a dropped factor."""
import numpy as np
import pytest

from oracle import compress as C


def _shared_space_loras(rs, n, d_out, d_in, r_l, rt):
    """LoRAs whose A_i rows lie in one rt-dim row space and B_i columns in one
    rt-dim column space: r~ = rt exactly (Prop. 1)."""
    Ra = rs.standard_normal((rt, d_in))
    Lb = rs.standard_normal((d_out, rt))
    A = np.stack([rs.standard_normal((r_l, rt)) @ Ra for _ in range(n)])
    B = np.stack([Lb @ rs.standard_normal((rt, r_l)) for _ in range(n)])
    return A, B


def _random_loras(rs, n, d_out, d_in, r_l):
    return rs.standard_normal((n, r_l, d_in)), rs.standard_normal((n, d_out, r_l))


def _rtilde(A, B):
    return max(np.linalg.matrix_rank(np.concatenate(list(A), axis=0)),
               np.linalg.matrix_rank(np.concatenate([b.T for b in B], axis=0)))


# ------------------------------------------------------------- Prop. 1
@pytest.mark.parametrize("solver", ["alternating", "eig"])
def test_prop1_lossless_at_rtilde(solver):
    rs = np.random.default_rng(1)
    A, B = _shared_space_loras(rs, n=7, d_out=14, d_in=11, r_l=2, rt=4)
    assert _rtilde(A, B) == 4
    jd = C.jd_full_alternating if solver == "alternating" else C.jd_full_eig
    U0, V0 = C.random_orthonormal(rs, 14, 4), C.random_orthonormal(rs, 11, 4)
    U, V, S, _ = jd(A, B, 4, U0, V0, iters=5)
    assert C.recon_error(U, V, S, A, B) < 1e-24
    assert np.allclose(U.T @ U, np.eye(4), atol=1e-12) and np.allclose(V.T @ V, np.eye(4), atol=1e-12)


@pytest.mark.parametrize("solver", ["alternating", "eig"])
def test_prop1_lossy_below_rtilde(solver):
    rs = np.random.default_rng(2)
    A, B = _shared_space_loras(rs, n=7, d_out=14, d_in=11, r_l=2, rt=4)
    jd = C.jd_full_alternating if solver == "alternating" else C.jd_full_eig
    U0, V0 = C.random_orthonormal(rs, 14, 3), C.random_orthonormal(rs, 11, 3)
    U, V, S, _ = jd(A, B, 3, U0, V0, iters=60)
    assert C.recon_error(U, V, S, A, B) > 1e-4


# ------------------------------------------------------------- Thm. 1
def _thm1_quantities(A, B, r):
    Ps = C.products(A, B)
    L = np.stack([P.reshape(-1) for P in Ps], axis=1)          # columns vec(B_i A_i)
    sig = np.linalg.svd(L, compute_uv=False)
    sbar = np.linalg.svd(Ps.sum(axis=0), compute_uv=False)
    lower = (sbar[:r] ** 2).sum()
    upper = (sig[:min(r * r, len(Ps))] ** 2).sum()
    return lower, upper, (sig ** 2).sum()


@pytest.mark.parametrize("seed,n,r", [(3, 12, 2), (4, 20, 3), (5, 6, 4)])
def test_thm1_bounds(seed, n, r):
    rs = np.random.default_rng(seed)
    A, B = _random_loras(rs, n, 10, 9, 2)
    lower, upper, total = _thm1_quantities(A, B, r)
    U0, V0 = C.svd_of_sum_init(A, B, r)
    U, V, S, hist = C.jd_full_alternating(A, B, r, U0, V0, iters=15)
    kept = (S ** 2).sum()
    recon = sum(np.linalg.norm(U @ S[i] @ V.T) ** 2 for i in range(n))
    assert abs(kept - recon) <= 1e-10 * kept                    # ||Sigma_i|| = ||U Sigma_i V^T||
    assert lower / n <= kept * (1 + 1e-12)                       # Jensen: sum ||x_i||^2 >= ||sum x_i||^2 / n
    assert kept <= upper * (1 + 1e-12)
    err = C.recon_error(U, V, S, A, B)
    assert err >= 1 - upper / total - 1e-12                      # relative-error corollary
    assert kept / total <= upper / total + 1e-12 <= 1 + 1e-12
    # the upper bound holds for any orthonormal bases; the eigenvalue iteration too
    Ur, Vr = C.random_orthonormal(rs, 10, r), C.random_orthonormal(rs, 9, r)
    assert (C.sigma_star(Ur, Vr, A, B) ** 2).sum() <= upper * (1 + 1e-12)
    _, _, Se, _ = C.jd_full_eig(A, B, r, U0, V0, iters=15)
    assert (Se ** 2).sum() <= upper * (1 + 1e-12)


def test_thm1_lower_bound_needs_one_over_n():
    """The proof's Jensen step gives sum_i ||x_i||^2 >= ||sum_i x_i||^2 / n; the
    printed bound has no 1/n.  With n identical LoRAs the JD optimum keeps
    n * (top-r energy of one LoRA), while the top-r energy of their sum is n^2
    times that: the corrected bound is met with equality, the printed one fails."""
    rs = np.random.default_rng(31)
    n, r = 5, 2
    A1, B1 = _random_loras(rs, 1, 8, 7, 3)
    A, B = np.repeat(A1, n, axis=0), np.repeat(B1, n, axis=0)
    lower, _, _ = _thm1_quantities(A, B, r)
    U0, V0 = C.svd_of_sum_init(A, B, r)
    _, _, S, _ = C.jd_full_alternating(A, B, r, U0, V0, iters=3)
    kept = (S ** 2).sum()
    assert abs(kept - lower / n) <= 1e-10 * kept
    assert kept < lower


def test_corollary_orthogonal_unit_loras():
    # rank-one unit-norm LoRAs e_a e_b^T at distinct rows and columns are
    # orthogonal in the trace inner product; the reading of the garbled
    # display is 1 - 1/n >= err >= 1 - min(r^2/n, 1)
    d, n = 9, 7
    rs = np.random.default_rng(6)
    rows, cols = rs.permutation(d)[:n], rs.permutation(d)[:n]
    A = np.zeros((n, 1, d))
    B = np.zeros((n, d, 1))
    for i in range(n):
        A[i, 0, cols[i]] = 1.0
        B[i, rows[i], 0] = 1.0
    Ps = C.products(A, B)
    gram = np.array([[np.trace(P @ Q.T) for Q in Ps] for P in Ps])
    assert np.allclose(gram, np.eye(n))
    for r in (1, 2, 3):
        U0, V0 = C.svd_of_sum_init(A, B, r)
        U, V, S, _ = C.jd_full_alternating(A, B, r, U0, V0, iters=10)
        kept = (S ** 2).sum()
        assert 1 - 1e-12 <= kept <= min(r * r, n) + 1e-12
        err = C.recon_error(U, V, S, A, B)
        assert 1 - 1 / n + 1e-12 >= err >= 1 - min(r * r / n, 1) - 1e-12


# ------------------------------------------------------------- monotone decrease
def test_alternating_objective_decreases():
    rs = np.random.default_rng(7)
    A, B = _random_loras(rs, 9, 12, 10, 3)
    U0, V0 = C.random_orthonormal(rs, 12, 4), C.random_orthonormal(rs, 10, 4)
    f0 = C.objective(U0, V0, C.sigma_star(U0, V0, A, B), A, B)
    _, _, _, hist = C.jd_full_alternating(A, B, 4, U0, V0, iters=12)
    seq = [f0] + [f for h in hist for f in h[:2]]
    assert all(b <= a * (1 + 1e-12) for a, b in zip(seq, seq[1:]))
    assert seq[-1] < seq[0]


@pytest.mark.parametrize("normalize", [False, True])
def test_als_objective_decreases(normalize):
    rs = np.random.default_rng(8)
    A, B = _random_loras(rs, 8, 10, 9, 2)
    U0, V0 = rs.standard_normal((10, 3)), rs.standard_normal((9, 3))
    f0 = C.objective(U0, V0, C.diag_sigma(U0, V0, A, B), A, B)
    U, V, s, hist = C.jd_diag_als(A, B, 3, U0, V0, sweeps=12, normalize=normalize)
    seq = [f0] + [f for h in hist for f in h]
    assert all(b <= a * (1 + 1e-10) for a, b in zip(seq, seq[1:]))
    assert seq[-1] < seq[0]
    assert abs(C.objective(U, V, s, A, B) - seq[-1]) <= 1e-10 * seq[-1]
    if normalize:
        assert abs((s ** 2).sum() - 1.0) < 1e-12


# ------------------------------------------------------------- k = n: SVD
def test_single_lora_is_truncated_svd():
    rs = np.random.default_rng(9)
    # a 10x8 update of rank 5 with a clear gap after 3 singular values
    Uq = np.linalg.qr(rs.standard_normal((10, 5)))[0]
    Vq = np.linalg.qr(rs.standard_normal((8, 5)))[0]
    sv = np.array([9.0, 6.0, 4.0, 1.0, 0.5])
    P = Uq @ np.diag(sv) @ Vq.T
    A = (np.diag(sv) @ Vq.T)[None]                            # B A = P with r_l = 5
    B = Uq[None]
    U0, V0 = C.random_orthonormal(rs, 10, 3), C.random_orthonormal(rs, 8, 3)
    for jd in (C.jd_full_alternating, C.jd_full_eig):
        U, V, S, _ = jd(A, B, 3, U0, V0, iters=40)
        assert abs(C.objective(U, V, S, A, B) - (1.0 ** 2 + 0.5 ** 2)) < 1e-10
        assert np.allclose(U @ S[0] @ V.T, Uq[:, :3] @ np.diag(sv[:3]) @ Vq[:, :3].T, atol=1e-8)
    assert np.allclose(P, B[0] @ A[0])


def test_cluster_k_equals_n_is_per_lora_svd():
    rs = np.random.default_rng(10)
    n, r = 4, 2
    A, B = _random_loras(rs, n, 9, 8, 3)
    U0, V0 = C.random_orthonormal(rs, 9, r), C.random_orthonormal(rs, 8, r)
    Uc = [C.random_orthonormal(rs, 9, r) for _ in range(n)]
    Vc = [C.random_orthonormal(rs, 8, r) for _ in range(n)]
    labels, Us, Vs, S, _ = C.jd_cluster(A, B, n, r, U0, V0, Uc, Vc, list(range(n)), jd_iters=200)
    assert sorted(labels.tolist()) == list(range(n))
    want = sum((np.linalg.svd(P, compute_uv=False)[r:] ** 2).sum() for P in C.products(A, B))
    got = sum(np.linalg.norm(C.products(A, B)[i] - Us[labels[i]] @ S[i] @ Vs[labels[i]].T) ** 2
              for i in range(n))
    assert abs(got - want) <= 1e-8 * want


# ------------------------------------------------------------- closed forms
def test_sigma_star_is_least_squares():
    rs = np.random.default_rng(11)
    A, B = _random_loras(rs, 3, 7, 6, 2)
    U, V = C.random_orthonormal(rs, 7, 3), C.random_orthonormal(rs, 6, 3)
    S = C.sigma_star(U, V, A, B)
    design = np.kron(V, U)                                      # vec(U S V^T) = (V (x) U) vec(S)
    for i, P in enumerate(C.products(A, B)):
        sol = np.linalg.lstsq(design, P.reshape(-1, order="F"), rcond=None)[0]
        assert np.allclose(sol.reshape(3, 3, order="F"), S[i], atol=1e-12)


def test_diag_sigma_is_least_squares():
    rs = np.random.default_rng(12)
    A, B = _random_loras(rs, 4, 7, 6, 2)
    U, V = rs.standard_normal((7, 3)), rs.standard_normal((6, 3))   # not orthonormal
    s = C.diag_sigma(U, V, A, B)
    design = np.stack([np.outer(U[:, j], V[:, j]).reshape(-1) for j in range(3)], axis=1)
    for i, P in enumerate(C.products(A, B)):
        sol = np.linalg.lstsq(design, P.reshape(-1), rcond=None)[0]
        assert np.allclose(sol, s[i], atol=1e-10)


def test_als_u_step_is_least_squares():
    # one sweep from (U0, V0): the U it takes minimizes sum_i ||P_i - U S_i V0^T||
    # for the diagonals s0 of (U0, V0)
    rs = np.random.default_rng(13)
    A, B = _random_loras(rs, 5, 5, 4, 2)
    U0, V0 = rs.standard_normal((5, 2)), rs.standard_normal((4, 2))
    s0 = C.diag_sigma(U0, V0, A, B)
    rows, rhs = [], []
    for i, P in enumerate(C.products(A, B)):
        M = V0 @ np.diag(s0[i])                                 # P_i ~ U M^T, vec row-major
        rows.append(np.kron(np.eye(5), M))
        rhs.append(P.reshape(-1))
    u = np.linalg.lstsq(np.concatenate(rows), np.concatenate(rhs), rcond=None)[0].reshape(5, 2)
    num = sum(P @ V0 @ np.diag(s0[i]) for i, P in enumerate(C.products(A, B)))
    den = sum(np.diag(s0[i]) @ V0.T @ V0 @ np.diag(s0[i]) for i in range(5))
    assert np.allclose(num @ np.linalg.inv(den), u, atol=1e-10)
    _, _, _, hist = C.jd_diag_als(A, B, 2, U0, V0, sweeps=1)
    assert abs(hist[0][0] - C.objective(u, V0, s0, A, B)) < 1e-9


def _eig_stationarity(jd):
    """Residuals of the stationarity conditions M U = U X, N V = V Y (App. A.2)
    after running `jd` to convergence from the merged initialization."""
    rs = np.random.default_rng(14)
    A, B = _random_loras(rs, 6, 10, 9, 2)
    U0, V0 = C.svd_of_sum_init(A, B, 3)
    U, V, S, crits = jd(A, B, 3, U0, V0, iters=400, tau=1e-13)
    Ps = C.products(A, B)
    M = sum(P @ V @ V.T @ P.T for P in Ps)
    N = sum(P.T @ U @ U.T @ P for P in Ps)
    ru = np.linalg.norm(M @ U - U @ (U.T @ M @ U)) / np.linalg.norm(M)
    rv = np.linalg.norm(N @ V - V @ (V.T @ N @ V)) / np.linalg.norm(N)
    return ru, rv, (A, B, U0, V0, U, V, S, crits)


def test_eig_iteration_stationary_point():
    ru, rv, (A, B, U0, V0, U, V, S, crits) = _eig_stationarity(C.jd_full_eig)
    assert crits[-1] < 1e-12
    assert ru < 1e-9 and rv < 1e-9
    Ua, Va, Sa, _ = C.jd_full_alternating(A, B, 3, U0, V0, iters=400, tau=1e-13)
    fa, fe = C.objective(Ua, Va, Sa, A, B), C.objective(U, V, S, A, B)
    assert abs(fa - fe) <= 1e-9 * fa


def test_criterion_closed_forms():
    rs = np.random.default_rng(15)
    U = C.random_orthonormal(rs, 8, 3)
    R = np.linalg.qr(rs.standard_normal((3, 3)))[0]
    assert C.criterion(U, U @ R, U, U) < 1e-14                  # same subspaces
    E = np.eye(8)
    assert abs(C.criterion(E[:, :3], E[:, 3:6], E[:, :3], E[:, :3]) - 1.0) < 1e-14


def test_orthogonalize_is_positive_qr():
    rs = np.random.default_rng(16)
    X = rs.standard_normal((9, 4))
    Q = C.orthogonalize(X)
    R = Q.T @ X
    assert np.allclose(Q.T @ Q, np.eye(4), atol=1e-13)
    assert np.allclose(np.tril(R, -1), 0, atol=1e-12) and np.all(np.diag(R) > 0)
    assert np.allclose(Q @ R, X, atol=1e-12)


def test_frob_normalize_and_restore():
    rs = np.random.default_rng(17)
    A, B = _shared_space_loras(rs, n=5, d_out=9, d_in=8, r_l=2, rt=3)
    An, Bn, norms = C.frob_normalize(A, B)
    assert np.allclose([np.linalg.norm(P) for P in C.products(An, Bn)], 1.0)
    U, V, S, _ = C.jd_full_alternating(An, Bn, 3, C.random_orthonormal(rs, 9, 3),
                                       C.random_orthonormal(rs, 8, 3), iters=4)
    S_restored = S * norms[:, None, None]
    assert C.recon_error(U, V, S_restored, A, B) < 1e-24


# ------------------------------------------------------------- clustering
def _two_groups(rs):
    A1, B1 = _shared_space_loras(rs, n=5, d_out=12, d_in=10, r_l=2, rt=2)
    A2, B2 = _shared_space_loras(rs, n=5, d_out=12, d_in=10, r_l=2, rt=2)
    order = rs.permutation(10)
    A = np.concatenate([A1, A2])[order]
    B = np.concatenate([B1, B2])[order]
    truth = (order >= 5).astype(int)
    return A, B, truth


def test_cluster_recovers_groups():
    rs = np.random.default_rng(18)
    A, B, truth = _two_groups(rs)
    U0, V0 = C.random_orthonormal(rs, 12, 2), C.random_orthonormal(rs, 10, 2)
    Uc = [C.random_orthonormal(rs, 12, 2) for _ in range(2)]
    Vc = [C.random_orthonormal(rs, 10, 2) for _ in range(2)]
    init = [int(np.where(truth == 0)[0][0]), int(np.where(truth == 1)[0][0])]
    labels, Us, Vs, S, rounds = C.jd_cluster(A, B, 2, 2, U0, V0, Uc, Vc, init, jd_iters=10)
    same = np.array_equal(labels, truth) or np.array_equal(labels, 1 - truth)
    assert same and rounds >= 1
    err = sum(np.linalg.norm(C.products(A, B)[i] - Us[labels[i]] @ S[i] @ Vs[labels[i]].T) ** 2
              for i in range(10))
    assert err < 1e-20 * sum(np.linalg.norm(P) ** 2 for P in C.products(A, B))


def test_assign_scores_pick_least_squares_cluster():
    rs = np.random.default_rng(19)
    A, B = _random_loras(rs, 6, 7, 6, 2)
    Us = [C.random_orthonormal(rs, 7, 2) for _ in range(3)]
    Vs = [C.random_orthonormal(rs, 6, 2) for _ in range(3)]
    sc = C.assign_scores(Us, Vs, A, B)
    for i, P in enumerate(C.products(A, B)):
        errs = []
        for j in range(3):
            design = np.kron(Vs[j], Us[j])
            sol = np.linalg.lstsq(design, P.reshape(-1, order="F"), rcond=None)[0]
            errs.append(np.linalg.norm(design @ sol - P.reshape(-1, order="F")) ** 2)
        assert np.argmin(errs) == np.argmax(sc[i])
        assert np.allclose(np.linalg.norm(P) ** 2 - sc[i], errs, atol=1e-10)


def test_kmeans_fixed_point_and_blobs():
    rs = np.random.default_rng(20)
    centers = np.array([[0.0, 0.0], [10.0, 0.0], [0.0, 10.0]])
    X = np.concatenate([c + rs.standard_normal((15, 2)) for c in centers])
    labels = C.kmeans(X, [0, 15, 30])
    assert np.array_equal(labels, np.repeat([0, 1, 2], 15))
    cent = np.stack([X[labels == j].mean(axis=0) for j in range(3)])
    d = ((X[:, None] - cent[None]) ** 2).sum(axis=2)
    assert np.array_equal(np.argmin(d, axis=1), labels)


# ------------------------------------------------------------- planted mistakes
def test_planted_mistakes_fail_the_pins():
    rs = np.random.default_rng(21)
    A, B = _shared_space_loras(rs, n=6, d_out=10, d_in=10, r_l=2, rt=3)
    U0, V0 = C.random_orthonormal(rs, 10, 3), C.random_orthonormal(rs, 10, 3)
    U, V, S, _ = C.jd_full_eig(A, B, 3, U0, V0, iters=5)
    assert C.recon_error(U, V, S, A, B) < 1e-24
    # transposed core: Sigma_i = V^T (B_i A_i) U breaks Prop. 1
    bad = np.stack([V.T @ P @ U for P in C.products(A, B)])
    assert C.recon_error(U, V, bad, A, B) > 1e-3
    # the eigenvalue iteration with a wrong index (the next LoRA's B in the
    # last factor of U's update): the stationarity pin fails
    def bad_eig(A, B, r, U0, V0, iters=10, tau=None):
        U, V = U0, V0
        n = A.shape[0]
        for _ in range(iters):
            Un0 = sum(B[i] @ (A[i] @ V) @ (V.T @ A[i].T) @ (B[(i + 1) % n].T @ U) for i in range(n))
            Vn0 = sum(A[i].T @ (B[i].T @ U) @ (U.T @ B[i]) @ (A[i] @ V) for i in range(n))
            U, V = C.orthogonalize(Un0), C.orthogonalize(Vn0)
        return U, V, C.sigma_star(U, V, A, B), [1.0]
    ru, rv, _ = _eig_stationarity(bad_eig)
    assert max(ru, rv) > 1e-4


# ----------------------------------- App. A.3 Step 1 for a cluster below rank
def test_span_bases_reconstruct_small_cluster_exactly():
    """A cluster whose m members supply fewer than r directions (m r_l < r):
    span_bases returns orthonormal bases containing every member's B_i
    columns and A_i^T columns, so the members' optimal cores (eq. sigmastar)
    reconstruct them with zero residual (Prop. 1) -- the minimum of the
    cluster's Step 1 objective.  The given bases alone (what the cluster had
    before Step 1) do not."""
    rs = np.random.default_rng(70)
    d_out, d_in, r_l, r = 30, 26, 3, 16
    for m in (1, 2, 5):
        A, B = _random_loras(rs, m, d_out, d_in, r_l)
        Uc, Vc = C.random_orthonormal(rs, d_out, r), C.random_orthonormal(rs, d_in, r)
        U, V = C.span_bases(A, B, r, Uc, Vc)
        assert U.shape == (d_out, r) and V.shape == (d_in, r)
        assert np.abs(U.T @ U - np.eye(r)).max() < 1e-12
        assert np.abs(V.T @ V - np.eye(r)).max() < 1e-12
        S = C.sigma_star(U, V, A, B)
        total = sum(np.linalg.norm(P) ** 2 for P in C.products(A, B))
        assert C.objective(U, V, S, A, B) < 1e-24 * total
        # the leading m r_l columns span the members' B_i columns (A_i^T rows)
        Bs = np.concatenate(list(B), axis=1)
        As = np.concatenate([a.T for a in A], axis=1)
        Ul, Vl = U[:, :m * r_l], V[:, :m * r_l]
        assert np.abs(Bs - Ul @ (Ul.T @ Bs)).max() < 1e-10 * np.abs(Bs).max()
        assert np.abs(As - Vl @ (Vl.T @ As)).max() < 1e-10 * np.abs(As).max()
        # the rest of the rank comes from the given bases' leading columns
        q = r - m * r_l
        Xu = np.concatenate([Bs, Uc[:, :q]], axis=1)
        assert np.abs(Xu - U @ (U.T @ Xu)).max() < 1e-10 * np.abs(Xu).max()
        # planted mistake: keeping the given bases leaves a residual
        S0 = C.sigma_star(Uc, Vc, A, B)
        assert C.objective(Uc, Vc, S0, A, B) > 0.1 * total
    with pytest.raises(ValueError):
        C.span_bases(*_random_loras(rs, 6, d_out, d_in, r_l), r, Uc, Vc)   # 6 x 3 >= 16


def test_cluster_small_clusters_reconstruct_their_members():
    """Clustering with K = 3 on a collection where the k-means labels leave
    clusters below rank: after the rounds, every member of a cluster with
    members x r_l < r is reconstructed exactly by its cluster's bases, and
    every cluster with at least r directions by its JD bases to the JD's
    accuracy -- Step 1 minimized for every non-empty cluster."""
    rs = np.random.default_rng(71)
    d_out, d_in, r_l, r, K = 40, 36, 4, 16, 3
    # a large group of 10 LoRAs sharing 16-dim spaces and two LoRAs of their own
    A1, B1 = _shared_space_loras(rs, n=10, d_out=d_out, d_in=d_in, r_l=r_l, rt=16)
    A2, B2 = _random_loras(rs, 2, d_out, d_in, r_l)
    A, B = np.concatenate([A1, A2 * 8.0]), np.concatenate([B1, B2 * 8.0])
    U0, V0 = C.random_orthonormal(rs, d_out, r), C.random_orthonormal(rs, d_in, r)
    Uc = [C.random_orthonormal(rs, d_out, r) for _ in range(K)]
    Vc = [C.random_orthonormal(rs, d_in, r) for _ in range(K)]
    labels, Us, Vs, S, rounds = C.jd_cluster(A, B, K, r, U0, V0, Uc, Vc, [0, 10, 11], jd_iters=30)
    P = C.products(A, B)
    sizes = np.bincount(labels, minlength=K)
    small = [j for j in range(K) if 0 < sizes[j] * r_l < r]
    assert small, sizes                                  # the case under test occurs
    for i in range(len(A)):
        j = labels[i]
        err = np.linalg.norm(P[i] - Us[j] @ S[i] @ Vs[j].T) ** 2 / np.linalg.norm(P[i]) ** 2
        assert err < (1e-20 if j in small else 1e-6), (i, j, err)
