"""Pins of the fp64 oracle against what the paper and the mathematics fix.

Each test compares the oracle with something other than itself: a value
worked by hand, a different route to the same number (the factored order of
App. D, the uncompressed product), an identity the paper states (Prop. 1,
eq. svd, the merging remark) or an invariance of the definition.  A final
group plants plausible mistakes in a copy of the oracle's inputs and checks
that the pins catch them.
"""
import json
import os

import numpy as np
import pytest

from paper_2407_00066_amd import workloads as wl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "hand_worked_example.json")


def _golden():
    with open(GOLDEN) as f:
        g = json.load(f)
    arr = lambda k, dt=np.float64: np.asarray(g[k], dtype=dt)
    return g, arr


def _rand_case(rs, T, d_in, d_out, r, n, K):
    x = rs.standard_normal((T, d_in))
    W = rs.standard_normal((d_out, d_in))
    U = rs.standard_normal((K, d_out, r))
    Vt = rs.standard_normal((K, r, d_in))
    S = rs.standard_normal((n, r, r))
    aid = rs.integers(0, n, T).astype(np.int32)
    cof = rs.integers(0, K, n).astype(np.int32)
    return x, aid, cof, W, U, Vt, S


def _rel(a, b):
    return np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300)


# --------------------------------------------------------------------------
# hand-worked example (Sec. 3, 3.1, 3.2 definitions)

def test_golden_compressed(oracle_mod):
    g, arr = _golden()
    y = oracle_mod.apply(arr("x"), g["adapter_id"], g["cluster_of"], arr("W"), arr("U"),
                         arr("Vt"), arr("Sigma"))
    np.testing.assert_array_equal(y, arr("y_compressed"))


def test_golden_uncompressed(oracle_mod):
    g, arr = _golden()
    y = oracle_mod.apply_uncompressed(arr("x"), g["adapter_id"], arr("W"), arr("A"), arr("B"))
    np.testing.assert_array_equal(y, arr("y_uncompressed"))


def test_golden_sort(oracle_mod):
    g, arr = _golden()
    perm, offs = oracle_mod.sort_by_cluster(g["adapter_id"], g["cluster_of"], g["n"], g["K"])
    assert perm.tolist() == g["perm"] and offs.tolist() == g["cluster_offsets"]


def test_golden_subset_and_order(oracle_mod):
    """Requested tokens come back in the requested order (rows follow `tokens`)."""
    g, arr = _golden()
    y = oracle_mod.apply(arr("x"), g["adapter_id"], g["cluster_of"], arr("W"), arr("U"),
                         arr("Vt"), arr("Sigma"), tokens=[3, 1])
    np.testing.assert_array_equal(y, arr("y_compressed")[[3, 1]])


# --------------------------------------------------------------------------
# brute force on tiny inputs, by two routes the oracle does not take

@pytest.mark.parametrize("seed", [0, 1, 2])
def test_bruteforce_dense_and_factored(oracle_mod, seed):
    rs = np.random.default_rng(seed)
    T, d_in, d_out, r, n, K = 8, 13, 11, 5, 4, 3
    x, aid, cof, W, U, Vt, S = _rand_case(rs, T, d_in, d_out, r, n, K)
    y = oracle_mod.apply(x, aid, cof, W, U, Vt, S)
    # (a) dense: y_t = (W + U_k S_i Vt_k) x_t via einsum over all index pairs
    dense = np.stack([np.einsum("op,pq,qc->oc", U[cof[a]], S[a], Vt[cof[a]]) for a in range(n)])
    y_dense = np.einsum("toc,tc->to", W[None] + dense[aid], x)
    # (b) factored order of App. D: V^T x, then Sigma, then U, plus W x
    y_fact = np.empty_like(y)
    for t in range(T):
        k = cof[aid[t]]
        y_fact[t] = W @ x[t] + U[k] @ (S[aid[t]] @ (Vt[k] @ x[t]))
    assert _rel(y, y_dense) < 1e-13
    assert _rel(y, y_fact) < 1e-13


def test_bruteforce_uncompressed(oracle_mod):
    rs = np.random.default_rng(7)
    T, d_in, d_out, r_l, n = 9, 10, 7, 3, 4
    x = rs.standard_normal((T, d_in))
    W = rs.standard_normal((d_out, d_in))
    A = rs.standard_normal((n, r_l, d_in))
    B = rs.standard_normal((n, d_out, r_l))
    aid = rs.integers(0, n, T).astype(np.int32)
    y = oracle_mod.apply_uncompressed(x, aid, W, A, B)
    ref = np.stack([W @ x[t] + B[aid[t]] @ (A[aid[t]] @ x[t]) for t in range(T)])
    assert _rel(y, ref) < 1e-13


# --------------------------------------------------------------------------
# Prop. 1: lossless at r = r~ (with Sigma_i = U^T B_i A_i V from App. A.1)

def _lora_collection(rs, n, r_l, d_in, d_out):
    A = rs.standard_normal((n, r_l, d_in)) / np.sqrt(d_in)
    B = rs.standard_normal((n, d_out, r_l))
    return A, B


def test_prop1_exact_reconstruction(oracle_mod):
    rs = np.random.default_rng(11)
    n, r_l, d_in, d_out, T = 3, 4, 24, 20, 10
    A, B = _lora_collection(rs, n, r_l, d_in, d_out)
    U, Vt, S = oracle_mod.exact_compress(A, B)
    assert U.shape == (d_out, n * r_l)            # r~ = sum r_i for generic LoRAs
    x = rs.standard_normal((T, d_in))
    W = rs.standard_normal((d_out, d_in))
    aid = rs.integers(0, n, T).astype(np.int32)
    y_c = oracle_mod.apply(x, aid, np.zeros(n, np.int32), W, U[None], Vt[None], S)
    y_u = oracle_mod.apply_uncompressed(x, aid, W, A, B)
    assert _rel(y_c, y_u) < 1e-12


def test_prop1_lossy_below_rtilde(oracle_mod):
    """Dropping one basis direction (r < r~) must change the output: guards
    the exactness pin against being vacuous."""
    rs = np.random.default_rng(12)
    n, r_l, d_in, d_out, T = 3, 4, 24, 20, 10
    A, B = _lora_collection(rs, n, r_l, d_in, d_out)
    U, Vt, S = oracle_mod.exact_compress(A, B)
    x = rs.standard_normal((T, d_in))
    W = np.zeros((d_out, d_in))
    aid = np.arange(T, dtype=np.int32) % n
    y_u = oracle_mod.apply_uncompressed(x, aid, W, A, B)
    y_c = oracle_mod.apply(x, aid, np.zeros(n, np.int32), W, U[None, :, :-1], Vt[None, :-1],
                           S[:, :-1, :-1])
    assert _rel(y_c, y_u) > 1e-3


def test_tiny_exact_variant_matches_uncompressed(oracle_mod):
    """The 'Tiny-exact' case used on the GPU: the tiny fp32 collection (8
    rank-4 LoRAs, d=256) compressed losslessly at r = 32."""
    w = wl.make("tiny_fp32")
    U, Vt, S = oracle_mod.exact_compress(w.A, w.B)
    assert U.shape[1] == 32
    y_c = oracle_mod.apply(w.x, w.adapter_id, np.zeros(w.n, np.int32), w.W, U[None], Vt[None], S)
    y_u = oracle_mod.apply_uncompressed(w.x, w.adapter_id, w.W, w.A, w.B)
    assert _rel(y_c, y_u) < 1e-12


# --------------------------------------------------------------------------
# eq. svd: one adapter per cluster (k = n) reduces to a per-LoRA SVD, and a
# single adapter is plain LoRA

def test_k_equals_n_svd_form(oracle_mod):
    rs = np.random.default_rng(13)
    n, r_l, d_in, d_out, T = 4, 3, 12, 9, 12
    A, B = _lora_collection(rs, n, r_l, d_in, d_out)
    U = np.empty((n, d_out, r_l)); Vt = np.empty((n, r_l, d_in)); S = np.zeros((n, r_l, r_l))
    for i in range(n):
        u, s, vt = np.linalg.svd(B[i] @ A[i])
        U[i], Vt[i] = u[:, :r_l], vt[:r_l]
        S[i] = np.diag(s[:r_l])
    x = rs.standard_normal((T, d_in))
    W = rs.standard_normal((d_out, d_in))
    aid = rs.integers(0, n, T).astype(np.int32)
    y_c = oracle_mod.apply(x, aid, np.arange(n, dtype=np.int32), W, U, Vt, S)
    y_u = oracle_mod.apply_uncompressed(x, aid, W, A, B)
    assert _rel(y_c, y_u) < 1e-12


def test_single_adapter_is_plain_lora(oracle_mod):
    rs = np.random.default_rng(14)
    d_in, d_out, r_l, T = 16, 12, 4, 6
    A, B = _lora_collection(rs, 1, r_l, d_in, d_out)
    U, Vt, S = oracle_mod.exact_compress(A, B)
    x = rs.standard_normal((T, d_in))
    W = rs.standard_normal((d_out, d_in))
    y = oracle_mod.apply(x, np.zeros(T, np.int32), np.zeros(1, np.int32), W, U[None], Vt[None], S)
    ref = x @ (W + B[0] @ A[0]).T
    assert _rel(y, ref) < 1e-12


# --------------------------------------------------------------------------
# special cases and invariances of the definition

def test_zero_sigma_is_base_layer(oracle_mod):
    rs = np.random.default_rng(15)
    x, aid, cof, W, U, Vt, S = _rand_case(rs, 7, 10, 9, 4, 3, 2)
    y = oracle_mod.apply(x, aid, cof, W, U, Vt, np.zeros_like(S))
    assert _rel(y, x @ W.T) < 1e-14


def test_identity_bases_and_sigma(oracle_mod):
    """r = d, U = V = I, Sigma_i = I  ->  y = (W + I) x."""
    rs = np.random.default_rng(16)
    d, T, n = 8, 5, 2
    x = rs.standard_normal((T, d)); W = rs.standard_normal((d, d))
    I = np.eye(d)
    y = oracle_mod.apply(x, np.array([0, 1, 0, 1, 1], np.int32), np.zeros(n, np.int32), W,
                         I[None], I[None], np.stack([I, I]))
    assert _rel(y, x @ W.T + x) < 1e-14


def test_equal_sigma_is_merged_model(oracle_mod):
    """Remark (lower bound and merging): equal Sigma_i inside a cluster give
    one merged update, so tokens of different adapters see the same layer."""
    rs = np.random.default_rng(17)
    x, aid, cof, W, U, Vt, S = _rand_case(rs, 12, 10, 9, 4, 4, 1)
    S[:] = S[0]
    y = oracle_mod.apply(x, aid, cof, W, U, Vt, S)
    merged = W + U[0] @ S[0] @ Vt[0]
    assert _rel(y, x @ merged.T) < 1e-13


def test_linearity_in_x(oracle_mod):
    rs = np.random.default_rng(18)
    x1, aid, cof, W, U, Vt, S = _rand_case(rs, 6, 10, 9, 4, 3, 2)
    x2 = rs.standard_normal(x1.shape)
    a, b = 0.75, -2.5
    f = lambda xx: oracle_mod.apply(xx, aid, cof, W, U, Vt, S)
    assert _rel(f(a * x1 + b * x2), a * f(x1) + b * f(x2)) < 1e-12


def test_token_permutation_equivariance(oracle_mod):
    rs = np.random.default_rng(19)
    x, aid, cof, W, U, Vt, S = _rand_case(rs, 10, 8, 7, 3, 4, 2)
    p = rs.permutation(10)
    y = oracle_mod.apply(x, aid, cof, W, U, Vt, S)
    yp = oracle_mod.apply(x[p], aid[p], cof, W, U, Vt, S)
    np.testing.assert_array_equal(yp, y[p])


def test_cluster_relabel_invariance(oracle_mod):
    rs = np.random.default_rng(20)
    x, aid, cof, W, U, Vt, S = _rand_case(rs, 10, 8, 7, 3, 5, 3)
    q = np.array([2, 0, 1])                      # new label of old cluster k is q[k]
    U2 = np.empty_like(U); V2 = np.empty_like(Vt)
    U2[q] = U; V2[q] = Vt
    y = oracle_mod.apply(x, aid, cof, W, U, Vt, S)
    y2 = oracle_mod.apply(x, aid, q[cof].astype(np.int32), W, U2, V2, S)
    np.testing.assert_array_equal(y2, y)


def test_bf16_inputs_widen_exactly(oracle_mod):
    """uint16 arrays are bf16 bit patterns: 0x3F80 = 1.0, 0xC000 = -2.0, 0x3E80 = 0.25."""
    np.testing.assert_array_equal(oracle_mod.to_f64(np.array([0x3F80, 0xC000, 0x3E80], np.uint16)),
                                  [1.0, -2.0, 0.25])
    g, arr = _golden()
    bits = lambda k: wl.f32_to_bf16_bits(arr(k).astype(np.float32))
    y = oracle_mod.apply(bits("x"), g["adapter_id"], g["cluster_of"], bits("W"), bits("U"),
                         bits("Vt"), bits("Sigma"))
    np.testing.assert_array_equal(y, arr("y_compressed"))


# --------------------------------------------------------------------------
# sort: brute force with Python's sorted() over key tuples, and invariants

def _sort_ref(aid, cof):
    keys = sorted((int(cof[a]) if cof is not None else int(a), int(a), t) for t, a in enumerate(aid))
    return [t for _, _, t in keys]


@pytest.mark.parametrize("T,n,K,kind", [
    (0, 5, 2, "uniform"), (1, 5, 2, "uniform"), (63, 8, 3, "uniform"), (64, 8, 3, "uniform"),
    (65, 100, 1, "uniform"), (4096, 1000, 25, "uniform"), (300, 1000, 1000, "uniform"),
    (200, 50, 10, "same"), (200, 50, 10, "sorted"), (200, 50, 10, "reverse"), (200, 40, 40, "empty"),
])
def test_sort_bruteforce(oracle_mod, T, n, K, kind):
    rs = np.random.default_rng(T * 7 + n)
    aid = rs.integers(0, n, T).astype(np.int32)
    if kind == "same":
        aid[:] = 3
    elif kind == "sorted":
        aid = np.sort(aid)
    elif kind == "reverse":
        aid = np.sort(aid)[::-1].copy()
    if K == n and kind != "empty":
        cof = None
    else:
        cof = rs.integers(0, K, n).astype(np.int32)
        if kind == "empty":
            cof = (np.arange(n) % 3 * 7).astype(np.int32)   # only clusters 0, 7, 14 used
    perm, offs = oracle_mod.sort_by_cluster(aid, cof, n, K)
    assert perm.tolist() == _sort_ref(aid, cof)
    clus = (cof[aid] if cof is not None else aid)
    assert sorted(perm.tolist()) == list(range(T))
    assert offs[0] == 0 and offs[-1] == T
    for k in range(K):
        assert offs[k + 1] - offs[k] == int(np.sum(clus == k))
        assert np.all(clus[perm[offs[k]:offs[k + 1]]] == k)


def test_sort_rejects_bad_ids(oracle_mod):
    with pytest.raises(ValueError):
        oracle_mod.sort_by_cluster([0, 5], [0, 0], 2, 1)
    with pytest.raises(ValueError):
        oracle_mod.sort_by_cluster([0, 1], [0, 3], 2, 2)


# --------------------------------------------------------------------------
# planted mistakes: each would slip into a plausible oracle; a pin must fail

def test_planted_transposed_sigma_is_caught(oracle_mod):
    g, arr = _golden()
    S = arr("Sigma").transpose(0, 2, 1).copy()
    y = oracle_mod.apply(arr("x"), g["adapter_id"], g["cluster_of"], arr("W"), arr("U"), arr("Vt"), S)
    assert not np.array_equal(y, arr("y_compressed"))


def test_planted_transposed_u_is_caught(oracle_mod):
    g, arr = _golden()
    U = arr("U").transpose(0, 2, 1).copy()
    y = oracle_mod.apply(arr("x"), g["adapter_id"], g["cluster_of"], arr("W"), U, arr("Vt"), arr("Sigma"))
    assert not np.array_equal(y, arr("y_compressed"))


def test_planted_wrong_cluster_is_caught(oracle_mod):
    g, arr = _golden()
    y = oracle_mod.apply(arr("x"), g["adapter_id"], [0, 0, 0], arr("W"), arr("U"), arr("Vt"), arr("Sigma"))
    assert not np.array_equal(y, arr("y_compressed"))


def test_planted_dropped_base_term_is_caught(oracle_mod):
    g, arr = _golden()
    y = oracle_mod.apply(arr("x"), g["adapter_id"], g["cluster_of"], np.zeros((2, 3)), arr("U"),
                         arr("Vt"), arr("Sigma"))
    assert not np.array_equal(y, arr("y_compressed"))


# --------------------------------------------------------------------------
# generator sanity (no method arithmetic: shapes, seeds, distributions)

def test_workload_recipe():
    w = wl.make("tiny_fp32")
    assert w.x.dtype == np.float32 and w.W.shape == (256, 256) and w.U.shape == (1, 256, 16)
    Q = w.U[0].astype(np.float64)
    assert np.abs(Q.T @ Q - np.eye(16)).max() < 1e-5
    w2 = wl.make("tiny_fp32")
    np.testing.assert_array_equal(w.x, w2.x)
    lens = wl.prefill_lengths(np.random.default_rng(0), 32, 4096, 32, 256)
    assert lens.sum() == 4096 and lens.min() >= 32 and lens.max() <= 256
    c = wl.balanced_clusters(np.random.default_rng(0), 1000, 25)
    assert np.all(np.bincount(c, minlength=25) == 40)
    b = wl.f32_to_bf16_bits(np.array([1.0, 1.00390625, 1.01171875, -3.0], np.float32))
    # 1+2^-8 and 1+3*2^-8 are ties: they round to the even neighbours 0x3F80 and 0x3F82
    assert b.tolist() == [0x3F80, 0x3F80, 0x3F82, 0xC040]


def test_apply_multi_stacking_against_bruteforce(oracle_mod):
    """Multi-module batching (modules of one layer on the same x, ids and
    cluster map, Sec. 3.1, 3.2 per projection): apply_multi with module m's
    V_k^T in rows m r .. m r + r - 1 of the stacked array equals, per module,
    the dense brute force (W_m + U_k^(m) S_i^(m) V_k^(m)T) x_t built from
    that module's own arrays.  Planted mistake: the same modules stacked
    interleaved (row q of module m at q M + m) must not match."""
    rs = np.random.default_rng(91)
    T, d_in, r, n, K, d_outs = 7, 12, 4, 5, 3, (9, 6, 6)
    x = rs.standard_normal((T, d_in))
    aid = rs.integers(0, n, T).astype(np.int32)
    cof = rs.integers(0, K, n).astype(np.int32)
    Ws = [rs.standard_normal((d, d_in)) for d in d_outs]
    Us = [rs.standard_normal((K, d, r)) for d in d_outs]
    Vts = [rs.standard_normal((K, r, d_in)) for _ in d_outs]
    Ss = [rs.standard_normal((n, r, r)) for _ in d_outs]
    M = len(d_outs)
    stacked = np.zeros((K, M * r, d_in))
    for m in range(M):
        for q in range(r):
            stacked[:, m * r + q, :] = Vts[m][:, q, :]
    ys = oracle_mod.apply_multi(x, aid, cof, Ws, Us, stacked, Ss)
    for m in range(M):
        dense = np.stack([Us[m][cof[a]] @ Ss[m][a] @ Vts[m][cof[a]] for a in range(n)])
        want = np.einsum("toc,tc->to", Ws[m][None] + dense[aid], x)
        assert _rel(ys[m], want) < 1e-13, m
    inter = np.zeros_like(stacked)
    for m in range(M):
        for q in range(r):
            inter[:, q * M + m, :] = Vts[m][:, q, :]
    bad = oracle_mod.apply_multi(x, aid, cof, Ws, Us, inter, Ss)
    assert max(_rel(bad[m], ys[m]) for m in range(M)) > 1e-2
