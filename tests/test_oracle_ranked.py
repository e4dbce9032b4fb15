"""Pins of the oracle's mixed-rank functions (Sec. 3.2: each cluster its own
rank; App. H: LoRAs of different ranks).  Arrays are stored at the largest
rank; a cluster (or uncompressed adapter) uses only its leading block.  The
pins: a hand-worked example with poison in the unused entries, the full-rank
oracles on zero-padded arrays, NaN in every unused entry, the plain-LoRA
reduction, and planted mistakes."""
import json
import os

import numpy as np
import pytest

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "ranked_worked_example.json")


def _rel(a, b):
    return np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300)


def _case(rs, T=9, d_in=10, d_out=8, r=6, n=5, K=3):
    x = rs.standard_normal((T, d_in))
    W = rs.standard_normal((d_out, d_in))
    U = rs.standard_normal((K, d_out, r))
    Vt = rs.standard_normal((K, r, d_in))
    S = rs.standard_normal((n, r, r))
    aid = rs.integers(0, n, T).astype(np.int32)
    cof = rs.integers(0, K, n).astype(np.int32)
    rk = rs.integers(0, r + 1, K).astype(np.int32)
    return x, aid, cof, W, U, Vt, S, rk


def _pad_compressed(U, Vt, S, cof, rk, fill):
    """Entries past each cluster's rank replaced by `fill`."""
    U, Vt, S = U.copy(), Vt.copy(), S.copy()
    for k, r_k in enumerate(rk):
        U[k][:, r_k:] = fill
        Vt[k][r_k:, :] = fill
    for i, k in enumerate(cof):
        r_k = rk[k]
        S[i][r_k:, :] = fill
        S[i][:, r_k:] = fill
    return U, Vt, S


def test_ranked_golden(oracle_mod):
    with open(GOLDEN) as f:
        g = json.load(f)
    a = lambda k: np.asarray(g[k], np.float64)
    y = oracle_mod.apply_ranked(a("x"), g["adapter_id"], g["cluster_of"], a("W"), a("U"), a("Vt"),
                                a("Sigma"), g["rank_of_cluster"])
    np.testing.assert_array_equal(y, a("y"))


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_ranked_equals_full_oracle_on_zero_padding(oracle_mod, seed):
    rs = np.random.default_rng(200 + seed)
    x, aid, cof, W, U, Vt, S, rk = _case(rs)
    Uz, Vz, Sz = _pad_compressed(U, Vt, S, cof, rk, 0.0)
    y_r = oracle_mod.apply_ranked(x, aid, cof, W, U, Vt, S, rk)
    y_f = oracle_mod.apply(x, aid, cof, W, Uz, Vz, Sz)
    assert _rel(y_r, y_f) < 1e-13


def test_ranked_never_reads_past_the_rank(oracle_mod):
    rs = np.random.default_rng(203)
    x, aid, cof, W, U, Vt, S, rk = _case(rs)
    Un, Vn, Sn = _pad_compressed(U, Vt, S, cof, rk, np.nan)
    y_clean = oracle_mod.apply_ranked(x, aid, cof, W, U, Vt, S, rk)
    y_nan = oracle_mod.apply_ranked(x, aid, cof, W, Un, Vn, Sn, rk)
    assert np.isfinite(y_nan).all()
    np.testing.assert_array_equal(y_nan, y_clean)


def test_ranked_full_ranks_is_apply(oracle_mod):
    rs = np.random.default_rng(204)
    x, aid, cof, W, U, Vt, S, rk = _case(rs)
    rk[:] = U.shape[2]
    assert _rel(oracle_mod.apply_ranked(x, aid, cof, W, U, Vt, S, rk),
                oracle_mod.apply(x, aid, cof, W, U, Vt, S)) < 1e-14


def test_ranked_single_adapter_is_plain_lora(oracle_mod):
    rs = np.random.default_rng(205)
    x, _, _, W, U, Vt, S, _ = _case(rs, n=1, K=1)
    r_k = 4
    aid, cof = np.zeros(len(x), np.int32), np.zeros(1, np.int32)
    B = U[0][:, :r_k] @ S[0][:r_k, :r_k]
    A = Vt[0][:r_k, :]
    y = oracle_mod.apply_ranked(x, aid, cof, W, U, Vt, S, np.array([r_k], np.int32))
    assert _rel(y, x @ (W + B @ A).T) < 1e-13


def test_uncompressed_ranked(oracle_mod):
    rs = np.random.default_rng(206)
    T, d_in, d_out, r_l, n = 8, 10, 7, 6, 4
    x = rs.standard_normal((T, d_in)); W = rs.standard_normal((d_out, d_in))
    A = rs.standard_normal((n, r_l, d_in)); B = rs.standard_normal((n, d_out, r_l))
    aid = rs.integers(0, n, T).astype(np.int32)
    ra = np.array([0, 2, 6, 3], np.int32)
    Az, Bz, An, Bn = A.copy(), B.copy(), A.copy(), B.copy()
    for i, r_i in enumerate(ra):
        Az[i][r_i:] = 0; Bz[i][:, r_i:] = 0
        An[i][r_i:] = np.nan; Bn[i][:, r_i:] = np.nan
    y = oracle_mod.apply_uncompressed_ranked(x, aid, W, A, B, ra)
    assert _rel(y, oracle_mod.apply_uncompressed(x, aid, W, Az, Bz)) < 1e-13
    np.testing.assert_array_equal(oracle_mod.apply_uncompressed_ranked(x, aid, W, An, Bn, ra), y)
    zero = aid == 0
    assert _rel(y[zero], x[zero] @ W.T) < 1e-14          # rank 0: the base layer


def test_ranked_rejects_bad_ranks(oracle_mod):
    rs = np.random.default_rng(207)
    x, aid, cof, W, U, Vt, S, rk = _case(rs)
    rk[0] = U.shape[2] + 1
    with pytest.raises(ValueError):
        oracle_mod.apply_ranked(x, aid, cof, W, U, Vt, S, rk)


def test_ranked_planted_mistakes_are_caught(oracle_mod):
    with open(GOLDEN) as f:
        g = json.load(f)
    a = lambda k: np.asarray(g[k], np.float64)
    want = a("y")
    run = lambda rk, cof=g["cluster_of"]: oracle_mod.apply_ranked(a("x"), g["adapter_id"], cof, a("W"),
                                                                   a("U"), a("Vt"), a("Sigma"), rk)
    assert not np.array_equal(run([2, 2]), want)          # the rank ignored: poison read
    assert not np.array_equal(run([2, 1]), want)          # ranks swapped between clusters
    assert not np.array_equal(run([1, 2], cof=[1, 0]), want)   # wrong cluster
