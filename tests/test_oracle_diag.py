"""Pins of the oracle's diagonal-Sigma variant (Sec. 3.1, eq. JD-Diag):
y_t = (W + U_k diag(sigma_i) V_k^T) x_t.  Each test compares it with something
other than itself: a hand-worked example, the factored order written out as
loops, the full-Sigma oracle with a diagonal Sigma, the uncompressed oracle
(plain LoRA), and planted mistakes that must be caught."""
import json
import os

import numpy as np
import pytest

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "diag_worked_example.json")


def _golden():
    with open(GOLDEN) as f:
        g = json.load(f)
    arr = lambda k, dt=np.float64: np.asarray(g[k], dtype=dt)
    return g, arr


def _case(rs, T, d_in, d_out, r, n, K):
    x = rs.standard_normal((T, d_in))
    W = rs.standard_normal((d_out, d_in))
    U = rs.standard_normal((K, d_out, r))
    Vt = rs.standard_normal((K, r, d_in))
    sig = rs.standard_normal((n, r))
    aid = rs.integers(0, n, T).astype(np.int32)
    cof = rs.integers(0, K, n).astype(np.int32)
    return x, aid, cof, W, U, Vt, sig


def _rel(a, b):
    return np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300)


def _loops(x, aid, cof, W, U, Vt, sig):
    """The factored order V_k^T x -> scale by sigma_i -> U_k (.) plus W x, as
    plain loops (a different association from the oracle's explicit Delta_i)."""
    T, d_in = x.shape
    d_out, r = W.shape[0], sig.shape[1]
    y = np.zeros((T, d_out))
    for t in range(T):
        a = int(aid[t]); k = int(cof[a])
        z = [sum(Vt[k][q][j] * x[t][j] for j in range(d_in)) for q in range(r)]
        zs = [sig[a][q] * z[q] for q in range(r)]
        for o in range(d_out):
            y[t][o] = sum(W[o][j] * x[t][j] for j in range(d_in)) + sum(U[k][o][q] * zs[q] for q in range(r))
    return y


def test_diag_golden(oracle_mod):
    g, arr = _golden()
    y = oracle_mod.apply_diag(arr("x"), g["adapter_id"], g["cluster_of"], arr("W"), arr("U"), arr("Vt"),
                              arr("sigma"))
    np.testing.assert_array_equal(y, arr("y"))


@pytest.mark.parametrize("seed", [0, 1])
def test_diag_loops(oracle_mod, seed):
    rs = np.random.default_rng(100 + seed)
    args = _case(rs, 7, 6, 5, 3, 4, 2)
    assert _rel(oracle_mod.apply_diag(*args), _loops(*args)) < 1e-13


def test_diag_equals_full_sigma_with_diagonal(oracle_mod):
    rs = np.random.default_rng(102)
    x, aid, cof, W, U, Vt, sig = _case(rs, 11, 12, 10, 4, 5, 3)
    S = np.stack([np.diag(s) for s in sig])
    y_d = oracle_mod.apply_diag(x, aid, cof, W, U, Vt, sig)
    y_f = oracle_mod.apply(x, aid, cof, W, U, Vt, S)
    assert _rel(y_d, y_f) < 1e-14


def test_diag_single_adapter_is_plain_lora(oracle_mod):
    """One adapter in one cluster: B = U diag(sigma), A = V^T is a plain LoRA."""
    rs = np.random.default_rng(103)
    x, _, _, W, U, Vt, sig = _case(rs, 6, 9, 8, 3, 1, 1)
    aid, cof = np.zeros(6, np.int32), np.zeros(1, np.int32)
    B = (U[0] * sig[0][None, :])[None]
    A = Vt[0][None]
    y = oracle_mod.apply_diag(x, aid, cof, W, U, Vt, sig)
    assert _rel(y, oracle_mod.apply_uncompressed(x, aid, W, A, B)) < 1e-13


def test_diag_zero_sigma_is_base_layer(oracle_mod):
    rs = np.random.default_rng(104)
    x, aid, cof, W, U, Vt, sig = _case(rs, 5, 7, 6, 3, 3, 2)
    y = oracle_mod.apply_diag(x, aid, cof, W, U, Vt, np.zeros_like(sig))
    assert _rel(y, x @ W.T) < 1e-14


def test_diag_sampled_tokens_match_all(oracle_mod):
    rs = np.random.default_rng(105)
    args = _case(rs, 9, 6, 5, 2, 3, 2)
    tok = np.array([8, 0, 3, 3], np.int64)
    assert np.array_equal(oracle_mod.apply_diag(*args, tokens=tok), oracle_mod.apply_diag(*args)[tok])


# planted mistakes: each must move the result away from the loops / golden

def test_diag_planted_mistakes_are_caught(oracle_mod):
    g, arr = _golden()
    base = dict(x=arr("x"), aid=g["adapter_id"], cof=g["cluster_of"], W=arr("W"), U=arr("U"),
                Vt=arr("Vt"), sig=arr("sigma"))
    want = arr("y")

    def run(**kw):
        a = dict(base, **kw)
        return oracle_mod.apply_diag(a["x"], a["aid"], a["cof"], a["W"], a["U"], a["Vt"], a["sig"])

    assert not np.array_equal(run(sig=base["sig"][:, ::-1].copy()), want)          # diagonal order
    assert not np.array_equal(run(sig=base["sig"][::-1].copy()), want)             # wrong adapter
    assert not np.array_equal(run(U=np.transpose(base["U"], (0, 2, 1)).copy()), want)   # U^T
    assert not np.array_equal(run(cof=[1, 0]), want)                               # wrong cluster
    assert not np.array_equal(run(W=np.zeros((2, 2))), want)                       # dropped base
