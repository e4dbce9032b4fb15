"""Python face of the fp64 CPU oracle (``cts_oracle.c``).

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the benchmark's CPU
baseline leg are the only callers.  Nothing here is imported by the GPU
library, and nothing here imports it.

Conventions
-----------
* Arrays are numpy.  A ``uint16`` array holds bfloat16 bit patterns; it is
  widened exactly (bits << 16 reinterpreted as float32) before use.  float32
  and float64 arrays are widened exactly.  Every computation is in float64.
* Layouts follow the C file: ``x[T][d_in]``, ``W[d_out][d_in]``,
  ``U[K][d_out][r]``, ``Vt[K][r][d_in]`` (= V_k transposed), ``Sigma[n][r][r]``,
  ``A[n][r_l][d_in]``, ``B[n][d_out][r_l]``.

``apply_diag`` is the diagonal-Sigma variant of Sec. 3.1 (eq. JD-Diag) with
``sigma[n][r]`` holding the diagonals.  ``apply_ranked`` and
``apply_uncompressed_ranked`` take mixed ranks (a rank per cluster, Sec. 3.2;
a rank per uncompressed LoRA, App. H) over arrays stored at the largest rank.

Besides the apply/sort oracles this module holds ``exact_compress``: the
lossless JD-Full construction of Proposition 1 with Sigma_i taken from the
stationarity condition of App. A.1 (Sigma_i = U^T B_i A_i V).  It builds the
inputs of the exactness pins; it is not part of the serving path.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import time

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "cts_oracle.c")
# CTS_ORACLE_LIB names another build of the oracle (the sanitizer check's)
_LIB = os.environ.get("CTS_ORACLE_LIB") or os.path.join(_HERE, "libcts_oracle.so")
_lib = None


def build(force: bool = True, out: str | None = None, sanitize: bool = False) -> str:
    """Compile the oracle with gcc (fp64, OpenMP, no fast-math).  sanitize:
    with ROCm's clang and -fsanitize=address,undefined (the shared sanitizer
    runtime) into `out`, for the sanitizer check of the CPU tests."""
    lib = out or _LIB
    if force or not os.path.exists(lib):
        tmp = lib + ".tmp%d" % os.getpid()
        if sanitize:
            cmd = ["/opt/rocm/llvm/bin/clang", "-std=c11", "-O1", "-g", "-fno-omit-frame-pointer",
                   "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-shared-libsan",
                   "-fopenmp", "-fPIC", "-shared", "-Wall", "-Wextra", "-o", tmp, _SRC]
        else:
            cmd = ["gcc", "-std=c11", "-O3", "-fopenmp", "-fPIC", "-shared",
                   "-Wall", "-Wextra", "-o", tmp, _SRC]
        subprocess.run(cmd, check=True)
        os.replace(tmp, lib)
    return lib


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=True)
        lib = ctypes.CDLL(_LIB)
        i64, i32p, f64p = ctypes.c_int64, ctypes.POINTER(ctypes.c_int32), ctypes.POINTER(ctypes.c_double)
        i64p = ctypes.POINTER(ctypes.c_int64)
        lib.cts_oracle_num_threads.restype = ctypes.c_int
        lib.cts_oracle_sort_by_cluster.argtypes = [i32p, i64, i32p, i64, i64, i32p, i32p]
        lib.cts_oracle_sort_by_cluster.restype = ctypes.c_int
        lib.cts_oracle_apply.argtypes = [i64, i64, i64, i64, i64, i64, f64p, i32p, i32p,
                                         f64p, f64p, f64p, f64p, i64p, i64, f64p]
        lib.cts_oracle_apply.restype = ctypes.c_int
        lib.cts_oracle_apply_diag.argtypes = lib.cts_oracle_apply.argtypes
        lib.cts_oracle_apply_diag.restype = ctypes.c_int
        lib.cts_oracle_apply_ranked.argtypes = [i64, i64, i64, i64, i64, i64, f64p, i32p, i32p,
                                                f64p, f64p, f64p, f64p, i32p, i64p, i64, f64p]
        lib.cts_oracle_apply_ranked.restype = ctypes.c_int
        lib.cts_oracle_apply_uncompressed_ranked.argtypes = [i64, i64, i64, i64, i64, f64p, i32p,
                                                             f64p, f64p, f64p, i32p, i64p, i64, f64p]
        lib.cts_oracle_apply_uncompressed_ranked.restype = ctypes.c_int
        lib.cts_oracle_apply_uncompressed.argtypes = [i64, i64, i64, i64, i64, f64p, i32p,
                                                      f64p, f64p, f64p, i64p, i64, f64p]
        lib.cts_oracle_apply_uncompressed.restype = ctypes.c_int
        _lib = lib
    return _lib


def num_threads() -> int:
    return int(_load().cts_oracle_num_threads())


def to_f64(a) -> np.ndarray:
    """Exact widening to float64; uint16 means bfloat16 bit patterns."""
    a = np.asarray(a)
    if a.dtype == np.uint16:
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    if a.dtype in (np.float32, np.float64):
        return a.astype(np.float64)
    raise TypeError("oracle input must be float32, float64 or bf16 bits (uint16), got %s" % a.dtype)


def _c(a, ctype):
    return a.ctypes.data_as(ctypes.POINTER(ctype))


def _ids(a):
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


def sort_by_cluster(adapter_id, cluster_of, n: int, K: int):
    """(perm, offsets) for the key (cluster, adapter, token); cluster_of=None
    makes every adapter its own cluster (K == n)."""
    aid = _ids(adapter_id)
    T = aid.shape[0]
    perm = np.zeros(max(T, 1), np.int32)
    offs = np.zeros(K + 1, np.int32)
    cof = _ids(cluster_of) if cluster_of is not None else None
    rc = _load().cts_oracle_sort_by_cluster(
        _c(aid, ctypes.c_int32), T,
        _c(cof, ctypes.c_int32) if cof is not None else None, n, K,
        _c(perm, ctypes.c_int32), _c(offs, ctypes.c_int32))
    if rc != 0:
        raise ValueError("oracle sort rejected its input (code %d)" % rc)
    return perm[:T], offs


def _tokens(tokens, T):
    if tokens is None:
        tokens = np.arange(T, dtype=np.int64)
    return np.ascontiguousarray(np.asarray(tokens, dtype=np.int64))


def apply(x, adapter_id, cluster_of, W, U, Vt, Sigma, tokens=None, timing=None):
    """y[s] = (W + U_k Sigma_i V_k^T) x_t for t = tokens[s] (all tokens by
    default); returns float64 [len(tokens)][d_out].  If ``timing`` is a dict,
    the seconds spent inside the C call are stored under ``timing['s']``."""
    x64, W64, U64, V64, S64 = (np.ascontiguousarray(to_f64(a)) for a in (x, W, U, Vt, Sigma))
    aid, cof = _ids(adapter_id), _ids(cluster_of)
    T, d_in = x64.shape
    d_out = W64.shape[0]
    K, _, r = U64.shape
    n = S64.shape[0]
    assert W64.shape == (d_out, d_in) and V64.shape == (K, r, d_in) and S64.shape == (n, r, r)
    assert aid.shape == (T,) and cof.shape == (n,)
    tok = _tokens(tokens, T)
    y = np.zeros((max(len(tok), 1), d_out), np.float64)
    f = ctypes.c_double
    t0 = time.perf_counter()
    rc = _load().cts_oracle_apply(T, d_in, d_out, r, n, K, _c(x64, f), _c(aid, ctypes.c_int32),
                                  _c(cof, ctypes.c_int32), _c(W64, f), _c(U64, f), _c(V64, f),
                                  _c(S64, f), _c(tok, ctypes.c_int64), len(tok), _c(y, f))
    if timing is not None:
        timing["s"] = time.perf_counter() - t0
    if rc != 0:
        raise ValueError("oracle apply rejected its input (code %d)" % rc)
    return y[:len(tok)]


def apply_diag(x, adapter_id, cluster_of, W, U, Vt, sigma, tokens=None, timing=None):
    """Diagonal variant (Sec. 3.1, eq. JD-Diag): y[s] = (W + U_k diag(sigma_i)
    V_k^T) x_t for t = tokens[s], sigma [n][r] holding the diagonals; float64
    [len(tokens)][d_out]."""
    x64, W64, U64, V64, s64 = (np.ascontiguousarray(to_f64(a)) for a in (x, W, U, Vt, sigma))
    aid, cof = _ids(adapter_id), _ids(cluster_of)
    T, d_in = x64.shape
    d_out = W64.shape[0]
    K, _, r = U64.shape
    n = s64.shape[0]
    assert W64.shape == (d_out, d_in) and V64.shape == (K, r, d_in) and s64.shape == (n, r)
    assert aid.shape == (T,) and cof.shape == (n,)
    tok = _tokens(tokens, T)
    y = np.zeros((max(len(tok), 1), d_out), np.float64)
    f = ctypes.c_double
    t0 = time.perf_counter()
    rc = _load().cts_oracle_apply_diag(T, d_in, d_out, r, n, K, _c(x64, f), _c(aid, ctypes.c_int32),
                                       _c(cof, ctypes.c_int32), _c(W64, f), _c(U64, f), _c(V64, f),
                                       _c(s64, f), _c(tok, ctypes.c_int64), len(tok), _c(y, f))
    if timing is not None:
        timing["s"] = time.perf_counter() - t0
    if rc != 0:
        raise ValueError("oracle apply_diag rejected its input (code %d)" % rc)
    return y[:len(tok)]


def apply_multi(x, adapter_id, cluster_of, Ws, Us, Vt, Sigmas, tokens=None):
    """Several modules of one layer on the same x, ids and cluster map (Sec.
    3.1, 3.2 applied to each projection): module m is the layer with W_m, U_m,
    Sigma_m and the rows m r .. m r + r - 1 of the stacked Vt [K][M r][d_in].
    Returns the list of y_m."""
    r = np.asarray(Us[0]).shape[2]
    Vt = np.asarray(Vt)
    return [apply(x, adapter_id, cluster_of, Ws[m], Us[m], np.ascontiguousarray(Vt[:, m * r:(m + 1) * r, :]),
                  Sigmas[m], tokens=tokens) for m in range(len(Ws))]


def apply_ranked(x, adapter_id, cluster_of, W, U, Vt, Sigma, rank_of_cluster, tokens=None, timing=None):
    """Mixed ranks (Sec. 3.2: each cluster its own rank): y[s] = (W + U_k[:, :r_k]
    Sigma_i[:r_k, :r_k] V_k^T[:r_k, :]) x_t with r_k = rank_of_cluster[k]; U,
    Vt and Sigma are stored at the largest rank and the rest is never read."""
    x64, W64, U64, V64, S64 = (np.ascontiguousarray(to_f64(a)) for a in (x, W, U, Vt, Sigma))
    aid, cof, rk = _ids(adapter_id), _ids(cluster_of), _ids(rank_of_cluster)
    T, d_in = x64.shape
    d_out = W64.shape[0]
    K, _, r = U64.shape
    n = S64.shape[0]
    assert W64.shape == (d_out, d_in) and V64.shape == (K, r, d_in) and S64.shape == (n, r, r)
    assert aid.shape == (T,) and cof.shape == (n,) and rk.shape == (K,)
    tok = _tokens(tokens, T)
    y = np.zeros((max(len(tok), 1), d_out), np.float64)
    f = ctypes.c_double
    t0 = time.perf_counter()
    rc = _load().cts_oracle_apply_ranked(T, d_in, d_out, r, n, K, _c(x64, f), _c(aid, ctypes.c_int32),
                                         _c(cof, ctypes.c_int32), _c(W64, f), _c(U64, f), _c(V64, f),
                                         _c(S64, f), _c(rk, ctypes.c_int32), _c(tok, ctypes.c_int64),
                                         len(tok), _c(y, f))
    if timing is not None:
        timing["s"] = time.perf_counter() - t0
    if rc != 0:
        raise ValueError("oracle apply_ranked rejected its input (code %d)" % rc)
    return y[:len(tok)]


def apply_uncompressed_ranked(x, adapter_id, W, A, B, rank_of_adapter, tokens=None, timing=None):
    """Uncompressed LoRAs of different ranks (App. H): y[s] = (W + B_i[:, :r_i]
    A_i[:r_i, :]) x_t with r_i = rank_of_adapter[i]; A, B stored at the
    largest rank."""
    x64, W64, A64, B64 = (np.ascontiguousarray(to_f64(a)) for a in (x, W, A, B))
    aid, ra = _ids(adapter_id), _ids(rank_of_adapter)
    T, d_in = x64.shape
    d_out = W64.shape[0]
    n, r_l, _ = A64.shape
    assert W64.shape == (d_out, d_in) and A64.shape == (n, r_l, d_in) and B64.shape == (n, d_out, r_l)
    assert aid.shape == (T,) and ra.shape == (n,)
    tok = _tokens(tokens, T)
    y = np.zeros((max(len(tok), 1), d_out), np.float64)
    f = ctypes.c_double
    t0 = time.perf_counter()
    rc = _load().cts_oracle_apply_uncompressed_ranked(T, d_in, d_out, r_l, n, _c(x64, f),
                                                      _c(aid, ctypes.c_int32), _c(W64, f), _c(A64, f),
                                                      _c(B64, f), _c(ra, ctypes.c_int32),
                                                      _c(tok, ctypes.c_int64), len(tok), _c(y, f))
    if timing is not None:
        timing["s"] = time.perf_counter() - t0
    if rc != 0:
        raise ValueError("oracle apply_uncompressed_ranked rejected its input (code %d)" % rc)
    return y[:len(tok)]


def apply_uncompressed(x, adapter_id, W, A, B, tokens=None, timing=None):
    """y[s] = (W + B_i A_i) x_t for t = tokens[s]; float64 [len(tokens)][d_out]."""
    x64, W64, A64, B64 = (np.ascontiguousarray(to_f64(a)) for a in (x, W, A, B))
    aid = _ids(adapter_id)
    T, d_in = x64.shape
    d_out = W64.shape[0]
    n, r_l, _ = A64.shape
    assert W64.shape == (d_out, d_in) and A64.shape == (n, r_l, d_in) and B64.shape == (n, d_out, r_l)
    assert aid.shape == (T,)
    tok = _tokens(tokens, T)
    y = np.zeros((max(len(tok), 1), d_out), np.float64)
    f = ctypes.c_double
    t0 = time.perf_counter()
    rc = _load().cts_oracle_apply_uncompressed(T, d_in, d_out, r_l, n, _c(x64, f),
                                               _c(aid, ctypes.c_int32), _c(W64, f), _c(A64, f),
                                               _c(B64, f), _c(tok, ctypes.c_int64), len(tok),
                                               _c(y, f))
    if timing is not None:
        timing["s"] = time.perf_counter() - t0
    if rc != 0:
        raise ValueError("oracle apply_uncompressed rejected its input (code %d)" % rc)
    return y[:len(tok)]


def exact_compress(A, B):
    """Lossless single-cluster JD-Full of a LoRA collection (Prop. 1).

    U spans the columns of [B_1 ... B_n], V spans those of [A_1^T ... A_n^T]
    (orthonormal bases from QR), so r = r~ when the stacks have full column
    rank; Sigma_i = U^T B_i A_i V is the optimal core for fixed U, V (App. A.1,
    case 1).  Returns (U [d_out][r], Vt [r][d_in], Sigma [n][r][r]) in float64.
    """
    A64, B64 = to_f64(A), to_f64(B)
    n, r_l, d_in = A64.shape
    d_out = B64.shape[1]
    Bcat = np.concatenate([B64[i] for i in range(n)], axis=1)          # d_out x n r_l
    Acat = np.concatenate([A64[i].T for i in range(n)], axis=1)        # d_in  x n r_l
    U, _ = np.linalg.qr(Bcat)
    V, _ = np.linalg.qr(Acat)
    Sigma = np.stack([U.T @ (B64[i] @ (A64[i] @ V)) for i in range(n)])
    return U, np.ascontiguousarray(V.T), Sigma
