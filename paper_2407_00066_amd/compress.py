"""Offline compressor (include/cts_compress.h): JD-Full by the eigenvalue
iteration of App. A.2, JD-Diag by the alternating least squares of App. A.1
case 2 and the clustering of App. A.3, on the GPU.

Argument marshalling only, like the layer's binding: every step runs in
libcts.so's kernels.  Arrays are fp32 torch tensors on one device, in the
layouts of the C header: A [n][r_lora][d_in], B [n][d_out][r_lora], U
[d_out][r] (or [K][d_out][r]), Vt [r][d_in] (or [K][r][d_in]), Sigma [n][r][r].
"""
from __future__ import annotations

import ctypes

import torch

from ._binding import JdProblem, _check, _dev, _stream, _workspace, lib

F32 = torch.float32


def _problem(A, B, r):
    n, r_l, d_in = A.shape
    d_out = B.shape[1]
    return JdProblem(n, d_out, d_in, r_l, r), n, r_l, d_in, d_out


def workspace_size(A, B, r, K=0) -> int:
    p, *_ = _problem(A, B, r)
    if K:
        return int(lib().cts_jd_cluster_workspace_size(ctypes.byref(p), int(K)))
    return int(lib().cts_jd_workspace_size(ctypes.byref(p)))


def lora_norms2(A, B, r=16, workspace=None):
    """||B_i A_i||_F^2 for every LoRA ([n] fp32).  `r` only sizes the shared
    workspace plan (any valid JD rank)."""
    dev = A.device
    p, n, r_l, d_in, d_out = _problem(A, B, r)
    out = torch.empty(n, dtype=F32, device=dev)
    ws = _workspace(dev, workspace_size(A, B, r), workspace)
    _check(lib().cts_lora_norms2(ctypes.byref(p), _dev(A, "A", dev, F32, (n, r_l, d_in)),
                                 _dev(B, "B", dev, F32, (n, d_out, r_l)), _dev(out, "norms2", dev, F32, (n,)),
                                 ctypes.c_void_p(ws.data_ptr()), ws.numel(), _stream(dev)), "cts_lora_norms2")
    return out


def jd_full(A, B, U0, Vt0, iters=10, tau=0.0, normalize=False, workspace=None):
    """JD-Full by the eigenvalue iteration (cts_jd_full).  Returns
    (U, Vt, Sigma, crit[iters], iterations run)."""
    dev = A.device
    r = U0.shape[1]
    p, n, r_l, d_in, d_out = _problem(A, B, r)
    U = torch.empty((d_out, r), dtype=F32, device=dev)
    Vt = torch.empty((r, d_in), dtype=F32, device=dev)
    S = torch.empty((n, r, r), dtype=F32, device=dev)
    crit = torch.zeros(max(int(iters), 1), dtype=F32, device=dev)
    done = ctypes.c_int32(0)
    ws = _workspace(dev, workspace_size(A, B, r), workspace)
    _check(lib().cts_jd_full(ctypes.byref(p), _dev(A, "A", dev, F32, (n, r_l, d_in)),
                             _dev(B, "B", dev, F32, (n, d_out, r_l)), _dev(U0, "U0", dev, F32, (d_out, r)),
                             _dev(Vt0, "Vt0", dev, F32, (r, d_in)), int(iters), float(tau), int(bool(normalize)),
                             _dev(U, "U", dev, F32), _dev(Vt, "Vt", dev, F32), _dev(S, "Sigma", dev, F32),
                             _dev(crit, "crit", dev, F32), ctypes.byref(done), ctypes.c_void_p(ws.data_ptr()),
                             ws.numel(), _stream(dev)), "cts_jd_full")
    return U, Vt, S, crit, int(done.value)


def jd_diag(A, B, U0, Vt0, sweeps=10, normalize=False, workspace=None):
    """JD-Diag by alternating least squares (cts_jd_diag).  Returns
    (U [d_out][r], Vt [r][d_in], sigma [n][r])."""
    dev = A.device
    r = U0.shape[1]
    p, n, r_l, d_in, d_out = _problem(A, B, r)
    U = torch.empty((d_out, r), dtype=F32, device=dev)
    Vt = torch.empty((r, d_in), dtype=F32, device=dev)
    sig = torch.empty((n, r), dtype=F32, device=dev)
    ws = _workspace(dev, workspace_size(A, B, r), workspace)
    _check(lib().cts_jd_diag(ctypes.byref(p), _dev(A, "A", dev, F32, (n, r_l, d_in)),
                             _dev(B, "B", dev, F32, (n, d_out, r_l)), _dev(U0, "U0", dev, F32, (d_out, r)),
                             _dev(Vt0, "Vt0", dev, F32, (r, d_in)), int(sweeps), int(bool(normalize)),
                             _dev(U, "U", dev, F32), _dev(Vt, "Vt", dev, F32), _dev(sig, "sigma", dev, F32),
                             ctypes.c_void_p(ws.data_ptr()), ws.numel(), _stream(dev)), "cts_jd_diag")
    return U, Vt, sig


def jd_sigma(A, B, U, Vt, workspace=None):
    """Sigma_i = U^T B_i A_i V for given orthonormal bases (cts_jd_sigma)."""
    dev = A.device
    r = U.shape[1]
    p, n, r_l, d_in, d_out = _problem(A, B, r)
    S = torch.empty((n, r, r), dtype=F32, device=dev)
    ws = _workspace(dev, workspace_size(A, B, r), workspace)
    _check(lib().cts_jd_sigma(ctypes.byref(p), _dev(A, "A", dev, F32, (n, r_l, d_in)),
                              _dev(B, "B", dev, F32, (n, d_out, r_l)), _dev(U, "U", dev, F32, (d_out, r)),
                              _dev(Vt, "Vt", dev, F32, (r, d_in)), _dev(S, "Sigma", dev, F32),
                              ctypes.c_void_p(ws.data_ptr()), ws.numel(), _stream(dev)), "cts_jd_sigma")
    return S


def jd_cluster(A, B, K, U0, Vt0, Uc0, Vtc0, init_idx, jd_iters=10, max_rounds=20, normalize=False,
               workspace=None):
    """Clustering of App. A.3 (cts_jd_cluster).  init_idx: K LoRA indices
    (host sequence).  Returns (cluster_of [n] int32, U [K][d_out][r],
    Vt [K][r][d_in], Sigma [n][r][r], rounds)."""
    dev = A.device
    r = U0.shape[1]
    p, n, r_l, d_in, d_out = _problem(A, B, r)
    init = (ctypes.c_int32 * int(K))(*[int(v) for v in init_idx])
    if len(init_idx) != K:
        raise ValueError("init_idx must hold K indices")
    cof = torch.empty(n, dtype=torch.int32, device=dev)
    U = torch.empty((K, d_out, r), dtype=F32, device=dev)
    Vt = torch.empty((K, r, d_in), dtype=F32, device=dev)
    S = torch.empty((n, r, r), dtype=F32, device=dev)
    rounds = ctypes.c_int32(0)
    ws = _workspace(dev, workspace_size(A, B, r, K), workspace)
    _check(lib().cts_jd_cluster(ctypes.byref(p), int(K), _dev(A, "A", dev, F32, (n, r_l, d_in)),
                                _dev(B, "B", dev, F32, (n, d_out, r_l)), _dev(U0, "U0", dev, F32, (d_out, r)),
                                _dev(Vt0, "Vt0", dev, F32, (r, d_in)), _dev(Uc0, "Uc0", dev, F32, (K, d_out, r)),
                                _dev(Vtc0, "Vtc0", dev, F32, (K, r, d_in)), init, int(jd_iters), int(max_rounds),
                                int(bool(normalize)), _dev(cof, "cluster_of", dev, torch.int32),
                                _dev(U, "U", dev, F32), _dev(Vt, "Vt", dev, F32), _dev(S, "Sigma", dev, F32),
                                ctypes.byref(rounds), ctypes.c_void_p(ws.data_ptr()), ws.numel(), _stream(dev)),
           "cts_jd_cluster")
    return cof, U, Vt, S, int(rounds.value)
