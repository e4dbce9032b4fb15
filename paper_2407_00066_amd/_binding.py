"""ctypes binding of libcts.so (include/cts.h, include/cts_compress.h).

Argument marshalling only: shapes, dtypes and devices are checked, raw
device pointers and the current HIP stream are handed to the C library, and
every step of the layer runs in the library's kernels.  There is no fallback:
if libcts.so is missing, every call raises.
"""
from __future__ import annotations

import ctypes
import os
import threading

import torch

# CTS_LIB names another build of the library (the sanitizer check's)
_LIB_PATH = os.environ.get("CTS_LIB") or os.path.join(os.path.dirname(os.path.abspath(__file__)), "libcts.so")
_lib = None
_lock = threading.Lock()

CTS_OK, CTS_ERR_INVALID_ARG, CTS_ERR_UNSUPPORTED, CTS_ERR_WORKSPACE, CTS_ERR_HIP, CTS_ERR_BAD_IDS = range(6)
CTS_F32, CTS_BF16 = 0, 1

# every symbol include/cts.h declares
EXPORTED = ("cts_status_string", "cts_workspace_size", "cts_workspace_size_uncompressed",
            "cts_sort_by_cluster", "cts_apply", "cts_apply_diag", "cts_apply_ranked",
            "cts_apply_uncompressed", "cts_apply_uncompressed_ranked", "cts_validate_ids",
            "cts_set_stage_events", "cts_workspace_size_multi", "cts_apply_multi", "cts_apply_noalloc",
            "cts_workspace_bucketing", "cts_bucketing_size", "cts_apply_multi_sorted", "cts_apply_multi_packed",
            # include/cts_compress.h
            "cts_jd_workspace_size", "cts_jd_cluster_workspace_size", "cts_lora_norms2", "cts_jd_full",
            "cts_jd_diag", "cts_jd_sigma", "cts_jd_cluster")
N_STAGE_EVENTS = 6


class CtsError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        super().__init__("%s: %s" % (where, status_string(code)))


class JdProblem(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int32), ("d_out", ctypes.c_int32), ("d_in", ctypes.c_int32),
                ("r_lora", ctypes.c_int32), ("r", ctypes.c_int32)]


class Problem(ctypes.Structure):
    _fields_ = [("T", ctypes.c_int32), ("d_in", ctypes.c_int32), ("d_out", ctypes.c_int32),
                ("r", ctypes.c_int32), ("n_adapters", ctypes.c_int32),
                ("n_clusters", ctypes.c_int32), ("r_lora", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("out_dtype", ctypes.c_int32)]


def lib() -> ctypes.CDLL:
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        with _lock:
            if _lib is None:
                if not os.path.exists(_LIB_PATH):
                    raise RuntimeError("libcts.so is not built (%s); run "
                                       "`python -m paper_2407_00066_amd.build`" % _LIB_PATH)
                L = ctypes.CDLL(_LIB_PATH)
                vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
                pp = ctypes.POINTER(Problem)
                L.cts_status_string.argtypes = [ctypes.c_int]
                L.cts_status_string.restype = ctypes.c_char_p
                L.cts_workspace_size.argtypes = [pp]
                L.cts_workspace_size.restype = sz
                L.cts_workspace_size_uncompressed.argtypes = [pp]
                L.cts_workspace_size_uncompressed.restype = sz
                L.cts_workspace_bucketing.argtypes = [pp, i32, ctypes.POINTER(sz)]
                L.cts_workspace_bucketing.restype = ctypes.c_int
                L.cts_sort_by_cluster.argtypes = [vp, vp, i32, i32, i32, vp, vp, vp, sz, vp]
                L.cts_sort_by_cluster.restype = ctypes.c_int
                L.cts_bucketing_size.argtypes = [i32, i32, i32]
                L.cts_bucketing_size.restype = sz
                L.cts_apply.argtypes = [pp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
                L.cts_apply.restype = ctypes.c_int
                L.cts_apply_noalloc.argtypes = [pp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
                L.cts_apply_noalloc.restype = ctypes.c_int
                L.cts_apply_diag.argtypes = [pp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
                L.cts_apply_diag.restype = ctypes.c_int
                L.cts_apply_ranked.argtypes = [pp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
                L.cts_apply_ranked.restype = ctypes.c_int
                L.cts_apply_uncompressed_ranked.argtypes = [pp, vp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
                L.cts_apply_uncompressed_ranked.restype = ctypes.c_int
                L.cts_apply_uncompressed.argtypes = [pp, vp, vp, vp, vp, vp, vp, vp, sz, vp]
                L.cts_apply_uncompressed.restype = ctypes.c_int
                L.cts_validate_ids.argtypes = [pp, vp, vp, vp]
                L.cts_validate_ids.restype = ctypes.c_int
                L.cts_set_stage_events.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
                L.cts_set_stage_events.restype = ctypes.c_int
                i32p = ctypes.POINTER(i32)
                vpp = ctypes.POINTER(ctypes.c_void_p)
                L.cts_workspace_size_multi.argtypes = [pp, i32, i32p]
                L.cts_workspace_size_multi.restype = sz
                L.cts_apply_multi.argtypes = [pp, i32, i32p, vp, vp, vp, vpp, vpp, vp, vpp, vpp, vp, sz, vp]
                L.cts_apply_multi.restype = ctypes.c_int
                L.cts_apply_multi_sorted.argtypes = [pp, i32, i32p, vp, vp, sz, vp, vpp, vpp, vp, vpp, vpp, vp, sz, vp]
                L.cts_apply_multi_sorted.restype = ctypes.c_int
                L.cts_apply_multi_packed.argtypes = [pp, i32, i32p, vp, vp, vp, vp, sz, vp, vpp, vpp, vp, vpp, vp, i32,
                                                     vp, sz, vp]
                L.cts_apply_multi_packed.restype = ctypes.c_int
                jp, fl = ctypes.POINTER(JdProblem), ctypes.c_float
                L.cts_jd_workspace_size.argtypes = [jp]
                L.cts_jd_workspace_size.restype = sz
                L.cts_jd_cluster_workspace_size.argtypes = [jp, i32]
                L.cts_jd_cluster_workspace_size.restype = sz
                L.cts_lora_norms2.argtypes = [jp, vp, vp, vp, vp, sz, vp]
                L.cts_lora_norms2.restype = ctypes.c_int
                L.cts_jd_full.argtypes = [jp, vp, vp, vp, vp, i32, fl, i32, vp, vp, vp, vp,
                                          ctypes.POINTER(i32), vp, sz, vp]
                L.cts_jd_full.restype = ctypes.c_int
                L.cts_jd_diag.argtypes = [jp, vp, vp, vp, vp, i32, i32, vp, vp, vp, vp, sz, vp]
                L.cts_jd_diag.restype = ctypes.c_int
                L.cts_jd_sigma.argtypes = [jp, vp, vp, vp, vp, vp, vp, sz, vp]
                L.cts_jd_sigma.restype = ctypes.c_int
                L.cts_jd_cluster.argtypes = [jp, i32, vp, vp, vp, vp, vp, vp, ctypes.POINTER(i32), i32, i32,
                                             i32, vp, vp, vp, vp, ctypes.POINTER(i32), vp, sz, vp]
                L.cts_jd_cluster.restype = ctypes.c_int
                _lib = L
    return _lib


def status_string(code: int) -> str:
    return lib().cts_status_string(int(code)).decode()


def _check(code: int, where: str):
    if code != CTS_OK:
        raise CtsError(code, where)


_TORCH_DT = {torch.float32: CTS_F32, torch.bfloat16: CTS_BF16}


def _dt(t: torch.Tensor, name: str) -> int:
    if t.dtype not in _TORCH_DT:
        raise TypeError("%s must be float32 or bfloat16, got %s" % (name, t.dtype))
    return _TORCH_DT[t.dtype]


def _dev(t: torch.Tensor, name: str, device: torch.device, dtype=None, shape=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a torch.Tensor" % name)
    if t.device != device:
        raise ValueError("%s is on %s, expected %s" % (name, t.device, device))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    if dtype is not None and t.dtype != dtype:
        raise TypeError("%s must be %s, got %s" % (name, dtype, t.dtype))
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError("%s has shape %s, expected %s" % (name, tuple(t.shape), tuple(shape)))
    return ctypes.c_void_p(t.data_ptr()) if t.numel() else None


def _stream(device: torch.device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


_ws_cache: dict = {}


def _workspace(device: torch.device, nbytes: int, workspace):
    if workspace is not None:
        if workspace.device != device or workspace.dtype != torch.uint8:
            raise ValueError("workspace must be a uint8 tensor on %s" % device)
        return workspace
    ws = _ws_cache.get(device)
    if ws is None or ws.numel() < nbytes:
        ws = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=device)
        _ws_cache[device] = ws
    return ws


def make_problem(T, d_in, d_out, r=0, n_adapters=1, n_clusters=1, r_lora=0,
                 dtype=CTS_BF16, out_dtype=None) -> Problem:
    return Problem(T, d_in, d_out, r, n_adapters, n_clusters, r_lora, dtype,
                   dtype if out_dtype is None else out_dtype)


def workspace_size(p: Problem, compressed: bool = True) -> int:
    f = lib().cts_workspace_size if compressed else lib().cts_workspace_size_uncompressed
    return int(f(ctypes.byref(p)))


def workspace_bucketing(p: Problem, compressed: bool = True) -> dict:
    """Byte offsets of the bucketing a completed call leaves in its workspace
    (cts_workspace_bucketing): keys perm, seg, aid, items, n_items."""
    offs = (ctypes.c_size_t * 5)()
    _check(lib().cts_workspace_bucketing(ctypes.byref(p), 1 if compressed else 0, offs), "cts_workspace_bucketing")
    return dict(zip(("perm", "seg", "aid", "items", "n_items"), (int(v) for v in offs)))


def bucketing_size(T: int, n: int, K: int) -> int:
    return int(lib().cts_bucketing_size(T, n, K))


def sort_by_cluster(adapter_id: torch.Tensor, cluster_of: torch.Tensor | None, n: int, K: int,
                    perm: torch.Tensor | None = None, offsets: torch.Tensor | None = None,
                    bucketing=None):
    """(perm, cluster_offsets): tokens sorted by (cluster, adapter, token).
    bucketing: None, True (a new buffer) or a uint8 tensor of at least
    bucketing_size(T, n, K) bytes that receives the rest of the bucketing;
    then (perm, cluster_offsets, bucketing) is returned, and (perm,
    bucketing) can be passed to apply_multi_sorted."""
    dev = adapter_id.device
    T = adapter_id.numel()
    if perm is None:
        perm = torch.empty(T, dtype=torch.int32, device=dev)
    if offsets is None:
        offsets = torch.empty(K + 1, dtype=torch.int32, device=dev)
    a = _dev(adapter_id, "adapter_id", dev, torch.int32, (T,))
    c = _dev(cluster_of, "cluster_of", dev, torch.int32, (n,)) if cluster_of is not None else None
    pp = _dev(perm, "perm", dev, torch.int32, (T,))
    oo = _dev(offsets, "offsets", dev, torch.int32, (K + 1,))
    bk, bp, bn = None, None, 0
    if bucketing is not None:
        bk = bucketing if isinstance(bucketing, torch.Tensor) else \
            torch.empty(max(bucketing_size(T, n, K), 1), dtype=torch.uint8, device=dev)
        if bk.device != dev or bk.dtype != torch.uint8:
            raise ValueError("bucketing must be a uint8 tensor on %s" % dev)
        bp, bn = ctypes.c_void_p(bk.data_ptr()), bk.numel()
    _check(lib().cts_sort_by_cluster(a, c, T, n, K, pp, oo, bp, bn, _stream(dev)), "cts_sort_by_cluster")
    return (perm, offsets) if bk is None else (perm, offsets, bk)


def apply(x, adapter_id, cluster_of, W, U, Vt, Sigma, out=None, out_dtype=None, workspace=None):
    """y = W x_t + U_k Sigma_i V_k^T x_t per token (see include/cts.h)."""
    dev = x.device
    T, d_in = x.shape
    d_out = W.shape[0]
    K, _, r = U.shape
    n = Sigma.shape[0]
    dt = _dt(x, "x")
    tdt = x.dtype
    odt = tdt if out_dtype is None else out_dtype
    if out is None:
        out = torch.empty((T, d_out), dtype=odt, device=dev)
    p = make_problem(T, d_in, d_out, r=r, n_adapters=n, n_clusters=K, dtype=dt,
                     out_dtype=_dt(out, "out"))
    args = [_dev(x, "x", dev, tdt, (T, d_in)),
            _dev(adapter_id, "adapter_id", dev, torch.int32, (T,)),
            _dev(cluster_of, "cluster_of", dev, torch.int32, (n,)),
            _dev(W, "W", dev, tdt, (d_out, d_in)),
            _dev(U, "U", dev, tdt, (K, d_out, r)),
            _dev(Vt, "Vt", dev, tdt, (K, r, d_in)),
            _dev(Sigma, "Sigma", dev, tdt, (n, r, r)),
            _dev(out, "out", dev, None, (T, d_out))]
    nbytes = workspace_size(p, True)   # 0 for an invalid problem: cts_apply reports why
    ws = _workspace(dev, nbytes, workspace)
    _check(lib().cts_apply(ctypes.byref(p), *args, ctypes.c_void_p(ws.data_ptr()), ws.numel(),
                           _stream(dev)), "cts_apply")
    return out


# scratch bytes of cts_apply_noalloc (CTS_NOALLOC_SCRATCH_BYTES in include/cts.h)
NOALLOC_SCRATCH_BYTES = 48 << 20


def apply_noalloc(x, adapter_id, cluster_of, W, U, Vt, Sigma, out=None, out_dtype=None):
    """As apply, through cts_apply_noalloc: no workspace, the library's static
    per-device scratch array instead (see include/cts.h).  `out` is the
    caller's; when it is None a new output tensor is made here."""
    dev = x.device
    T, d_in = x.shape
    d_out = W.shape[0]
    K, _, r = U.shape
    n = Sigma.shape[0]
    dt = _dt(x, "x")
    tdt = x.dtype
    odt = tdt if out_dtype is None else out_dtype
    if out is None:
        out = torch.empty((T, d_out), dtype=odt, device=dev)
    p = make_problem(T, d_in, d_out, r=r, n_adapters=n, n_clusters=K, dtype=dt,
                     out_dtype=_dt(out, "out"))
    args = [_dev(x, "x", dev, tdt, (T, d_in)),
            _dev(adapter_id, "adapter_id", dev, torch.int32, (T,)),
            _dev(cluster_of, "cluster_of", dev, torch.int32, (n,)),
            _dev(W, "W", dev, tdt, (d_out, d_in)),
            _dev(U, "U", dev, tdt, (K, d_out, r)),
            _dev(Vt, "Vt", dev, tdt, (K, r, d_in)),
            _dev(Sigma, "Sigma", dev, tdt, (n, r, r)),
            _dev(out, "out", dev, None, (T, d_out))]
    _check(lib().cts_apply_noalloc(ctypes.byref(p), *args, _stream(dev)), "cts_apply_noalloc")
    return out


def apply_diag(x, adapter_id, cluster_of, W, U, Vt, sigma, out=None, out_dtype=None, workspace=None):
    """y = W x_t + U_k diag(sigma_i) V_k^T x_t per token, sigma [n][r] (see
    cts_apply_diag in include/cts.h)."""
    dev = x.device
    T, d_in = x.shape
    d_out = W.shape[0]
    K, _, r = U.shape
    n = sigma.shape[0]
    dt = _dt(x, "x")
    tdt = x.dtype
    odt = tdt if out_dtype is None else out_dtype
    if out is None:
        out = torch.empty((T, d_out), dtype=odt, device=dev)
    p = make_problem(T, d_in, d_out, r=r, n_adapters=n, n_clusters=K, dtype=dt,
                     out_dtype=_dt(out, "out"))
    args = [_dev(x, "x", dev, tdt, (T, d_in)),
            _dev(adapter_id, "adapter_id", dev, torch.int32, (T,)),
            _dev(cluster_of, "cluster_of", dev, torch.int32, (n,)),
            _dev(W, "W", dev, tdt, (d_out, d_in)),
            _dev(U, "U", dev, tdt, (K, d_out, r)),
            _dev(Vt, "Vt", dev, tdt, (K, r, d_in)),
            _dev(sigma, "sigma", dev, tdt, (n, r)),
            _dev(out, "out", dev, None, (T, d_out))]
    nbytes = workspace_size(p, True)
    ws = _workspace(dev, nbytes, workspace)
    _check(lib().cts_apply_diag(ctypes.byref(p), *args, ctypes.c_void_p(ws.data_ptr()), ws.numel(),
                                _stream(dev)), "cts_apply_diag")
    return out


def apply_ranked(x, adapter_id, cluster_of, W, U, Vt, Sigma, rank_of_cluster, out=None, out_dtype=None,
                 workspace=None):
    """Mixed ranks: as apply, cluster k using U_k[:, :r_k], Sigma_i[:r_k, :r_k],
    V_k^T[:r_k] with r_k = rank_of_cluster[k] (see cts_apply_ranked)."""
    dev = x.device
    T, d_in = x.shape
    d_out = W.shape[0]
    K, _, r = U.shape
    n = Sigma.shape[0]
    dt = _dt(x, "x")
    tdt = x.dtype
    odt = tdt if out_dtype is None else out_dtype
    if out is None:
        out = torch.empty((T, d_out), dtype=odt, device=dev)
    p = make_problem(T, d_in, d_out, r=r, n_adapters=n, n_clusters=K, dtype=dt,
                     out_dtype=_dt(out, "out"))
    args = [_dev(x, "x", dev, tdt, (T, d_in)),
            _dev(adapter_id, "adapter_id", dev, torch.int32, (T,)),
            _dev(cluster_of, "cluster_of", dev, torch.int32, (n,)),
            _dev(W, "W", dev, tdt, (d_out, d_in)),
            _dev(U, "U", dev, tdt, (K, d_out, r)),
            _dev(Vt, "Vt", dev, tdt, (K, r, d_in)),
            _dev(Sigma, "Sigma", dev, tdt, (n, r, r)),
            _dev(rank_of_cluster, "rank_of_cluster", dev, torch.int32, (K,)),
            _dev(out, "out", dev, None, (T, d_out))]
    nbytes = workspace_size(p, True)
    ws = _workspace(dev, nbytes, workspace)
    _check(lib().cts_apply_ranked(ctypes.byref(p), *args, ctypes.c_void_p(ws.data_ptr()), ws.numel(),
                                  _stream(dev)), "cts_apply_ranked")
    return out


def apply_uncompressed_ranked(x, adapter_id, W, A, B, rank_of_adapter, out=None, out_dtype=None,
                              workspace=None):
    """LoRAs of different ranks: as apply_uncompressed, adapter i using
    B_i[:, :r_i] A_i[:r_i] (see cts_apply_uncompressed_ranked)."""
    dev = x.device
    T, d_in = x.shape
    d_out = W.shape[0]
    n, r_l, _ = A.shape
    dt = _dt(x, "x")
    tdt = x.dtype
    odt = tdt if out_dtype is None else out_dtype
    if out is None:
        out = torch.empty((T, d_out), dtype=odt, device=dev)
    p = make_problem(T, d_in, d_out, n_adapters=n, r_lora=r_l, dtype=dt, out_dtype=_dt(out, "out"))
    args = [_dev(x, "x", dev, tdt, (T, d_in)),
            _dev(adapter_id, "adapter_id", dev, torch.int32, (T,)),
            _dev(W, "W", dev, tdt, (d_out, d_in)),
            _dev(A, "A", dev, tdt, (n, r_l, d_in)),
            _dev(B, "B", dev, tdt, (n, d_out, r_l)),
            _dev(rank_of_adapter, "rank_of_adapter", dev, torch.int32, (n,)),
            _dev(out, "out", dev, None, (T, d_out))]
    nbytes = workspace_size(p, False)
    ws = _workspace(dev, nbytes, workspace)
    _check(lib().cts_apply_uncompressed_ranked(ctypes.byref(p), *args, ctypes.c_void_p(ws.data_ptr()),
                                               ws.numel(), _stream(dev)), "cts_apply_uncompressed_ranked")
    return out


def apply_uncompressed(x, adapter_id, W, A, B, out=None, out_dtype=None, workspace=None):
    """y = W x_t + B_i A_i x_t per token (see include/cts.h)."""
    dev = x.device
    T, d_in = x.shape
    d_out = W.shape[0]
    n, r_l, _ = A.shape
    dt = _dt(x, "x")
    tdt = x.dtype
    odt = tdt if out_dtype is None else out_dtype
    if out is None:
        out = torch.empty((T, d_out), dtype=odt, device=dev)
    p = make_problem(T, d_in, d_out, n_adapters=n, r_lora=r_l, dtype=dt, out_dtype=_dt(out, "out"))
    args = [_dev(x, "x", dev, tdt, (T, d_in)),
            _dev(adapter_id, "adapter_id", dev, torch.int32, (T,)),
            _dev(W, "W", dev, tdt, (d_out, d_in)),
            _dev(A, "A", dev, tdt, (n, r_l, d_in)),
            _dev(B, "B", dev, tdt, (n, d_out, r_l)),
            _dev(out, "out", dev, None, (T, d_out))]
    nbytes = workspace_size(p, False)
    ws = _workspace(dev, nbytes, workspace)
    _check(lib().cts_apply_uncompressed(ctypes.byref(p), *args, ctypes.c_void_p(ws.data_ptr()),
                                        ws.numel(), _stream(dev)), "cts_apply_uncompressed")
    return out


def workspace_size_multi(p: Problem, d_out) -> int:
    arr = (ctypes.c_int32 * len(d_out))(*[int(v) for v in d_out])
    return int(lib().cts_workspace_size_multi(ctypes.byref(p), len(d_out), arr))


def apply_multi(x, adapter_id, cluster_of, Ws, Us, Vt, Sigmas, outs=None, out_dtype=None, workspace=None):
    """Several modules sharing x, the adapter ids and the cluster map
    (cts_apply_multi): Ws, Us, Sigmas are sequences of the modules' W_m,
    U_m, Sigma_m; Vt [K][M r][d_in] stacks their V_k^T along r.  Returns the
    list of outputs y_m [T][d_out_m]."""
    dev = x.device
    T, d_in = x.shape
    M = len(Ws)
    if not (len(Us) == len(Sigmas) == M):
        raise ValueError("Ws, Us and Sigmas must have one entry per module")
    K, _, r = Us[0].shape
    n = Sigmas[0].shape[0]
    dt = _dt(x, "x")
    tdt = x.dtype
    odt = tdt if out_dtype is None else out_dtype
    d_out = [int(w.shape[0]) for w in Ws]
    if outs is None:
        outs = [torch.empty((T, dm), dtype=odt, device=dev) for dm in d_out]
    p = make_problem(T, d_in, 8, r=r, n_adapters=n, n_clusters=K, dtype=dt, out_dtype=_dt(outs[0], "out"))
    vp = ctypes.c_void_p
    Wp = (vp * M)(*[_dev(w, "W[%d]" % m, dev, tdt, (d_out[m], d_in)) for m, w in enumerate(Ws)])
    Up = (vp * M)(*[_dev(u, "U[%d]" % m, dev, tdt, (K, d_out[m], r)) for m, u in enumerate(Us)])
    Sp = (vp * M)(*[_dev(sg, "Sigma[%d]" % m, dev, tdt, (n, r, r)) for m, sg in enumerate(Sigmas)])
    Yp = (vp * M)(*[_dev(y, "out[%d]" % m, dev, None, (T, d_out[m])) for m, y in enumerate(outs)])
    dims = (ctypes.c_int32 * M)(*d_out)
    nbytes = workspace_size_multi(p, d_out)
    ws = _workspace(dev, nbytes, workspace)
    _check(lib().cts_apply_multi(ctypes.byref(p), M, dims, _dev(x, "x", dev, tdt, (T, d_in)),
                                 _dev(adapter_id, "adapter_id", dev, torch.int32, (T,)),
                                 _dev(cluster_of, "cluster_of", dev, torch.int32, (n,)), Wp, Up,
                                 _dev(Vt, "Vt", dev, tdt, (K, M * r, d_in)), Sp, Yp,
                                 ctypes.c_void_p(ws.data_ptr()), ws.numel(), _stream(dev)), "cts_apply_multi")
    return outs


def apply_multi_sorted(perm, bucketing, x, Ws, Us, Vt, Sigmas, outs=None, out_dtype=None, workspace=None):
    """apply_multi with the bucketing of one sort_by_cluster(..., bucketing=...)
    call for this batch (cts_apply_multi_sorted): no ids, no sort here.
    Returns the list of outputs y_m [T][d_out_m]."""
    dev = x.device
    T, d_in = x.shape
    M = len(Ws)
    if not (len(Us) == len(Sigmas) == M):
        raise ValueError("Ws, Us and Sigmas must have one entry per module")
    K, _, r = Us[0].shape
    n = Sigmas[0].shape[0]
    dt = _dt(x, "x")
    tdt = x.dtype
    odt = tdt if out_dtype is None else out_dtype
    d_out = [int(w.shape[0]) for w in Ws]
    if outs is None:
        outs = [torch.empty((T, dm), dtype=odt, device=dev) for dm in d_out]
    p = make_problem(T, d_in, 8, r=r, n_adapters=n, n_clusters=K, dtype=dt, out_dtype=_dt(outs[0], "out"))
    vp = ctypes.c_void_p
    Wp = (vp * M)(*[_dev(w, "W[%d]" % m, dev, tdt, (d_out[m], d_in)) for m, w in enumerate(Ws)])
    Up = (vp * M)(*[_dev(u, "U[%d]" % m, dev, tdt, (K, d_out[m], r)) for m, u in enumerate(Us)])
    Sp = (vp * M)(*[_dev(sg, "Sigma[%d]" % m, dev, tdt, (n, r, r)) for m, sg in enumerate(Sigmas)])
    Yp = (vp * M)(*[_dev(y, "out[%d]" % m, dev, None, (T, d_out[m])) for m, y in enumerate(outs)])
    dims = (ctypes.c_int32 * M)(*d_out)
    if bucketing.device != dev or bucketing.dtype != torch.uint8:
        raise ValueError("bucketing must be a uint8 tensor on %s" % dev)
    nbytes = workspace_size_multi(p, d_out)
    ws = _workspace(dev, nbytes, workspace)
    _check(lib().cts_apply_multi_sorted(ctypes.byref(p), M, dims, _dev(perm, "perm", dev, torch.int32, (T,)),
                                        ctypes.c_void_p(bucketing.data_ptr()), bucketing.numel(),
                                        _dev(x, "x", dev, tdt, (T, d_in)), Wp, Up,
                                        _dev(Vt, "Vt", dev, tdt, (K, M * r, d_in)), Sp, Yp,
                                        ctypes.c_void_p(ws.data_ptr()), ws.numel(), _stream(dev)),
           "cts_apply_multi_sorted")
    return outs


def apply_multi_packed(x, Ws, Us, Vt, Sigmas, adapter_id=None, cluster_of=None, perm=None, bucketing=None,
                       out=None, out_dtype=None, workspace=None):
    """The multi-module layer into one packed output (cts_apply_multi_packed):
    module m's columns follow module m-1's in every row of out [T][ldy]
    (ldy = out's row length, at least the sum of the modules' d_out).  Give
    either (adapter_id, cluster_of) or (perm, bucketing) from
    sort_by_cluster.  Returns out."""
    dev = x.device
    T, d_in = x.shape
    M = len(Ws)
    if not (len(Us) == len(Sigmas) == M):
        raise ValueError("Ws, Us and Sigmas must have one entry per module")
    if (adapter_id is None) == (perm is None) or (adapter_id is None) != (cluster_of is None) or \
            (perm is None) != (bucketing is None):
        raise ValueError("give either (adapter_id, cluster_of) or (perm, bucketing)")
    K, _, r = Us[0].shape
    n = Sigmas[0].shape[0]
    dt = _dt(x, "x")
    tdt = x.dtype
    d_out = [int(w.shape[0]) for w in Ws]
    if out is None:
        out = torch.empty((T, sum(d_out)), dtype=tdt if out_dtype is None else out_dtype, device=dev)
    if out.dim() != 2 or out.shape[0] != T:
        raise ValueError("out must be [T][ldy]")
    p = make_problem(T, d_in, 8, r=r, n_adapters=n, n_clusters=K, dtype=dt, out_dtype=_dt(out, "out"))
    vp = ctypes.c_void_p
    Wp = (vp * M)(*[_dev(w, "W[%d]" % m, dev, tdt, (d_out[m], d_in)) for m, w in enumerate(Ws)])
    Up = (vp * M)(*[_dev(u, "U[%d]" % m, dev, tdt, (K, d_out[m], r)) for m, u in enumerate(Us)])
    Sp = (vp * M)(*[_dev(sg, "Sigma[%d]" % m, dev, tdt, (n, r, r)) for m, sg in enumerate(Sigmas)])
    dims = (ctypes.c_int32 * M)(*d_out)
    if bucketing is not None and (bucketing.device != dev or bucketing.dtype != torch.uint8):
        raise ValueError("bucketing must be a uint8 tensor on %s" % dev)
    ids = (_dev(adapter_id, "adapter_id", dev, torch.int32, (T,)), _dev(cluster_of, "cluster_of", dev, torch.int32,
                                                                      (n,))) if adapter_id is not None else (None, None)
    srt = (_dev(perm, "perm", dev, torch.int32, (T,)), ctypes.c_void_p(bucketing.data_ptr()),
           bucketing.numel()) if perm is not None else (None, None, 0)
    nbytes = workspace_size_multi(p, d_out)
    ws = _workspace(dev, nbytes, workspace)
    _check(lib().cts_apply_multi_packed(ctypes.byref(p), M, dims, *ids, *srt, _dev(x, "x", dev, tdt, (T, d_in)),
                                        Wp, Up, _dev(Vt, "Vt", dev, tdt, (K, M * r, d_in)), Sp,
                                        _dev(out, "out", dev, None, tuple(out.shape)), int(out.shape[1]),
                                        ctypes.c_void_p(ws.data_ptr()), ws.numel(), _stream(dev)),
           "cts_apply_multi_packed")
    return out


def validate_ids(adapter_id, cluster_of, n: int, K: int = 1) -> bool:
    """True if every id is in range (synchronous; for tests and debugging)."""
    dev = adapter_id.device
    T = adapter_id.numel()
    p = make_problem(T, 8, 8, n_adapters=n, n_clusters=K)
    a = _dev(adapter_id, "adapter_id", dev, torch.int32, (T,))
    c = _dev(cluster_of, "cluster_of", dev, torch.int32, (n,)) if cluster_of is not None else None
    code = lib().cts_validate_ids(ctypes.byref(p), a, c, _stream(dev))
    if code == CTS_ERR_BAD_IDS:
        return False
    _check(code, "cts_validate_ids")
    return True


def set_stage_events(events) -> None:
    """Profiling aid: `events` is None (off) or N_STAGE_EVENTS entries, each a
    torch.cuda.Event (enable_timing=True) or None (not recorded), recorded at
    the layer's stage boundaries by every later apply call (see
    cts_set_stage_events in include/cts.h)."""
    if events is None:
        _check(lib().cts_set_stage_events(None), "cts_set_stage_events")
        return
    if len(events) != N_STAGE_EVENTS:
        raise ValueError("need %d events" % N_STAGE_EVENTS)
    for e in events:
        if e is not None and e.cuda_event == 0:   # torch creates the HIP event at its first record
            e.record()
    arr = (ctypes.c_void_p * N_STAGE_EVENTS)(*[e.cuda_event if e is not None else None for e in events])
    _check(lib().cts_set_stage_events(arr), "cts_set_stage_events")
