"""The C-ABI library loads, exports every symbol include/*.h declares, and
rejects every host-detectable argument error before touching HIP.  CPU only:
no call here reaches a kernel launch."""
import ctypes
import os
import re

import pytest

import paper_2407_00066_amd as cts
from paper_2407_00066_amd import _binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = [os.path.join(ROOT, "include", f) for f in sorted(os.listdir(os.path.join(ROOT, "include")))
           if f.endswith(".h")]

FAKE = ctypes.c_void_p(0x10000)   # never dereferenced: validation fails first (16-byte aligned)


def _declared():
    names = set()
    for h in HEADERS:
        src = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        names |= set(re.findall(r"\b(cts_[a-z0-9_]+)\s*\(", src))
    return sorted(names)


def test_header_declares_binding_symbols():
    assert _declared() == sorted(B.EXPORTED)


def test_library_exports_every_declared_symbol():
    L = cts.lib()
    for name in _declared():
        assert hasattr(L, name), name


def test_status_strings():
    for code in range(6):
        assert cts.status_string(code).startswith("CTS_")
    assert cts.status_string(99) == "CTS_ERR_UNKNOWN"


def _p(**kw):
    base = dict(T=64, d_in=4096, d_out=4096, r=64, n_adapters=100, n_clusters=1, r_lora=16)
    base.update(kw)
    return cts.make_problem(**base)


def _apply(p, ptrs=None, ws_bytes=1 << 40, y=None, ws=None):
    ptrs = ptrs or [FAKE] * 7
    y = y if y is not None else ctypes.c_void_p(0x7000_0000_0000)
    ws = ws if ws is not None else ctypes.c_void_p(0x6000_0000_0000)
    return cts.lib().cts_apply(ctypes.byref(p), *ptrs[:7], y, ws, ws_bytes, None)


def _apply_u(p, ws_bytes=1 << 40):
    return cts.lib().cts_apply_uncompressed(ctypes.byref(p), *[FAKE] * 5,
                                            ctypes.c_void_p(0x7000_0000_0000),
                                            ctypes.c_void_p(0x6000_0000_0000), ws_bytes, None)


@pytest.mark.parametrize("kw,code", [
    (dict(T=-1), B.CTS_ERR_INVALID_ARG), (dict(d_in=0), B.CTS_ERR_INVALID_ARG),
    (dict(d_out=-8), B.CTS_ERR_INVALID_ARG), (dict(r=0), B.CTS_ERR_INVALID_ARG),
    (dict(n_adapters=0), B.CTS_ERR_INVALID_ARG), (dict(n_clusters=0), B.CTS_ERR_INVALID_ARG),
    (dict(d_in=4100), B.CTS_ERR_UNSUPPORTED), (dict(d_out=12), B.CTS_ERR_UNSUPPORTED),
    (dict(r=12), B.CTS_ERR_UNSUPPORTED), (dict(r=136), B.CTS_ERR_UNSUPPORTED),
    (dict(n_adapters=65537), B.CTS_ERR_UNSUPPORTED),
    (dict(dtype=2), B.CTS_ERR_UNSUPPORTED), (dict(out_dtype=7), B.CTS_ERR_UNSUPPORTED),
    (dict(dtype=B.CTS_F32, out_dtype=B.CTS_BF16), B.CTS_ERR_UNSUPPORTED),
])
def test_apply_rejects_bad_problem(kw, code):
    assert _apply(_p(**kw)) == code
    assert cts.workspace_size(_p(**kw)) == 0


def test_apply_null_problem():
    assert cts.lib().cts_apply(None, *[FAKE] * 9, 0, None) == B.CTS_ERR_INVALID_ARG


def test_apply_null_pointers():
    p = _p()
    for i in range(7):
        ptrs = [FAKE] * 7
        ptrs[i] = None
        assert _apply(p, ptrs) == B.CTS_ERR_INVALID_ARG, i
    assert _apply(p, y=ctypes.c_void_p(0)) == B.CTS_ERR_INVALID_ARG


def test_apply_rejects_misaligned_pointers():
    p = _p()
    for i in range(7):
        ptrs = [ctypes.c_void_p(0x5000_0000_0000 + k * (1 << 32)) for k in range(7)]
        ptrs[i] = ctypes.c_void_p(ptrs[i].value + (2 if i in (1, 2) else 8))
        assert _apply(p, ptrs) == B.CTS_ERR_INVALID_ARG, i
    assert _apply(p, y=ctypes.c_void_p(0x7000_0000_0000 + 8)) == B.CTS_ERR_INVALID_ARG
    assert _apply(p, ws=ctypes.c_void_p(0x6000_0000_0000 + 4)) == B.CTS_ERR_INVALID_ARG


def test_apply_t0_is_noop_without_pointers():
    p = _p(T=0)
    assert cts.lib().cts_apply(ctypes.byref(p), *[None] * 9, 0, None) == B.CTS_OK
    assert cts.lib().cts_apply_uncompressed(ctypes.byref(p), *[None] * 7, 0, None) == B.CTS_OK


def test_apply_workspace_too_small():
    p = _p()
    need = cts.workspace_size(p)
    assert need > 0
    assert _apply(p, ws_bytes=need - 1) == B.CTS_ERR_WORKSPACE


def test_apply_rejects_overlaps():
    p = _p(T=64, d_in=64, d_out=64, r=8, n_adapters=4)
    base = 0x5000_0000_0000
    # inputs far apart; y placed inside W
    ptrs = [ctypes.c_void_p(base + i * (1 << 30)) for i in range(7)]
    assert _apply(p, ptrs, y=ctypes.c_void_p(base + 3 * (1 << 30) + 64)) == B.CTS_ERR_INVALID_ARG
    # workspace overlapping x
    assert _apply(p, ptrs, ws=ctypes.c_void_p(base + 128)) == B.CTS_ERR_INVALID_ARG
    # y overlapping the workspace
    assert _apply(p, ptrs, y=ctypes.c_void_p(0x6000_0000_0000 + 256)) == B.CTS_ERR_INVALID_ARG


@pytest.mark.parametrize("kw,code", [
    (dict(r_lora=0), B.CTS_ERR_INVALID_ARG), (dict(r_lora=12), B.CTS_ERR_UNSUPPORTED),
    (dict(r_lora=4, dtype=B.CTS_F32, out_dtype=B.CTS_F32, T=0), B.CTS_OK),
    (dict(r_lora=136), B.CTS_ERR_UNSUPPORTED),
])
def test_uncompressed_validation(kw, code):
    assert _apply_u(_p(**kw)) == code


def test_uncompressed_ignores_compressed_fields():
    p = _p(r=0, n_clusters=0, r_lora=16)
    assert cts.workspace_size(p, compressed=False) > 0
    assert _apply_u(p, ws_bytes=1) == B.CTS_ERR_WORKSPACE


def _pieces(T, cap=8192):
    """Token counts of the pieces a batch of T tokens runs as: ceil(T / cap)
    near-equal pieces, the larger ones first."""
    n = max(1, -(-T // cap))
    q, rem = divmod(T, n)
    return [q + 1] * rem + [q] * (n - rem)


@pytest.mark.parametrize("T", [8193, 16384, 16385, 20000, 100000])
def test_large_batches_run_in_pieces(T):
    """Above 8192 tokens a call runs as pieces of at most 8192 tokens: its
    workspace is the largest any piece needs, for every entry point, and the
    pieces' validation is the whole batch's."""
    pieces = _pieces(T)
    assert sum(pieces) == T and max(pieces) <= 8192 and max(pieces) - min(pieces) <= 1
    kw = dict(n_clusters=25, n_adapters=1000)
    ws = cts.workspace_size(_p(T=T, **kw))
    assert ws > 0 and ws == max(cts.workspace_size(_p(T=q, **kw)) for q in set(pieces))
    wsu = cts.workspace_size(_p(T=T, **kw), compressed=False)
    assert wsu == max(cts.workspace_size(_p(T=q, **kw), compressed=False) for q in set(pieces))
    wsm = cts.workspace_size_multi(_p(T=T, **kw), [64, 128])
    assert wsm == max(cts.workspace_size_multi(_p(T=q, **kw), [64, 128]) for q in set(pieces))
    # an undersized workspace is still refused for the whole call
    assert _apply(_p(T=T, **kw), ws_bytes=ws - 1) == B.CTS_ERR_WORKSPACE
    # the bucketing read-back describes one piece's sort: refused for pieces
    offs = (ctypes.c_size_t * 5)()
    assert cts.lib().cts_workspace_bucketing(ctypes.byref(_p(T=T, **kw)), 1, offs) == B.CTS_ERR_UNSUPPORTED
    assert cts.lib().cts_workspace_bucketing(ctypes.byref(_p(T=8192, **kw)), 1, offs) == B.CTS_OK


def test_workspace_grows_with_problem():
    small = cts.workspace_size(_p(T=32))
    big = cts.workspace_size(_p(T=4096, n_clusters=25, n_adapters=1000))
    assert 0 < small < big
    assert cts.workspace_size(_p(T=0)) >= 0


def test_sort_validation():
    L = cts.lib()
    f = lambda *a: L.cts_sort_by_cluster(*a, None, 0, None)
    assert f(FAKE, FAKE, -1, 4, 2, FAKE, FAKE) == B.CTS_ERR_INVALID_ARG
    assert f(FAKE, FAKE, 4, 0, 2, FAKE, FAKE) == B.CTS_ERR_INVALID_ARG
    assert f(FAKE, None, 4, 4, 2, FAKE, FAKE) == B.CTS_ERR_INVALID_ARG   # K must equal n
    assert f(None, FAKE, 4, 4, 2, FAKE, FAKE) == B.CTS_ERR_INVALID_ARG
    assert f(FAKE, FAKE, 4, 4, 2, FAKE, None) == B.CTS_ERR_INVALID_ARG
    assert f(FAKE, FAKE, 9000, 4, 2, ctypes.c_void_p(0x9000_0000), ctypes.c_void_p(0xA000_0000)) \
        == B.CTS_ERR_UNSUPPORTED
    # perm overlapping cluster_offsets
    assert f(ctypes.c_void_p(0x1000_0000), ctypes.c_void_p(0x2000_0000), 64, 4, 2,
             ctypes.c_void_p(0x3000_0000), ctypes.c_void_p(0x3000_0000 + 8)) == B.CTS_ERR_INVALID_ARG


def test_validate_ids_rejects_bad_problem():
    L = cts.lib()
    assert L.cts_validate_ids(None, FAKE, FAKE, None) == B.CTS_ERR_INVALID_ARG
    p = _p(T=4, n_adapters=0)
    assert L.cts_validate_ids(ctypes.byref(p), FAKE, FAKE, None) == B.CTS_ERR_INVALID_ARG


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(B, "_lib", None)
    monkeypatch.setattr(B, "_LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(RuntimeError, match="not built"):
        B.lib()


# the diagonal-Sigma entry point validates exactly as cts_apply does

def _apply_d(p, ptrs=None, ws_bytes=1 << 40, y=None, ws=None):
    ptrs = ptrs or [FAKE] * 7
    y = y if y is not None else ctypes.c_void_p(0x7000_0000_0000)
    ws = ws if ws is not None else ctypes.c_void_p(0x6000_0000_0000)
    return cts.lib().cts_apply_diag(ctypes.byref(p), *ptrs[:7], y, ws, ws_bytes, None)


@pytest.mark.parametrize("kw,code", [
    (dict(T=-1), B.CTS_ERR_INVALID_ARG), (dict(r=0), B.CTS_ERR_INVALID_ARG),
    (dict(n_clusters=0), B.CTS_ERR_INVALID_ARG), (dict(r=12), B.CTS_ERR_UNSUPPORTED),
    (dict(dtype=2), B.CTS_ERR_UNSUPPORTED),
])
def test_apply_diag_rejects_bad_problem(kw, code):
    assert _apply_d(_p(**kw)) == code


def test_apply_diag_null_and_misaligned_pointers():
    p = _p()
    assert cts.lib().cts_apply_diag(None, *[FAKE] * 9, 0, None) == B.CTS_ERR_INVALID_ARG
    for i in range(7):
        ptrs = [FAKE] * 7
        ptrs[i] = None
        assert _apply_d(p, ptrs) == B.CTS_ERR_INVALID_ARG, i
    ptrs = [ctypes.c_void_p(0x5000_0000_0000 + k * (1 << 32)) for k in range(7)]
    ptrs[6] = ctypes.c_void_p(ptrs[6].value + 8)          # sigma not 16-byte aligned
    assert _apply_d(p, ptrs) == B.CTS_ERR_INVALID_ARG
    assert _apply_d(p, ws_bytes=cts.workspace_size(p) - 1) == B.CTS_ERR_WORKSPACE
    assert cts.lib().cts_apply_diag(ctypes.byref(_p(T=0)), *[None] * 9, 0, None) == B.CTS_OK


def test_apply_diag_rejects_overlap_with_sigma():
    # y overlapping sigma: sigma is n x r here (not n x r x r)
    p = _p(n_adapters=4, r=64)
    base = 0x5000_0000_0000
    ptrs = [ctypes.c_void_p(base + k * (1 << 32)) for k in range(7)]
    y = ctypes.c_void_p(ptrs[6].value + 256)               # inside sigma's 4 * 64 * 2 bytes
    assert _apply_d(p, ptrs, y=y) == B.CTS_ERR_INVALID_ARG


# mixed-rank entry points: the rank table is one more checked pointer

def test_apply_ranked_validation():
    p = _p(n_clusters=4)
    L = cts.lib()
    ptr = lambda k: ctypes.c_void_p(0x5000_0000_0000 + k * (1 << 32))
    y, ws = ctypes.c_void_p(0x7000_0000_0000), ctypes.c_void_p(0x6000_0000_0000)
    ins = [ptr(k) for k in range(7)]
    assert L.cts_apply_ranked(None, *ins, ptr(7), y, ws, 1 << 40, None) == B.CTS_ERR_INVALID_ARG
    assert L.cts_apply_ranked(ctypes.byref(p), *ins, None, y, ws, 1 << 40, None) == B.CTS_ERR_INVALID_ARG
    bad = ctypes.c_void_p(ptr(7).value + 2)                # rank table not 4-byte aligned
    assert L.cts_apply_ranked(ctypes.byref(p), *ins, bad, y, ws, 1 << 40, None) == B.CTS_ERR_INVALID_ARG
    on_y = ctypes.c_void_p(y.value + 64)                   # rank table inside y
    assert L.cts_apply_ranked(ctypes.byref(p), *ins, on_y, y, ws, 1 << 40, None) == B.CTS_ERR_INVALID_ARG
    need = cts.workspace_size(p)
    assert L.cts_apply_ranked(ctypes.byref(p), *ins, ptr(7), y, ws, need - 1, None) == B.CTS_ERR_WORKSPACE
    assert L.cts_apply_ranked(ctypes.byref(_p(T=0)), *[None] * 8, None, None, 0, None) == B.CTS_OK
    assert L.cts_apply_ranked(ctypes.byref(_p(r=12)), *ins, ptr(7), y, ws, 1 << 40, None) == B.CTS_ERR_UNSUPPORTED


def test_apply_uncompressed_ranked_validation():
    p = _p()
    L = cts.lib()
    ptr = lambda k: ctypes.c_void_p(0x5000_0000_0000 + k * (1 << 32))
    y, ws = ctypes.c_void_p(0x7000_0000_0000), ctypes.c_void_p(0x6000_0000_0000)
    ins = [ptr(k) for k in range(5)]
    assert L.cts_apply_uncompressed_ranked(ctypes.byref(p), *ins, None, y, ws, 1 << 40, None) == B.CTS_ERR_INVALID_ARG
    bad = ctypes.c_void_p(ptr(5).value + 1)
    assert L.cts_apply_uncompressed_ranked(ctypes.byref(p), *ins, bad, y, ws, 1 << 40, None) == B.CTS_ERR_INVALID_ARG
    need = cts.workspace_size(p, compressed=False)
    assert L.cts_apply_uncompressed_ranked(ctypes.byref(p), *ins, ptr(5), y, ws, need - 1,
                                           None) == B.CTS_ERR_WORKSPACE
    assert L.cts_apply_uncompressed_ranked(ctypes.byref(_p(T=0)), *[None] * 6, None, None, 0,
                                           None) == B.CTS_OK


# ------------------------------------------------------------ compressor ABI
def _jp(**kw):
    d = dict(n=8, d_out=64, d_in=64, r_lora=4, r=16)
    d.update(kw)
    return B.JdProblem(d["n"], d["d_out"], d["d_in"], d["r_lora"], d["r"])


@pytest.mark.parametrize("kw,code", [
    (dict(n=0), B.CTS_ERR_INVALID_ARG), (dict(r=0), B.CTS_ERR_INVALID_ARG),
    (dict(r=24), B.CTS_ERR_UNSUPPORTED), (dict(r=144), B.CTS_ERR_UNSUPPORTED),
    (dict(r_lora=12), B.CTS_ERR_UNSUPPORTED), (dict(n=3, r=16), B.CTS_ERR_UNSUPPORTED),
    (dict(d_in=62), B.CTS_ERR_UNSUPPORTED), (dict(d_out=8), B.CTS_ERR_UNSUPPORTED),
])
def test_jd_rejects_bad_problem(kw, code):
    p = _jp(**kw)
    L = cts.lib()
    assert L.cts_jd_workspace_size(ctypes.byref(p)) == 0
    done = ctypes.c_int32(0)
    rc = L.cts_jd_full(ctypes.byref(p), FAKE, FAKE, FAKE, FAKE, 3, 0.0, 0, FAKE, FAKE, FAKE, FAKE,
                       ctypes.byref(done), FAKE, 1 << 30, None)
    assert rc == code
    assert L.cts_jd_sigma(ctypes.byref(p), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 30, None) == code
    assert L.cts_jd_diag(ctypes.byref(p), FAKE, FAKE, FAKE, FAKE, 3, 0, FAKE, FAKE, FAKE, FAKE, 1 << 30,
                         None) == code
    assert L.cts_lora_norms2(ctypes.byref(p), FAKE, FAKE, FAKE, FAKE, 1 << 30, None) == code


def test_jd_full_argument_errors():
    p = _jp()
    L = cts.lib()
    need = L.cts_jd_workspace_size(ctypes.byref(p))
    assert need > 0
    done = ctypes.c_int32(0)
    odd = ctypes.c_void_p(0x10004)
    args = [FAKE, FAKE, FAKE, FAKE, 3, 0.0, 0, FAKE, FAKE, FAKE, FAKE, ctypes.byref(done), FAKE, need, None]
    for i in (0, 1, 2, 3, 7, 8, 9, 10, 12):                 # each pointer null, then misaligned
        a = list(args)
        a[i] = None
        assert L.cts_jd_full(ctypes.byref(p), *a) == B.CTS_ERR_INVALID_ARG, i
        if i != 10:                                          # crit needs 4-byte alignment only
            a[i] = odd
            assert L.cts_jd_full(ctypes.byref(p), *a) == B.CTS_ERR_INVALID_ARG, i
    a = list(args)
    a[4] = 0                                                 # iters
    assert L.cts_jd_full(ctypes.byref(p), *a) == B.CTS_ERR_INVALID_ARG
    a = list(args)
    a[13] = need - 1
    assert L.cts_jd_full(ctypes.byref(p), *a) == B.CTS_ERR_WORKSPACE
    assert L.cts_jd_sigma(ctypes.byref(p), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, need - 1, None) == \
        B.CTS_ERR_WORKSPACE
    assert L.cts_lora_norms2(ctypes.byref(p), FAKE, FAKE, FAKE, FAKE, need - 1, None) == B.CTS_ERR_WORKSPACE
    assert L.cts_jd_full(None, *args) == B.CTS_ERR_INVALID_ARG


def test_jd_cluster_argument_errors():
    p = _jp()
    L = cts.lib()
    K = 2
    need = L.cts_jd_cluster_workspace_size(ctypes.byref(p), K)
    assert need > L.cts_jd_workspace_size(ctypes.byref(p))
    assert L.cts_jd_cluster_workspace_size(ctypes.byref(p), 0) == 0
    assert L.cts_jd_cluster_workspace_size(ctypes.byref(p), 9) == 0        # K > n
    rounds = ctypes.c_int32(0)

    def call(K=2, init=(0, 1), jd_iters=3, max_rounds=5, ws=need, **ptrs):
        arr = (ctypes.c_int32 * len(init))(*init)
        P = dict(A=FAKE, B=FAKE, U0=FAKE, Vt0=FAKE, Uc0=FAKE, Vtc0=FAKE, cof=FAKE, U=FAKE, Vt=FAKE, S=FAKE,
                 W=FAKE)
        P.update(ptrs)
        return L.cts_jd_cluster(ctypes.byref(p), K, P["A"], P["B"], P["U0"], P["Vt0"], P["Uc0"], P["Vtc0"], arr,
                                jd_iters, max_rounds, 0, P["cof"], P["U"], P["Vt"], P["S"],
                                ctypes.byref(rounds), P["W"], ws, None)

    assert call(K=0, init=(0,)) == B.CTS_ERR_INVALID_ARG
    assert call(K=9, init=tuple(range(9))) == B.CTS_ERR_INVALID_ARG
    assert call(init=(0, 8)) == B.CTS_ERR_INVALID_ARG                      # index out of range
    assert call(init=(-1, 0)) == B.CTS_ERR_INVALID_ARG
    assert call(jd_iters=0) == B.CTS_ERR_INVALID_ARG
    assert call(max_rounds=0) == B.CTS_ERR_INVALID_ARG
    for name in ("A", "B", "U0", "Vt0", "Uc0", "Vtc0", "cof", "U", "Vt", "S", "W"):
        assert call(**{name: None}) == B.CTS_ERR_INVALID_ARG, name
    assert call(ws=need - 1) == B.CTS_ERR_WORKSPACE


def test_jd_diag_argument_errors():
    p = _jp()
    L = cts.lib()
    need = L.cts_jd_workspace_size(ctypes.byref(p))
    args = [FAKE, FAKE, FAKE, FAKE, 3, 0, FAKE, FAKE, FAKE, FAKE, need, None]
    for i in (0, 1, 2, 3, 6, 7, 8, 9):
        a = list(args)
        a[i] = None
        assert L.cts_jd_diag(ctypes.byref(p), *a) == B.CTS_ERR_INVALID_ARG, i
        a[i] = ctypes.c_void_p(0x10004)
        assert L.cts_jd_diag(ctypes.byref(p), *a) == B.CTS_ERR_INVALID_ARG, i
    a = list(args)
    a[4] = -1
    assert L.cts_jd_diag(ctypes.byref(p), *a) == B.CTS_ERR_INVALID_ARG
    a = list(args)
    a[10] = need - 1
    assert L.cts_jd_diag(ctypes.byref(p), *a) == B.CTS_ERR_WORKSPACE


# ------------------------------------------------------------ multi-module ABI
def _mcall(p, M=2, d_out=(64, 32), W=None, U=None, S=None, Y=None, Vt=FAKE, ws_bytes=1 << 30, ws=FAKE):
    vp = ctypes.c_void_p
    dims = (ctypes.c_int32 * len(d_out))(*d_out)
    def arr(v):
        return (vp * max(M, 1))(*([FAKE] * max(M, 1) if v is None else v))
    return cts.lib().cts_apply_multi(ctypes.byref(p), M, dims, FAKE, FAKE, FAKE, arr(W), arr(U), Vt, arr(S),
                                     arr(Y), ws, ws_bytes, None)


def test_multi_validation():
    p = B.make_problem(32, 64, 8, r=16, n_adapters=4, n_clusters=2)
    L = cts.lib()
    d2 = (ctypes.c_int32 * 2)(64, 32)
    need = L.cts_workspace_size_multi(ctypes.byref(p), 2, d2)
    assert need > 0
    assert L.cts_workspace_size_multi(ctypes.byref(p), 0, d2) == 0
    assert _mcall(p, M=0, d_out=(64,)) == B.CTS_ERR_INVALID_ARG
    nine = tuple([64] * 9)
    assert _mcall(p, M=9, d_out=nine) == B.CTS_ERR_UNSUPPORTED
    assert _mcall(p, d_out=(64, 30)) == B.CTS_ERR_UNSUPPORTED               # d_out % 8
    for name in ("W", "U", "S", "Y"):
        kw = {name: [FAKE, None]}
        assert _mcall(p, ws_bytes=need, **kw) == B.CTS_ERR_INVALID_ARG, name
        kw = {name: [FAKE, ctypes.c_void_p(0x10008)]}
        assert _mcall(p, ws_bytes=need, **kw) == B.CTS_ERR_INVALID_ARG, name
    assert _mcall(p, Vt=None, ws_bytes=need) == B.CTS_ERR_INVALID_ARG
    assert _mcall(p, ws_bytes=need - 1) == B.CTS_ERR_WORKSPACE
    # the two outputs on the same memory
    assert _mcall(p, ws_bytes=need, Y=[ctypes.c_void_p(0x40000000), ctypes.c_void_p(0x40000000)],
                  ws=ctypes.c_void_p(0x80000000)) == B.CTS_ERR_INVALID_ARG
    p0 = B.make_problem(0, 64, 8, r=16, n_adapters=4, n_clusters=2)
    assert cts.lib().cts_apply_multi(ctypes.byref(p0), 2, d2, None, None, None, None, None, None, None, None, None,
                                     0, None) == B.CTS_OK


def _apply_na(p, ptrs=None, y=None):
    ptrs = ptrs or [FAKE] * 7
    y = y if y is not None else ctypes.c_void_p(0x7000_0000_0000)
    return cts.lib().cts_apply_noalloc(ctypes.byref(p), *ptrs[:7], y, None)


def test_noalloc_validation_before_any_launch():
    """cts_apply_noalloc: the argument checks of cts_apply, and a problem
    whose workspace exceeds the static scratch array is refused."""
    assert cts.lib().cts_apply_noalloc(ctypes.byref(_p(T=0)), *[None] * 8, None) == B.CTS_OK
    assert cts.lib().cts_apply_noalloc(None, *[FAKE] * 8, None) == B.CTS_ERR_INVALID_ARG
    for i in range(7):
        ptrs = [FAKE] * 7
        ptrs[i] = None
        assert _apply_na(_p(), ptrs) == B.CTS_ERR_INVALID_ARG, i
    assert _apply_na(_p(), y=ctypes.c_void_p(0x7000_0000_0000 + 8)) == B.CTS_ERR_INVALID_ARG
    assert _apply_na(_p(r=12)) == B.CTS_ERR_UNSUPPORTED
    base = 0x5000_0000_0000
    ptrs = [ctypes.c_void_p(base + i * (1 << 30)) for i in range(7)]
    assert _apply_na(_p(T=64, d_in=64, d_out=64, r=8, n_adapters=4), ptrs,
                     y=ctypes.c_void_p(base + 3 * (1 << 30) + 64)) == B.CTS_ERR_INVALID_ARG
    assert cts.workspace_size(_p()) <= B.NOALLOC_SCRATCH_BYTES


def test_noalloc_scratch_size_matches_header():
    src = open(os.path.join(ROOT, "include", "cts.h")).read()
    m = re.search(r"#define CTS_NOALLOC_SCRATCH_BYTES \((\d+)u << (\d+)\)", src)
    assert m and int(m.group(1)) << int(m.group(2)) == B.NOALLOC_SCRATCH_BYTES


def test_sort_bucketing_workspace_validation():
    """cts_sort_by_cluster's workspace (the bucketing for cts_apply_multi_sorted):
    its size, refused when too small, misaligned or overlapping an array."""
    L = cts.lib()
    assert cts.bucketing_size(512, 1000, 50) > 3 * 4 * 512
    assert cts.bucketing_size(0, 4, 2) > 0
    assert cts.bucketing_size(-1, 4, 2) == 0 and cts.bucketing_size(8193, 4, 2) == 0
    assert cts.bucketing_size(8, 0, 2) == 0 and cts.bucketing_size(8, 4, 65537) == 0
    need = cts.bucketing_size(64, 4, 2)
    a, c, pm, of = (ctypes.c_void_p(0x1000_0000 * (i + 1)) for i in range(4))
    ws = ctypes.c_void_p(0x8000_0000)
    f = lambda w, nb: L.cts_sort_by_cluster(a, c, 64, 4, 2, pm, of, w, nb, None)
    assert f(ws, need - 1) == B.CTS_ERR_WORKSPACE
    assert f(ctypes.c_void_p(0x8000_0008), need) == B.CTS_ERR_INVALID_ARG          # misaligned
    assert f(ctypes.c_void_p(0x3000_0000 + 64), need) == B.CTS_ERR_INVALID_ARG     # overlaps perm
    assert f(ctypes.c_void_p(0x1000_0000), need) == B.CTS_ERR_INVALID_ARG          # overlaps adapter_id


def _multi_sorted(p, perm, bk, bk_bytes, y=None, ws=None, M=1, d_out=None):
    d_out = d_out or [p.d_out] * M
    dims = (ctypes.c_int32 * M)(*d_out)
    vp = ctypes.c_void_p
    W = (vp * M)(*[vp(0x5000_0000_0000 + (m << 32)) for m in range(M)])
    U = (vp * M)(*[vp(0x5100_0000_0000 + (m << 32)) for m in range(M)])
    S = (vp * M)(*[vp(0x5200_0000_0000 + (m << 32)) for m in range(M)])
    Y = (vp * M)(*[vp((y or 0x7000_0000_0000) + (m << 32)) for m in range(M)])
    return cts.lib().cts_apply_multi_sorted(ctypes.byref(p), M, dims, perm, bk, bk_bytes,
                                            vp(0x5300_0000_0000), W, U, vp(0x5400_0000_0000), S, Y,
                                            vp(ws or 0x6000_0000_0000), 1 << 40, None)


def test_multi_sorted_validation():
    p = _p(T=512, d_in=4096, d_out=4096, r=64, n_adapters=1000, n_clusters=50)
    perm, bk = ctypes.c_void_p(0x4000_0000_0000), ctypes.c_void_p(0x4100_0000_0000)
    need = cts.bucketing_size(512, 1000, 50)
    assert _multi_sorted(p, perm, bk, need - 1) == B.CTS_ERR_WORKSPACE
    assert _multi_sorted(p, None, bk, need) == B.CTS_ERR_INVALID_ARG
    assert _multi_sorted(p, perm, None, need) == B.CTS_ERR_INVALID_ARG
    assert _multi_sorted(p, perm, ctypes.c_void_p(0x4100_0000_0008), need) == B.CTS_ERR_INVALID_ARG
    # an output over the bucketing
    assert _multi_sorted(p, perm, bk, need, y=0x4100_0000_0000) == B.CTS_ERR_INVALID_ARG
    assert _multi_sorted(_p(T=512, r=12), perm, bk, need) == B.CTS_ERR_UNSUPPORTED
    # a bucketing covers at most 8192 tokens (the sort's limit)
    assert _multi_sorted(_p(T=8193), perm, bk, 1 << 30) == B.CTS_ERR_UNSUPPORTED
    assert _multi_sorted(_p(T=0), None, None, 0) == B.CTS_OK


def _packed(p, d_out=(64, 32), ids=True, srt=False, y=0x7000_0000_0000, ldy=96, ws_bytes=1 << 30,
            ws=0x6000_0000_0000, bk_bytes=1 << 20):
    vp = ctypes.c_void_p
    M = len(d_out)
    dims = (ctypes.c_int32 * M)(*d_out)
    arr = lambda base: (vp * M)(*[vp(base + (m << 32)) for m in range(M)])
    a, c = (vp(0x5500_0000_0000), vp(0x5600_0000_0000)) if ids else (None, None)
    pm, bk = (vp(0x5700_0000_0000), vp(0x5800_0000_0000)) if srt else (None, None)
    return cts.lib().cts_apply_multi_packed(ctypes.byref(p), M, dims, a, c, pm, bk, bk_bytes if srt else 0,
                                            vp(0x5300_0000_0000), arr(0x5000_0000_0000), arr(0x5100_0000_0000),
                                            vp(0x5400_0000_0000), arr(0x5200_0000_0000), vp(y) if y else None,
                                            ldy, vp(ws) if ws else None, ws_bytes, None)


def test_multi_packed_validation():
    """cts_apply_multi_packed: exactly one of the ids and a bucketing, a row
    stride that holds every module's columns, one packed range checked
    against the inputs and the workspace."""
    p = B.make_problem(32, 64, 8, r=16, n_adapters=4, n_clusters=2)
    need = cts.workspace_size_multi(p, [64, 32])
    assert _packed(p, ids=False, srt=False) == B.CTS_ERR_INVALID_ARG             # neither
    assert _packed(p, ids=True, srt=True) == B.CTS_ERR_INVALID_ARG               # both
    assert _packed(p, y=0) == B.CTS_ERR_INVALID_ARG
    assert _packed(p, ldy=88) == B.CTS_ERR_INVALID_ARG                           # < 64 + 32
    assert _packed(p, ldy=100) == B.CTS_ERR_INVALID_ARG                          # not a multiple of 8
    assert _packed(p, y=0x7000_0000_0008) == B.CTS_ERR_INVALID_ARG               # misaligned
    assert _packed(p, ws_bytes=need - 1) == B.CTS_ERR_WORKSPACE
    assert _packed(p, ids=False, srt=True, ws_bytes=need - 1) == B.CTS_ERR_WORKSPACE
    assert _packed(p, ids=False, srt=True, bk_bytes=8) == B.CTS_ERR_WORKSPACE    # bucketing too small
    # the packed range reaches x (rows 1024 apart: row 31 ends past 0x5300...)
    assert _packed(p, y=0x5300_0000_0000 - 31 * 1024 * 2, ldy=1024, ws_bytes=need) == B.CTS_ERR_INVALID_ARG
    assert _packed(p, y=0x6000_0000_0000, ws=0x6000_0000_0000, ws_bytes=need) == B.CTS_ERR_INVALID_ARG
    p0 = B.make_problem(0, 64, 8, r=16, n_adapters=4, n_clusters=2)
    assert _packed(p0, ids=False, y=0, ws=0, ws_bytes=0) == B.CTS_OK
    assert cts.lib().cts_apply_multi_packed(None, 2, None, *[None] * 4, 0, *[None] * 6, 0, None, 0, None) \
        == B.CTS_ERR_INVALID_ARG
