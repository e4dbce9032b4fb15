"""GPU parity: the HIP library (through the C ABI) against the fp64 oracle.

Bucketing is compared bit for bit.  Outputs are compared per token with the
inf-norm relative error  max_o |y - y_ref| / max_o |y_ref|, which must stay
<= 1e-5 for fp32 inputs and <= 2e-2 for bf16 inputs (fp32 accumulation).
Small cases compare every output; the full-size workloads compare a sample
of tokens chosen at tile and cluster-segment boundaries (the oracle forms a
d_out x d_in update per sampled adapter).
"""
import numpy as np
import pytest
import torch

import paper_2407_00066_amd as cts
from paper_2407_00066_amd import workloads as wl

from _gpu_helpers import TOL, dev, host, row_rel_err, say

pytestmark = pytest.mark.gpu


def _sort_case(T, n, K, kind, seed):
    rs = np.random.default_rng(seed)
    aid = rs.integers(0, n, T).astype(np.int32)
    if kind == "same":
        aid[:] = n // 2
    elif kind == "sorted":
        aid = np.sort(aid)
    elif kind == "reverse":
        aid = np.sort(aid)[::-1].copy()
    elif kind == "zipf":
        aid = wl.zipf_ids(rs, n, T)
    elif kind.startswith("runs"):
        # kind "runsR": R maximal runs of equal ids (neighbouring runs differ;
        # an id may come back in a later run), run lengths random >= 1
        R = int(kind[4:])
        cuts = np.sort(rs.choice(np.arange(1, T), R - 1, replace=False))
        lens = np.diff(np.concatenate([[0], cuts, [T]]))
        ids = [int(rs.integers(0, n))]
        for _ in range(R - 1):
            nxt = int(rs.integers(0, n - 1))
            ids.append(nxt + (nxt >= ids[-1]))
        aid = np.repeat(np.array(ids, dtype=np.int32), lens)
    cof = None if kind == "identity" else rs.integers(0, K, n).astype(np.int32)
    if kind == "empty":
        cof = (np.arange(n) % 3 * (K // 3)).astype(np.int32)
    return aid, cof


SORT_CASES = [
    (0, 5, 2, "uniform"), (1, 5, 2, "uniform"), (63, 8, 3, "uniform"), (64, 8, 3, "uniform"),
    (65, 100, 1, "uniform"), (1, 1, 1, "uniform"), (500, 1, 1, "uniform"),
    (4096, 1000, 25, "uniform"), (4096, 1000, 25, "zipf"), (8192, 65536, 4096, "uniform"),
    (8192, 3, 2, "uniform"), (1000, 1000, 1000, "identity"), (777, 50, 10, "same"),
    (777, 50, 10, "sorted"), (777, 50, 10, "reverse"), (600, 40, 30, "empty"),
    (2049, 65536, 65536, "uniform"), (256, 1000, 50, "zipf"),
    # request runs: at most 256 runs are ranked as whole runs, more take the
    # token-level passes
    (4096, 1000, 25, "runs32"), (8192, 20, 4, "runs256"), (8192, 20, 4, "runs257"),
    (300, 1000, 50, "runs256"), (8192, 20, 4, "runs1024"),
    (3000, 2, 2, "runs1000"), (1024, 5000, 300, "runs1024"), (8192, 65536, 4096, "runs700"),
]


@pytest.mark.parametrize("T,n,K,kind", SORT_CASES)
def test_sort_bit_exact(oracle_mod, T, n, K, kind):
    aid, cof = _sort_case(T, n, K, kind, seed=T + 31 * n + K)
    if kind == "identity":
        K = n
    say("sort T=%d n=%d K=%d %s" % (T, n, K, kind))
    perm, offs = cts.sort_by_cluster(dev(aid), dev(cof) if cof is not None else None, n, K)
    torch.cuda.synchronize()
    rp, ro = oracle_mod.sort_by_cluster(aid, cof, n, K)
    np.testing.assert_array_equal(perm.cpu().numpy(), rp)
    np.testing.assert_array_equal(offs.cpu().numpy(), ro)


# --------------------------------------------------------------------------
# the bucketing each layer call actually runs (for T <= 128 bf16 batches it
# happens inside the shrink kernel, for larger ones in the sort kernel),
# read back from the call's workspace and compared bit for bit with the
# oracle's sort and the runs derived from it

BUCKET_CASES = [c for c in SORT_CASES if 0 < c[0] <= 128] + [
    (128, 1000, 50, "zipf"), (100, 65536, 65536, "uniform"), (128, 20, 4, "runs7"),
    (96, 300, 7, "runs30"), (17, 4, 4, "same"), (127, 6, 3, "reverse"), (2, 2, 2, "uniform"),
    (129, 1000, 50, "uniform"), (4096, 1000, 25, "zipf"), (600, 40, 30, "empty"),
]


def _expected_bucketing(aid, cof, perm):
    """seg, aid and core-product items of the sorted order perm: items are
    the sorted positions where a run of one (cluster, adapter) starts or
    crosses a multiple of 16."""
    a = aid[perm]
    seg = cof[a] if cof is not None else a
    T = len(perm)
    items = [j for j in range(T) if j % 16 == 0 or seg[j] != seg[j - 1] or a[j] != a[j - 1]]
    return seg.astype(np.int32), a.astype(np.int32), np.array(items + [T], np.int32)


def _read_i32(ws, off, count):
    return ws[off:off + 4 * count].cpu().numpy().view(np.int32).copy()


@pytest.mark.parametrize("T,n,K,kind", BUCKET_CASES)
def test_layer_bucketing_bit_exact(oracle_mod, T, n, K, kind):
    aid, cof = _sort_case(T, n, K, kind, seed=7 * T + 13 * n + K)
    compressed = kind != "identity"
    d, r = 64, 8
    say("layer bucketing T=%d n=%d K=%d %s (%s)" % (T, n, K, kind, "compressed" if compressed else "uncompressed"))
    z = lambda *shape: torch.zeros(shape, dtype=torch.bfloat16, device="cuda")
    if compressed:
        p = cts.make_problem(T, d, d, r=r, n_adapters=n, n_clusters=K)
        ws = torch.full((cts.workspace_size(p),), 0xAB, dtype=torch.uint8, device="cuda")
        cts.apply(z(T, d), dev(aid), dev(cof), z(d, d), z(K, d, r), z(K, r, d), z(n, r, r), workspace=ws)
    else:
        K = n
        p = cts.make_problem(T, d, d, n_adapters=n, r_lora=r)
        ws = torch.full((cts.workspace_size(p, compressed=False),), 0xAB, dtype=torch.uint8, device="cuda")
        cts.apply_uncompressed(z(T, d), dev(aid), z(d, d), z(n, r, d), z(n, d, r), workspace=ws)
    torch.cuda.synchronize()
    off = cts.workspace_bucketing(p, compressed)
    rp, _ = oracle_mod.sort_by_cluster(aid, cof if compressed else None, n, K)
    seg, a, items = _expected_bucketing(aid, cof if compressed else None, rp)
    np.testing.assert_array_equal(_read_i32(ws, off["perm"], T), rp)
    np.testing.assert_array_equal(_read_i32(ws, off["seg"], T), seg)
    np.testing.assert_array_equal(_read_i32(ws, off["aid"], T), a)
    c = int(_read_i32(ws, off["n_items"], 1)[0])
    assert c == len(items) - 1
    np.testing.assert_array_equal(_read_i32(ws, off["items"], c + 1), items)


# --------------------------------------------------------------------------
# small and medium cases: every output compared

SMALL = {
    # name: (synthetic kwargs)
    "tiny_fp32": dict(wl.CONFIGS["tiny_fp32"]),
    "f32_ragged": dict(cfg=100, T=45, d_in=136, d_out=200, r=24, n=10, K=3, dtype="f32"),
    "bf16_ragged": dict(cfg=101, T=203, d_in=392, d_out=328, r=32, n=37, K=5),
    "bf16_large_tiles": dict(cfg=102, T=1100, d_in=520, d_out=264, r=64, n=50, K=7, ids="prefill",
                             n_seq=9, seq_len=(40, 250)),
    "bf16_r128_zipf": dict(cfg=103, T=77, d_in=256, d_out=512, r=128, n=300, K=3, ids="zipf"),
    "bf16_T1": dict(cfg=104, T=1, d_in=64, d_out=64, r=16, n=3, K=2),
    "bf16_one_adapter": dict(cfg=105, T=130, d_in=128, d_out=136, r=16, n=1, K=1),
    "bf16_k_eq_n": dict(cfg=106, T=150, d_in=128, d_out=192, r=16, n=12, K=12),
    "bf16_r8": dict(cfg=107, T=70, d_in=64, d_out=72, r=8, n=5, K=2),
    # T >= 2048 takes the LDS-ring GEMM: ragged in every dimension, many segments
    "bf16_ring_ragged": dict(cfg=109, T=2300, d_in=328, d_out=280, r=24, n=90, K=11, ids="prefill",
                             n_seq=20, seq_len=(40, 200)),
    "bf16_empty_clusters": dict(cfg=108, T=90, d_in=64, d_out=64, r=16, n=4, K=9),
    # d_in >= 8192 takes the 256x128 ring tiles with an 8-way split along d_in
    "bf16_wide_split": dict(cfg=110, T=300, d_in=8200, d_out=264, r=32, n=40, K=6, ids="zipf"),
    # T <= 64 takes the 64x64 decode tiles (four-stage ring, weight loads issued
    # before the token setup): ragged d_in over two splits, and a whole-tile case
    "bf16_decode_ragged": dict(cfg=111, T=50, d_in=1000, d_out=200, r=32, n=20, K=3),
    "bf16_decode_split4": dict(cfg=112, T=64, d_in=2048, d_out=320, r=16, n=30, K=2),
    # 128x128 ring tiles (at least 128 of them, too few 256x128 tiles): ragged
    # token tail and d_in
    "bf16_mid_tiles": dict(cfg=113, T=200, d_in=200, d_out=8192, r=24, n=30, K=4, ids="zipf"),
    # the largest batch, rank and LoRA rank the ABI takes (T = 8192, r = r_lora = 128), ragged
    "bf16_max_T": dict(cfg=114, T=8192, d_in=264, d_out=200, r=128, n=2000, K=40, r_l=128, ids="prefill",
                       n_seq=48, seq_len=(60, 300)),
    # the largest id spaces (n = K = 65536), every token its own adapter and cluster
    "bf16_max_ids": dict(cfg=115, T=600, d_in=64, d_out=64, r=8, n=65536, K=65536, r_l=8),
}


def _inputs(w):
    return (dev(w.x), dev(w.adapter_id), dev(w.cluster_of), dev(w.W), dev(w.U), dev(w.Vt),
            dev(w.Sigma))


@pytest.fixture(scope="module")
def small_cases():
    return {k: wl.synthetic(k, **v) for k, v in SMALL.items()}


@pytest.mark.parametrize("name", list(SMALL))
def test_apply_small(oracle_mod, small_cases, name):
    w = small_cases[name]
    say("apply %s T=%d d_in=%d d_out=%d r=%d n=%d K=%d" % (name, w.T, w.d_in, w.d_out, w.r, w.n, w.K))
    y = cts.apply(*_inputs(w))
    torch.cuda.synchronize()
    ref = oracle_mod.apply(w.x, w.adapter_id, w.cluster_of, w.W, w.U, w.Vt, w.Sigma)
    err = row_rel_err(host(y), ref)
    assert err <= TOL[w.dtype], err


@pytest.mark.parametrize("name", ["tiny_fp32", "f32_ragged", "bf16_ragged", "bf16_large_tiles",
                                  "bf16_T1", "bf16_one_adapter", "bf16_ring_ragged", "bf16_max_T",
                                  "bf16_max_ids"])
def test_uncompressed_small(oracle_mod, small_cases, name):
    w = small_cases[name]
    say("apply_uncompressed %s T=%d r_l=%d n=%d" % (name, w.T, w.r_l, w.n))
    y = cts.apply_uncompressed(dev(w.x), dev(w.adapter_id), dev(w.W), dev(w.A), dev(w.B))
    torch.cuda.synchronize()
    ref = oracle_mod.apply_uncompressed(w.x, w.adapter_id, w.W, w.A, w.B)
    err = row_rel_err(host(y), ref)
    assert err <= TOL[w.dtype], err


# --------------------------------------------------------------------------
# the adapter term alone: W = 0, so y = U_k Sigma_i V_k^T x (resp. B_i A_i x)
# and the error is measured against that term's own row maximum (with W the
# adapter term is about 1/8 of the output, so an error in it would be hidden
# by the base term's scale).  Every bf16 tile shape: Narrow, Mid, Wide with a
# split along d_in, Large, Decode (split in four), the bucketing inside the
# shrink (T <= 128) and the separate sort.

ADAPTER_TERM_CASES = ["bf16_ragged", "bf16_large_tiles", "bf16_r128_zipf", "bf16_ring_ragged",
                      "bf16_wide_split", "bf16_decode_ragged", "bf16_decode_split4", "bf16_mid_tiles",
                      "bf16_k_eq_n", "bf16_T1"]


def _zero_base(w):
    return np.zeros_like(w.W)


@pytest.mark.parametrize("name", ADAPTER_TERM_CASES)
def test_adapter_term_alone(oracle_mod, small_cases, name):
    w = small_cases[name]
    W0 = _zero_base(w)
    say("adapter term alone %s T=%d" % (name, w.T))
    y = cts.apply(dev(w.x), dev(w.adapter_id), dev(w.cluster_of), dev(W0), dev(w.U), dev(w.Vt), dev(w.Sigma))
    yu = cts.apply_uncompressed(dev(w.x), dev(w.adapter_id), dev(W0), dev(w.A), dev(w.B))
    torch.cuda.synchronize()
    ref = oracle_mod.apply(w.x, w.adapter_id, w.cluster_of, W0, w.U, w.Vt, w.Sigma)
    refu = oracle_mod.apply_uncompressed(w.x, w.adapter_id, W0, w.A, w.B)
    assert np.abs(ref).max() > 0
    err, erru = row_rel_err(host(y), ref), row_rel_err(host(yu), refu)
    assert err <= TOL["bf16"], err
    assert erru <= TOL["bf16"], erru


@pytest.mark.parametrize("name", ["bf16_ragged", "bf16_decode_split4", "bf16_ring_ragged", "bf16_wide_split"])
def test_adapter_term_alone_variants(oracle_mod, small_cases, name):
    """W = 0 through the diagonal-Sigma, mixed-rank and multi-module entry
    points."""
    w = small_cases[name]
    kw = SMALL[name]
    W0 = _zero_base(w)
    x, aid, cof = dev(w.x), dev(w.adapter_id), dev(w.cluster_of)
    say("adapter term alone (diag, ranked, multi) %s" % name)
    sig = wl.sigma_diagonals(kw["cfg"], w.n, w.r, w.dtype)
    yd = cts.apply_diag(x, aid, cof, dev(W0), dev(w.U), dev(w.Vt), dev(sig))
    rk = wl.mixed_ranks(kw["cfg"], w.K, w.r, lo=8)
    yr = cts.apply_ranked(x, aid, cof, dev(W0), dev(w.U), dev(w.Vt), dev(w.Sigma), dev(rk))
    ra = wl.mixed_ranks(kw["cfg"] + 500, w.n, w.r_l, lo=8)
    yur = cts.apply_uncompressed_ranked(x, aid, dev(W0), dev(w.A), dev(w.B), dev(ra))
    # two modules: the layer's own arrays and a second set with W = 0 too
    w2 = wl.synthetic(name + "_m2", **dict(kw, cfg=kw["cfg"] + 900, with_lora=False))
    Vt2 = np.concatenate([w.Vt, w2.Vt], axis=1)
    ym = cts.apply_multi(x, aid, cof, [dev(W0), dev(np.zeros_like(w2.W))], [dev(w.U), dev(w2.U)], dev(Vt2),
                         [dev(w.Sigma), dev(w2.Sigma)])
    torch.cuda.synchronize()
    checks = [
        (yd, oracle_mod.apply_diag(w.x, w.adapter_id, w.cluster_of, W0, w.U, w.Vt, sig)),
        (yr, oracle_mod.apply_ranked(w.x, w.adapter_id, w.cluster_of, W0, w.U, w.Vt, w.Sigma, rk)),
        (yur, oracle_mod.apply_uncompressed_ranked(w.x, w.adapter_id, W0, w.A, w.B, ra)),
    ] + list(zip(ym, oracle_mod.apply_multi(w.x, w.adapter_id, w.cluster_of, [W0, np.zeros_like(w2.W)],
                                            [w.U, w2.U], Vt2, [w.Sigma, w2.Sigma])))
    for i, (y, ref) in enumerate(checks):
        assert np.abs(ref).max() > 0, i
        err = row_rel_err(host(y), ref)
        assert err <= TOL["bf16"], (i, err)


def test_tiny_exact_compressed_equals_uncompressed(oracle_mod):
    """Prop. 1 on the GPU: the tiny collection compressed losslessly at r = 32
    gives the uncompressed layer (both GPU paths and the oracle agree)."""
    w = wl.make("tiny_fp32")
    U, Vt, S = oracle_mod.exact_compress(w.A, w.B)
    U32, V32, S32 = (a.astype(np.float32) for a in (U[None], Vt[None], S))
    say("tiny-exact r=32")
    cof = np.zeros(w.n, np.int32)
    y_c = cts.apply(dev(w.x), dev(w.adapter_id), dev(cof), dev(w.W), dev(U32), dev(V32), dev(S32))
    y_u = cts.apply_uncompressed(dev(w.x), dev(w.adapter_id), dev(w.W), dev(w.A), dev(w.B))
    torch.cuda.synchronize()
    ref = oracle_mod.apply_uncompressed(w.x, w.adapter_id, w.W, w.A, w.B)
    assert row_rel_err(host(y_c), ref) <= 1e-5
    assert row_rel_err(host(y_u), ref) <= 1e-5
    assert row_rel_err(host(y_c), host(y_u)) <= 1e-5


def test_split_sum_repeatable(oracle_mod, small_cases):
    """The decode tiles split d_in four ways (fp32 partials summed in split
    order): repeated calls on one workspace give identical bits and match
    the oracle."""
    w = small_cases["bf16_decode_split4"]
    say("split-sum repeat")
    p = cts.make_problem(w.T, w.d_in, w.d_out, r=w.r, n_adapters=w.n, n_clusters=w.K)
    ws = torch.empty(cts.workspace_size(p), dtype=torch.uint8, device="cuda")
    ys = [cts.apply(*_inputs(w), workspace=ws) for _ in range(3)]
    torch.cuda.synchronize()
    for y in ys[1:]:
        assert torch.equal(y, ys[0])
    ref = oracle_mod.apply(w.x, w.adapter_id, w.cluster_of, w.W, w.U, w.Vt, w.Sigma)
    assert row_rel_err(host(ys[0]), ref) <= TOL[w.dtype]


def test_zero_sigma_is_exactly_base_layer(small_cases):
    """Sigma_i = 0 adds exactly nothing: bitwise equal to B_i = 0 on the
    uncompressed path (same base GEMM, zero adapter term)."""
    w = small_cases["bf16_ragged"]
    say("zero-sigma bitwise")
    S0 = np.zeros_like(w.Sigma)
    y_c = cts.apply(dev(w.x), dev(w.adapter_id), dev(w.cluster_of), dev(w.W), dev(w.U), dev(w.Vt), dev(S0))
    y_u = cts.apply_uncompressed(dev(w.x), dev(w.adapter_id), dev(w.W), dev(w.A), dev(np.zeros_like(w.B)))
    torch.cuda.synchronize()
    assert torch.equal(y_c, y_u)


def test_fp32_output_from_bf16(oracle_mod, small_cases):
    w = small_cases["bf16_ragged"]
    say("bf16 in / f32 out")
    y = cts.apply(*_inputs(w), out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert y.dtype == torch.float32
    ref = oracle_mod.apply(w.x, w.adapter_id, w.cluster_of, w.W, w.U, w.Vt, w.Sigma)
    assert row_rel_err(host(y), ref) <= TOL["bf16"]


def test_deterministic(small_cases):
    w = small_cases["bf16_large_tiles"]
    say("determinism")
    args = _inputs(w)
    y1 = cts.apply(*args)
    y2 = cts.apply(*args)
    u1 = cts.apply_uncompressed(dev(w.x), dev(w.adapter_id), dev(w.W), dev(w.A), dev(w.B))
    u2 = cts.apply_uncompressed(dev(w.x), dev(w.adapter_id), dev(w.W), dev(w.A), dev(w.B))
    torch.cuda.synchronize()
    assert torch.equal(y1, y2) and torch.equal(u1, u2)


def test_token_permutation_equivariance(small_cases):
    w = small_cases["bf16_ragged"]
    say("permutation equivariance")
    p = np.random.default_rng(5).permutation(w.T)
    y = cts.apply(*_inputs(w))
    yp = cts.apply(dev(w.x[p]), dev(w.adapter_id[p]), dev(w.cluster_of), dev(w.W), dev(w.U),
                   dev(w.Vt), dev(w.Sigma))
    torch.cuda.synchronize()
    assert row_rel_err(host(yp), host(y)[p]) <= 1e-6


def test_validate_ids():
    say("validate_ids")
    aid = torch.tensor([0, 3, 2], dtype=torch.int32, device="cuda")
    cof = torch.tensor([0, 1, 1, 0], dtype=torch.int32, device="cuda")
    assert cts.validate_ids(aid, cof, 4, 2)
    assert not cts.validate_ids(aid, cof[:3], 3, 2)      # adapter id 3 >= n
    assert not cts.validate_ids(aid, torch.tensor([0, 1, 2, 0], dtype=torch.int32, device="cuda"), 4, 2)


def test_out_of_range_ids_do_not_fault(small_cases):
    """Ids outside [0, n) are clamped inside the kernels; the call completes."""
    w = small_cases["bf16_r8"]
    say("out-of-range ids (clamped)")
    aid = w.adapter_id.copy()
    aid[0], aid[1] = -7, 1 << 20
    y = cts.apply(dev(w.x), dev(aid), dev(w.cluster_of), dev(w.W), dev(w.U), dev(w.Vt), dev(w.Sigma))
    torch.cuda.synchronize()
    assert torch.isfinite(y.float()).all()


def test_shrink_split_follows_tile_count(oracle_mod):
    """The shrink splits d_in by the tile count found on the device, and the
    core-product stage sums exactly that many pieces: a call with many tiles
    (one split piece) after a call with few (eight pieces) on the same
    workspace must not pick up the earlier call's stale partials."""
    T, d_in, d_out, n, r_l = 600, 4096, 64, 600, 16
    w = wl.synthetic("split_reuse", cfg=116, T=T, d_in=d_in, d_out=d_out, r=16, n=n, K=1, r_l=r_l)
    x, W, A, B = dev(w.x), dev(w.W), dev(w.A), dev(w.B)
    p = cts.make_problem(T, d_in, d_out, 16, n, 1, r_l, cts.CTS_BF16, cts.CTS_BF16)
    ws = torch.zeros(cts.workspace_size(p, compressed=False), dtype=torch.uint8, device="cuda")
    few = np.zeros(T, np.int32)                       # one adapter: 10 tiles
    many = np.arange(T, dtype=np.int32)               # 600 adapters: 600 tiles
    say("shrink split reuse T=%d d_in=%d n=%d" % (T, d_in, n))
    y_few = cts.apply_uncompressed(x, dev(few), W, A, B, workspace=ws)
    y_many = cts.apply_uncompressed(x, dev(many), W, A, B, workspace=ws)
    torch.cuda.synchronize()
    for ids, y in ((few, y_few), (many, y_many)):
        ref = oracle_mod.apply_uncompressed(w.x, ids, w.W, w.A, w.B)
        assert row_rel_err(host(y), ref) <= TOL["bf16"]
    ws.zero_()
    y_fresh = cts.apply_uncompressed(x, dev(many), W, A, B, workspace=ws)
    torch.cuda.synchronize()
    assert torch.equal(y_fresh, y_many)


# --------------------------------------------------------------------------
# full-size workloads: sampled tokens

def _sample_tokens(w, oracle_mod, extra=6, max_bounds=8):
    """Tokens at the positions a tiling can get wrong, in the cluster-sorted
    order: the first and last position, both sides of every multiple of 64
    (one token per 64-column tile at least), and both sides of the first
    max_bounds cluster boundaries; then `extra` random positions.  Every
    position of the first two kinds is kept (the oracle's cost is one
    d_out x d_in update per distinct adapter among them)."""
    perm, offs = oracle_mod.sort_by_cluster(w.adapter_id, w.cluster_of, w.n, w.K)
    pos = {0, w.T - 1}
    for b in range(64, w.T, 64):
        pos.update({b - 1, b})
    bounds = [int(o) for o in offs[1:-1] if 0 < o < w.T]
    for o in sorted(set(bounds))[:max_bounds]:
        pos.update({o - 1, o})
    rs = np.random.default_rng(w.T)
    pos.update(rs.integers(0, w.T, extra).tolist())
    return np.array(sorted({int(perm[j]) for j in pos}), np.int64)


@pytest.fixture(scope="module")
def full_cases():
    return {}


def _full(full_cases, name):
    if name not in full_cases:
        say("generating %s" % name)
        full_cases[name] = wl.make(name)
    return full_cases[name]


@pytest.mark.parametrize("name", ["decode_q", "prefill_mix", "mlp_up"])
def test_full_config_sampled(oracle_mod, full_cases, name):
    w = _full(full_cases, name)
    toks = _sample_tokens(w, oracle_mod)
    say("apply %s (full size), %d sampled tokens" % (name, len(toks)))
    y = cts.apply(*_inputs(w))
    torch.cuda.synchronize()
    yh = host(y)
    assert np.isfinite(yh).all()
    ref = oracle_mod.apply(w.x, w.adapter_id, w.cluster_of, w.W, w.U, w.Vt, w.Sigma, tokens=toks)
    err = row_rel_err(yh[toks], ref)
    assert err <= TOL["bf16"], err


@pytest.mark.parametrize("name", ["stack_q", "stack_kv", "stack_gate", "stack_down"])
def test_stack_projection_sampled(oracle_mod, full_cases, name):
    """Each distinct projection shape of the 32-layer decoder stack at full size."""
    w = _full(full_cases, name)
    toks = _sample_tokens(w, oracle_mod, max_bounds=4)
    say("apply %s (full size), %d sampled tokens" % (name, len(toks)))
    y = cts.apply(*_inputs(w))
    torch.cuda.synchronize()
    yh = host(y)
    assert np.isfinite(yh).all()
    ref = oracle_mod.apply(w.x, w.adapter_id, w.cluster_of, w.W, w.U, w.Vt, w.Sigma, tokens=toks)
    err = row_rel_err(yh[toks], ref)
    assert err <= TOL["bf16"], err
    full_cases.pop(name)


@pytest.mark.parametrize("name", ["decode_q", "prefill_mix", "mlp_up"])
def test_full_config_uncompressed_sampled(oracle_mod, full_cases, name):
    w = _full(full_cases, name)
    toks = _sample_tokens(w, oracle_mod)
    say("apply_uncompressed %s (full size), %d sampled tokens" % (name, len(toks)))
    y = cts.apply_uncompressed(dev(w.x), dev(w.adapter_id), dev(w.W), dev(w.A), dev(w.B))
    torch.cuda.synchronize()
    ref = oracle_mod.apply_uncompressed(w.x, w.adapter_id, w.W, w.A, w.B, tokens=toks)
    err = row_rel_err(host(y)[toks], ref)
    assert err <= TOL["bf16"], err
