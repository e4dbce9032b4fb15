"""GPU parity of decode-sized batches (T <= 64 bf16 tokens: the bucketing
runs inside the shrink kernel, the fused GEMM takes the 64 x 64 decode tiles
split along d_in) through the C ABI against the oracle: every token, the
adapter term alone (W = 0), the three core products (full Sigma, diagonal,
none = uncompressed), ranks that are not multiples of 16, fp32 output, a
workspace that starts with garbage, and one workspace shared by eager calls
and graph replays."""
import numpy as np
import pytest
import torch

import paper_2407_00066_amd as cts
from paper_2407_00066_amd import workloads as wl

from _gpu_helpers import TOL, dev, host, row_rel_err, say

pytestmark = pytest.mark.gpu

CASES = {
    # name: synthetic kwargs
    "T1_r16": dict(cfg=150, T=1, d_in=256, d_out=192, r=16, n=5, K=2),
    "T5_r8": dict(cfg=151, T=5, d_in=136, d_out=64, r=8, n=3, K=3),
    "T16_one_cluster": dict(cfg=152, T=16, d_in=1024, d_out=520, r=64, n=30, K=1),
    "T17_r24": dict(cfg=153, T=17, d_in=520, d_out=264, r=24, n=9, K=4, ids="zipf"),
    "T32_r128": dict(cfg=154, T=32, d_in=264, d_out=392, r=128, n=40, K=3),
    "T33_k_eq_n": dict(cfg=155, T=33, d_in=200, d_out=136, r=40, n=33, K=33),
    "T63_zipf": dict(cfg=156, T=63, d_in=2056, d_out=328, r=64, n=200, K=8, ids="zipf"),
    "T64_many": dict(cfg=157, T=64, d_in=4096, d_out=1024, r=64, n=1000, K=50),
    "T64_same": dict(cfg=158, T=64, d_in=384, d_out=256, r=32, n=1, K=1),
    "T48_r112": dict(cfg=159, T=48, d_in=128, d_out=120, r=112, n=7, K=2, r_l=24),
}


@pytest.fixture(scope="module")
def cases():
    return {k: wl.synthetic(k, **v) for k, v in CASES.items()}


def _args(w, W=None, sigma=None):
    return (dev(w.x), dev(w.adapter_id), dev(w.cluster_of), dev(w.W if W is None else W), dev(w.U), dev(w.Vt),
            dev(w.Sigma if sigma is None else sigma))


@pytest.mark.parametrize("name", sorted(CASES))
def test_decode_full_diag_uncompressed(oracle_mod, cases, name):
    w = cases[name]
    kw = CASES[name]
    assert w.T <= 64 and w.dtype == "bf16"
    say("decode %s T=%d d_in=%d d_out=%d r=%d n=%d K=%d" % (name, w.T, w.d_in, w.d_out, w.r, w.n, w.K))
    y = cts.apply(*_args(w))
    sig = wl.sigma_diagonals(kw["cfg"], w.n, w.r, w.dtype)
    yd = cts.apply_diag(*_args(w, sigma=sig))
    yu = cts.apply_uncompressed(dev(w.x), dev(w.adapter_id), dev(w.W), dev(w.A), dev(w.B))
    W0 = np.zeros_like(w.W)
    y0 = cts.apply(*_args(w, W=W0))
    yu0 = cts.apply_uncompressed(dev(w.x), dev(w.adapter_id), dev(W0), dev(w.A), dev(w.B))
    yf = cts.apply(*_args(w), out_dtype=torch.float32)
    torch.cuda.synchronize()
    checks = {
        "full": (y, oracle_mod.apply(w.x, w.adapter_id, w.cluster_of, w.W, w.U, w.Vt, w.Sigma)),
        "diag": (yd, oracle_mod.apply_diag(w.x, w.adapter_id, w.cluster_of, w.W, w.U, w.Vt, sig)),
        "uncompressed": (yu, oracle_mod.apply_uncompressed(w.x, w.adapter_id, w.W, w.A, w.B)),
        "adapter term": (y0, oracle_mod.apply(w.x, w.adapter_id, w.cluster_of, W0, w.U, w.Vt, w.Sigma)),
        "uncompressed adapter term": (yu0, oracle_mod.apply_uncompressed(w.x, w.adapter_id, W0, w.A, w.B)),
    }
    checks["fp32 out"] = (yf, checks["full"][1])
    assert yf.dtype == torch.float32
    for what, (got, ref) in checks.items():
        err = row_rel_err(host(got), ref)
        assert err <= TOL["bf16"], (what, err)


def test_decode_garbage_workspace(cases):
    """A workspace may hold anything before a call: all-ones, all-zero and
    patterned workspaces give the same bits as a fresh call, twice in a row."""
    w = cases["T63_zipf"]
    args = _args(w)
    p = cts.make_problem(w.T, w.d_in, w.d_out, r=w.r, n_adapters=w.n, n_clusters=w.K)
    n = cts.workspace_size(p)
    say("decode: garbage workspace")
    ref = cts.apply(*args)
    outs = []
    for fill in (0xFF, 0x00, 0x5A):
        ws = torch.full((n,), fill, dtype=torch.uint8, device="cuda")
        outs += [cts.apply(*args, workspace=ws), cts.apply(*args, workspace=ws)]
    torch.cuda.synchronize()
    for y in outs:
        assert torch.equal(y, ref)


def test_decode_eager_and_graph_share_a_workspace(cases):
    """One workspace: eager calls and replays of a graph captured on it,
    interleaved; every result bit for bit the first eager one."""
    w = cases["T64_many"]
    args = _args(w)
    p = cts.make_problem(w.T, w.d_in, w.d_out, r=w.r, n_adapters=w.n, n_clusters=w.K)
    ws = torch.empty(cts.workspace_size(p), dtype=torch.uint8, device="cuda")
    y = torch.empty((w.T, w.d_out), dtype=torch.bfloat16, device="cuda")
    say("decode: eager reference")
    cts.apply(*args, out=y, workspace=ws)
    torch.cuda.synchronize()
    ref = y.clone()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        cts.apply(*args, out=y, workspace=ws)
    torch.cuda.synchronize()
    for rep in range(4):
        y.fill_(float("nan"))
        say("decode: replay %d" % rep)
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, ref), rep
        y.fill_(float("nan"))
        cts.apply(*args, out=y, workspace=ws)
        torch.cuda.synchronize()
        assert torch.equal(y, ref), rep
    # two replays back to back, no eager call between
    y.fill_(float("nan"))
    g.replay()
    g.replay()
    torch.cuda.synchronize()
    assert torch.equal(y, ref)


def test_decode_full_size_every_token(oracle_mod):
    """decode_q at full size (T = 64, 4096 x 4096, 100 LoRAs, r = 64): every
    token against the oracle, with and without the base term."""
    w = wl.make("decode_q")
    say("decode_q full size, all tokens")
    y = cts.apply(*_args(w))
    W0 = np.zeros_like(w.W)
    y0 = cts.apply(*_args(w, W=W0))
    torch.cuda.synchronize()
    ref = oracle_mod.apply(w.x, w.adapter_id, w.cluster_of, w.W, w.U, w.Vt, w.Sigma)
    assert row_rel_err(host(y), ref) <= TOL["bf16"]
    ref0 = oracle_mod.apply(w.x, w.adapter_id, w.cluster_of, W0, w.U, w.Vt, w.Sigma)
    assert row_rel_err(host(y0), ref0) <= TOL["bf16"]
