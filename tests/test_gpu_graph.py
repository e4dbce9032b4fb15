"""cts_apply launched from a captured HIP graph: every replay must give the
eager result bit for bit (the layer's kernels are deterministic and issue no
allocation, copy or memset, so the whole call can be captured).  Replays are
interleaved with eager work and synchronisations."""
import numpy as np
import pytest
import torch

import paper_2407_00066_amd as cts
from paper_2407_00066_amd import workloads as wl

from _gpu_helpers import dev, say

pytestmark = pytest.mark.gpu


def _layer(name, **kw):
    w = wl.synthetic(name, **kw)
    args = [dev(a) for a in (w.x, w.adapter_id, w.cluster_of, w.W, w.U, w.Vt, w.Sigma)]
    return w, args


def test_graph_replay_matches_eager():
    # two layers of different shapes in one graph (the decode tiles with a
    # 4-way k split summed in the GEMM, and the 256x256 tiles), as a decoder
    # stack would capture them
    w1, a1 = _layer("graph_a", cfg=120, T=64, d_in=2048, d_out=320, r=32, n=40, K=5)
    w2, a2 = _layer("graph_b", cfg=121, T=2100, d_in=256, d_out=296, r=16, n=30, K=4, ids="prefill",
                    n_seq=12, seq_len=(60, 300))
    y1 = torch.empty((w1.T, w1.d_out), dtype=torch.bfloat16, device="cuda")
    y2 = torch.empty((w2.T, w2.d_out), dtype=torch.bfloat16, device="cuda")
    ws = []
    for w in (w1, w2):
        p = cts.make_problem(w.T, w.d_in, w.d_out, r=w.r, n_adapters=w.n, n_clusters=w.K)
        ws.append(torch.empty(cts.workspace_size(p), dtype=torch.uint8, device="cuda"))

    def layer_pair():
        cts.apply(*a1, out=y1, workspace=ws[0])
        cts.apply(*a2, out=y2, workspace=ws[1])

    say("graph: eager reference")
    layer_pair()
    torch.cuda.synchronize()
    e1, e2 = y1.clone(), y2.clone()

    say("graph: capture")
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        layer_pair()
    torch.cuda.synchronize()

    noise = torch.randn(1 << 20, device="cuda")
    for rep in range(4):
        # eager work between replays, including the same layer on other outputs
        y1.fill_(float("nan"))
        y2.fill_(float("nan"))
        noise.mul_(1.5).add_(1.0)
        z = cts.apply(*a1)
        say("graph: replay %d" % rep)
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(y1, e1), rep
        assert torch.equal(y2, e2), rep
        assert torch.equal(z, e1), rep


def test_graph_replay_sort_outputs():
    # the bucketing alone, captured: perm and offsets identical on every replay
    rs = np.random.default_rng(7)
    aid = dev(rs.integers(0, 300, 3000).astype(np.int32))
    cof = dev(rs.integers(0, 20, 300).astype(np.int32))
    perm0, offs0 = cts.sort_by_cluster(aid, cof, 300, 20)
    perm = torch.empty_like(perm0)
    offs = torch.empty_like(offs0)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        cts.sort_by_cluster(aid, cof, 300, 20, perm=perm, offsets=offs)
    for rep in range(3):
        perm.fill_(-1)
        offs.fill_(-1)
        say("graph sort: replay %d" % rep)
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(perm, perm0) and torch.equal(offs, offs0), rep


def test_graph_replay_multi_and_uncompressed():
    # cts_apply_multi (one shrink, one core-product launch for all modules)
    # and cts_apply_uncompressed, both with T > 128 (shrink split chosen on
    # the device), captured together; every replay bit for bit the eager result
    kw = dict(T=300, d_in=256, r=16, n=50, K=5, ids="zipf")
    mods = [wl.synthetic("gm%d" % m, cfg=150 + m, d_out=d, with_lora=False, **kw)
            for m, d in enumerate((256, 64, 64))]
    w0 = mods[0]
    Vt = dev(np.concatenate([m.Vt for m in mods], axis=1))
    x, aid, cof = dev(w0.x), dev(w0.adapter_id), dev(w0.cluster_of)
    Ws, Us, Ss = [dev(m.W) for m in mods], [dev(m.U) for m in mods], [dev(m.Sigma) for m in mods]
    ys = [torch.empty((w0.T, m.d_out), dtype=torch.bfloat16, device="cuda") for m in mods]
    p = cts.make_problem(w0.T, w0.d_in, 256, r=16, n_adapters=50, n_clusters=5)
    wsm = torch.empty(cts.workspace_size_multi(p, [m.d_out for m in mods]), dtype=torch.uint8, device="cuda")
    u = wl.synthetic("gu", cfg=155, T=600, d_in=512, d_out=128, r=16, n=300, K=1, r_l=16)
    ux, uaid, uW, uA, uB = dev(u.x), dev(u.adapter_id), dev(u.W), dev(u.A), dev(u.B)
    yu = torch.empty((u.T, u.d_out), dtype=torch.bfloat16, device="cuda")
    pu = cts.make_problem(u.T, u.d_in, u.d_out, n_adapters=u.n, r_lora=16)
    wsu = torch.empty(cts.workspace_size(pu, compressed=False), dtype=torch.uint8, device="cuda")

    def calls():
        cts.apply_multi(x, aid, cof, Ws, Us, Vt, Ss, outs=ys, workspace=wsm)
        cts.apply_uncompressed(ux, uaid, uW, uA, uB, out=yu, workspace=wsu)

    say("graph multi/uncompressed: eager reference")
    calls()
    torch.cuda.synchronize()
    ref = [y.clone() for y in ys] + [yu.clone()]
    say("graph multi/uncompressed: capture")
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        calls()
    torch.cuda.synchronize()
    for rep in range(3):
        for y in ys + [yu]:
            y.fill_(float("nan"))
        z = cts.apply_uncompressed(ux, uaid, uW, uA, uB)
        say("graph multi/uncompressed: replay %d" % rep)
        g.replay()
        torch.cuda.synchronize()
        for y, e in zip(ys + [yu], ref):
            assert torch.equal(y, e), rep
        assert torch.equal(z, ref[-1]), rep
