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
