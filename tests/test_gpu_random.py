"""GPU parity on a seeded sweep of problem shapes: the layer (cts_apply) and
the uncompressed path against the fp64 oracle, every output compared.

The shapes are drawn once from a fixed seed to cover the tile and split
choices together with ragged sizes: batches from one token to past 2048
(the bucketing inside the shrink for T <= 128, the separate sort above),
d_in up to past 8192 (the split along d_in), ranks 8..128, one to a few
hundred adapters in one to dozens of clusters, uniform, Zipf and
request-run ids, bf16 and fp32.  Tolerances as in the other parity tests.
"""
import numpy as np
import pytest
import torch

import paper_2407_00066_amd as cts
from paper_2407_00066_amd import workloads as wl

from _gpu_helpers import TOL, dev, host, row_rel_err, say

pytestmark = pytest.mark.gpu

N_CASES = 28


def _draw_cases(seed=20261202, count=N_CASES):
    rs = np.random.default_rng(seed)
    cases = []
    for i in range(count):
        band = i % 4
        if band == 0:
            T = int(rs.integers(1, 129))                     # bucketing inside the shrink
        elif band == 1:
            T = int(rs.integers(129, 700))
        elif band == 2:
            T = int(rs.integers(700, 2048))
        else:
            T = int(rs.integers(2048, 3100))                 # the ring GEMM's large tiles
        big_k = (i % 7 == 3)
        d_in = 8 * int(rs.integers(1030, 1100)) if big_k else 8 * int(rs.integers(1, 66))
        d_out = 8 * int(rs.integers(1, 34 if big_k else 66))
        f32 = (i % 5 == 4)
        r = 8 * int(rs.integers(1, min(16, d_in // 8, d_out // 8) + 1))      # orthonormal bases: r <= d
        n = int(rs.integers(1, 90))
        K = int(rs.integers(1, min(n, 24) + 1))
        r_l = (4 if f32 else 8) * int(rs.integers(1, (32 if f32 else 16) + 1))
        ids = ("uniform", "zipf", "prefill")[int(rs.integers(0, 3))]
        kw = dict(cfg=3000 + i, T=T, d_in=d_in, d_out=d_out, r=r, n=n, K=K, r_l=r_l,
                  dtype="f32" if f32 else "bf16", ids=ids)
        if ids == "prefill":
            kw["n_seq"] = min(T, int(rs.integers(1, 12)))
            kw["seq_len"] = (1, T)
        cases.append(kw)
    return cases


CASES = _draw_cases()


def _name(kw):
    return "T%d_%dx%d_r%d_n%d_K%d_%s_%s" % (kw["T"], kw["d_in"], kw["d_out"], kw["r"], kw["n"], kw["K"],
                                           kw["ids"], kw["dtype"])


@pytest.mark.parametrize("kw", CASES, ids=[_name(c) for c in CASES])
def test_random_shape(oracle_mod, kw):
    w = wl.synthetic(_name(kw), **kw)
    say("random shape %s" % _name(kw))
    x, aid, cof = dev(w.x), dev(w.adapter_id), dev(w.cluster_of)
    y = cts.apply(x, aid, cof, dev(w.W), dev(w.U), dev(w.Vt), dev(w.Sigma))
    yu = cts.apply_uncompressed(x, aid, dev(w.W), dev(w.A), dev(w.B))
    torch.cuda.synchronize()
    ref = oracle_mod.apply(w.x, w.adapter_id, w.cluster_of, w.W, w.U, w.Vt, w.Sigma)
    refu = oracle_mod.apply_uncompressed(w.x, w.adapter_id, w.W, w.A, w.B)
    err, erru = row_rel_err(host(y), ref), row_rel_err(host(yu), refu)
    assert err <= TOL[w.dtype], err
    assert erru <= TOL[w.dtype], erru
