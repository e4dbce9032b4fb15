"""cts_apply_noalloc (no workspace argument: the library's static per-device
scratch array) through the C ABI, against cts_apply on the same inputs and
against the oracle.  Two calls in a row share the scratch array; the second
has a smaller batch, so it runs over what the first left there.

Collected last (the round's end runs pytest -x): it must pass alone in a
fresh process and after every other GPU test.
"""
import numpy as np
import pytest
import torch

import paper_2407_00066_amd as cts
from paper_2407_00066_amd import workloads as wl

from _gpu_helpers import TOL, dev, host, row_rel_err, say

pytestmark = pytest.mark.gpu


def _inputs(w):
    return (dev(w.x), dev(w.adapter_id), dev(w.cluster_of), dev(w.W), dev(w.U), dev(w.Vt),
            dev(w.Sigma))


# (first call, second call with fewer tokens): decode-sized batches (the
# bucketing inside the shrink), a batch with the separate sort, and fp32
CASES = [
    (dict(cfg=130, T=300, d_in=520, d_out=264, r=32, n=40, K=5, ids="zipf"),
     dict(cfg=131, T=57, d_in=520, d_out=264, r=32, n=40, K=5)),
    (dict(cfg=132, T=2300, d_in=328, d_out=280, r=24, n=90, K=11, ids="prefill", n_seq=20,
          seq_len=(40, 200)),
     dict(cfg=133, T=700, d_in=328, d_out=280, r=24, n=90, K=11, ids="zipf")),
    (dict(cfg=134, T=64, d_in=2048, d_out=320, r=16, n=30, K=2),
     dict(cfg=135, T=13, d_in=2048, d_out=320, r=16, n=30, K=2)),
    (dict(cfg=136, T=90, d_in=136, d_out=200, r=24, n=10, K=3, dtype="f32"),
     dict(cfg=137, T=45, d_in=136, d_out=200, r=24, n=10, K=3, dtype="f32")),
]


@pytest.mark.parametrize("first,second", CASES)
def test_noalloc_matches_apply(oracle_mod, first, second):
    outs = []
    for kw in (first, second):
        w = wl.synthetic("noalloc", **kw)
        say("apply_noalloc T=%d d_in=%d d_out=%d r=%d n=%d K=%d %s" % (w.T, w.d_in, w.d_out, w.r, w.n, w.K, w.dtype))
        p = cts.make_problem(w.T, w.d_in, w.d_out, r=w.r, n_adapters=w.n, n_clusters=w.K,
                             dtype=cts.CTS_F32 if w.dtype == "f32" else cts.CTS_BF16)
        assert cts.workspace_size(p) <= cts.NOALLOC_SCRATCH_BYTES
        args = _inputs(w)
        y_na = cts.apply_noalloc(*args)
        outs.append((w, y_na))
    torch.cuda.synchronize()
    for w, y_na in outs:
        y = cts.apply(*_inputs(w))
        torch.cuda.synchronize()
        assert torch.equal(y_na, y), "cts_apply_noalloc differs from cts_apply"
        ref = oracle_mod.apply(w.x, w.adapter_id, w.cluster_of, w.W, w.U, w.Vt, w.Sigma)
        err = row_rel_err(host(y_na), ref)
        assert err <= TOL[w.dtype], err


def test_noalloc_repeated_calls_are_stable(oracle_mod):
    """The same call three times in a row on one stream gives the same bits
    (nothing the scratch array keeps from a call changes the next)."""
    w = wl.synthetic("noalloc_rep", cfg=138, T=100, d_in=256, d_out=192, r=32, n=20, K=3, ids="zipf")
    say("apply_noalloc repeated T=%d" % w.T)
    args = _inputs(w)
    ys = [cts.apply_noalloc(*args) for _ in range(3)]
    torch.cuda.synchronize()
    assert all(torch.equal(y, ys[0]) for y in ys[1:])
    ref = oracle_mod.apply(w.x, w.adapter_id, w.cluster_of, w.W, w.U, w.Vt, w.Sigma)
    assert row_rel_err(host(ys[0]), ref) <= TOL["bf16"]
