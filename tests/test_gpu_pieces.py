"""GPU parity of batches above 8192 tokens, which the library runs as
consecutive pieces of at most 8192 tokens (near-equal sizes, the larger ones
first): every output row against the fp64 oracle through each entry point,
and the whole call bit for bit equal to separate calls on the pieces' token
ranges (y_t depends on token t alone, so the pieces are complete layers)."""
import numpy as np
import pytest
import torch

import paper_2407_00066_amd as cts
from paper_2407_00066_amd import workloads as wl

from _gpu_helpers import TOL, dev, host, row_rel_err, say

pytestmark = pytest.mark.gpu

CASES = {
    # three pieces (5462, 5462, 5461 tokens), prefill-like runs of one adapter
    "bf16_T16385": dict(cfg=170, T=16385, d_in=136, d_out=72, r=16, n=50, K=5, ids="prefill",
                        n_seq=90, seq_len=(60, 300)),
    # two pieces of 4097 and 4096 tokens (the 256x256 tiles), Zipf ids
    "bf16_T8193": dict(cfg=171, T=8193, d_in=64, d_out=264, r=32, n=300, K=12, ids="zipf"),
    # fp32, three pieces of 6667, 6667 and 6666 tokens
    "f32_T20000": dict(cfg=172, T=20000, d_in=64, d_out=64, r=8, n=20, K=3, dtype="f32"),
}


def _pieces(T, cap=8192):
    n = max(1, -(-T // cap))
    q, rem = divmod(T, n)
    return [q + 1] * rem + [q] * (n - rem)


@pytest.fixture(scope="module")
def cases():
    return {k: wl.synthetic(k, **v) for k, v in CASES.items()}


@pytest.mark.parametrize("name", sorted(CASES))
def test_pieces_match_oracle(oracle_mod, cases, name):
    w = cases[name]
    kw = CASES[name]
    say("pieces %s T=%d (%s)" % (name, w.T, _pieces(w.T)))
    x, aid, cof = dev(w.x), dev(w.adapter_id), dev(w.cluster_of)
    y = cts.apply(x, aid, cof, dev(w.W), dev(w.U), dev(w.Vt), dev(w.Sigma))
    sig = wl.sigma_diagonals(kw["cfg"], w.n, w.r, w.dtype)
    yd = cts.apply_diag(x, aid, cof, dev(w.W), dev(w.U), dev(w.Vt), dev(sig))
    rk = wl.mixed_ranks(kw["cfg"], w.K, w.r, lo=8)
    yr = cts.apply_ranked(x, aid, cof, dev(w.W), dev(w.U), dev(w.Vt), dev(w.Sigma), dev(rk))
    yu = cts.apply_uncompressed(x, aid, dev(w.W), dev(w.A), dev(w.B))
    torch.cuda.synchronize()
    checks = {
        "full": (y, oracle_mod.apply(w.x, w.adapter_id, w.cluster_of, w.W, w.U, w.Vt, w.Sigma)),
        "diag": (yd, oracle_mod.apply_diag(w.x, w.adapter_id, w.cluster_of, w.W, w.U, w.Vt, sig)),
        "ranked": (yr, oracle_mod.apply_ranked(w.x, w.adapter_id, w.cluster_of, w.W, w.U, w.Vt, w.Sigma, rk)),
        "uncompressed": (yu, oracle_mod.apply_uncompressed(w.x, w.adapter_id, w.W, w.A, w.B)),
    }
    for what, (got, ref) in checks.items():
        err = row_rel_err(host(got), ref)
        assert err <= TOL[w.dtype], (what, err)


def test_pieces_equal_separate_calls(cases):
    """The call on 16385 tokens gives the same bits as three calls on its
    pieces' token ranges, for the compressed and the uncompressed path."""
    w = cases["bf16_T16385"]
    x, aid, cof = dev(w.x), dev(w.adapter_id), dev(w.cluster_of)
    W, U, Vt, S, A, B = (dev(a) for a in (w.W, w.U, w.Vt, w.Sigma, w.A, w.B))
    say("pieces: whole call against separate calls")
    y = cts.apply(x, aid, cof, W, U, Vt, S)
    yu = cts.apply_uncompressed(x, aid, W, A, B)
    parts, parts_u, t0 = [], [], 0
    for q in _pieces(w.T):
        sl = slice(t0, t0 + q)
        parts.append(cts.apply(x[sl].contiguous(), aid[sl].contiguous(), cof, W, U, Vt, S))
        parts_u.append(cts.apply_uncompressed(x[sl].contiguous(), aid[sl].contiguous(), W, A, B))
        t0 += q
    torch.cuda.synchronize()
    assert torch.equal(y, torch.cat(parts))
    assert torch.equal(yu, torch.cat(parts_u))


def test_pieces_multi(oracle_mod):
    """cts_apply_multi on 12000 tokens (two pieces of 6000): two modules with
    their V_k^T stacked, every row against the oracle."""
    base = dict(T=12000, d_in=128, r=16, n=40, K=4, ids="zipf")
    mods = [wl.synthetic("pm%d" % m, cfg=173 + 37 * m, d_out=d, with_lora=False, **base)
            for m, d in enumerate((64, 136))]
    w0 = mods[0]
    Vt = np.concatenate([m.Vt for m in mods], axis=1)
    say("pieces: apply_multi T=12000")
    ys = cts.apply_multi(dev(w0.x), dev(w0.adapter_id), dev(w0.cluster_of), [dev(m.W) for m in mods],
                         [dev(m.U) for m in mods], dev(Vt), [dev(m.Sigma) for m in mods])
    torch.cuda.synchronize()
    refs = oracle_mod.apply_multi(w0.x, w0.adapter_id, w0.cluster_of, [m.W for m in mods], [m.U for m in mods],
                                  Vt, [m.Sigma for m in mods])
    for m, (y, ref) in enumerate(zip(ys, refs)):
        assert row_rel_err(host(y), ref) <= TOL["bf16"], m
