"""GPU parity of multi-module batching (cts_apply_multi): M projections of one
layer on the same x, adapter ids and cluster map, the V_k^T stacked along r,
against the oracle's per-module layer and against cts_apply per module."""
import numpy as np
import pytest
import torch

import paper_2407_00066_amd as cts
from paper_2407_00066_amd import workloads as wl

from _gpu_helpers import TOL, dev, host, row_rel_err, say

pytestmark = pytest.mark.gpu

CASES = {
    # q, k, v of a decode batch: bucketing inside the shrink (T <= 128), 64x64 tiles split along d_in
    "qkv_decode": dict(cfg=140, T=64, d_in=512, d_outs=(512, 128, 128), r=32, n=40, K=4),
    # mid-size batch, Zipf ids
    "qkv_mid": dict(cfg=141, T=300, d_in=256, d_outs=(256, 64, 64), r=16, n=50, K=5, ids="zipf"),
    # gate and up of a prefill batch: 256x256 tiles
    "gate_up_prefill": dict(cfg=142, T=2100, d_in=128, d_outs=(512, 512), r=64, n=60, K=6, ids="prefill",
                            n_seq=12, seq_len=(60, 300)),
    # fp32, ragged
    "f32_pair": dict(cfg=143, T=77, d_in=128, d_outs=(96, 64), r=16, n=10, K=3, dtype="f32"),
    # the modules' GEMMs in one launch split along d_in (decode tile, split 4) with one split-K sum
    # over all modules' partials
    "qkv_grouped_split": dict(cfg=148, T=64, d_in=2048, d_outs=(512, 128, 128), r=32, n=40, K=4),
    # the same with 128x64 tiles (split 2), a module narrower than one row tile, Zipf ids
    "mixed_grouped_split": dict(cfg=149, T=200, d_in=1024, d_outs=(256, 128, 64), r=16, n=60, K=5, ids="zipf"),
}


def _modules(kw):
    kw = dict(kw)
    d_outs = kw.pop("d_outs")
    cfg = kw.pop("cfg")
    mods = [wl.synthetic("m%d" % m, cfg=cfg + 37 * m, d_out=d, with_lora=False, **kw) for m, d in enumerate(d_outs)]
    w0 = mods[0]
    Vt = np.concatenate([m.Vt for m in mods], axis=1)          # [K][M r][d_in]
    return w0, mods, Vt


@pytest.mark.parametrize("name", sorted(CASES))
def test_apply_multi_matches_oracle(oracle_mod, name):
    w0, mods, Vt = _modules(CASES[name])
    x, aid, cof = dev(w0.x), dev(w0.adapter_id), dev(w0.cluster_of)
    say("apply_multi %s (M=%d)" % (name, len(mods)))
    ys = cts.apply_multi(x, aid, cof, [dev(m.W) for m in mods], [dev(m.U) for m in mods], dev(Vt),
                         [dev(m.Sigma) for m in mods])
    torch.cuda.synchronize()
    refs = oracle_mod.apply_multi(w0.x, w0.adapter_id, w0.cluster_of, [m.W for m in mods], [m.U for m in mods],
                                  Vt, [m.Sigma for m in mods])
    for m, (y, ref) in enumerate(zip(ys, refs)):
        assert row_rel_err(host(y), ref) <= TOL[w0.dtype], m
    # and against the single-module call with that module's arrays
    for m, mod in enumerate(mods):
        y1 = cts.apply(x, aid, cof, dev(mod.W), dev(mod.U), dev(mod.Vt), dev(mod.Sigma))
        torch.cuda.synchronize()
        assert row_rel_err(host(ys[m]), host(y1)) <= TOL[w0.dtype], m


def test_apply_multi_one_module_is_apply():
    w0, mods, Vt = _modules(dict(cfg=144, T=500, d_in=256, d_outs=(320,), r=32, n=30, K=4, ids="zipf"))
    args = [dev(a) for a in (w0.x, w0.adapter_id, w0.cluster_of)]
    ys = cts.apply_multi(*args, [dev(w0.W)], [dev(w0.U)], dev(Vt), [dev(w0.Sigma)])
    y1 = cts.apply(*args, dev(w0.W), dev(w0.U), dev(w0.Vt), dev(w0.Sigma))
    torch.cuda.synchronize()
    assert torch.equal(ys[0], y1)


@pytest.mark.parametrize("name", sorted(CASES))
def test_apply_multi_sorted_shares_one_bucketing(oracle_mod, name):
    """One cts_sort_by_cluster for the batch, then cts_apply_multi_sorted for
    every module group and for single modules (M = 1): bit for bit the
    results of cts_apply_multi / cts_apply, which sort the ids themselves."""
    w0, mods, Vt = _modules(CASES[name])
    x, aid, cof = dev(w0.x), dev(w0.adapter_id), dev(w0.cluster_of)
    say("apply_multi_sorted %s (M=%d)" % (name, len(mods)))
    perm, offs, bk = cts.sort_by_cluster(aid, cof, w0.n, w0.K, bucketing=True)
    ys = cts.apply_multi_sorted(perm, bk, x, [dev(m.W) for m in mods], [dev(m.U) for m in mods], dev(Vt),
                                [dev(m.Sigma) for m in mods])
    ref = cts.apply_multi(x, aid, cof, [dev(m.W) for m in mods], [dev(m.U) for m in mods], dev(Vt),
                          [dev(m.Sigma) for m in mods])
    singles = [cts.apply_multi_sorted(perm, bk, x, [dev(m.W)], [dev(m.U)], dev(m.Vt), [dev(m.Sigma)])[0]
               for m in mods]
    torch.cuda.synchronize()
    for m in range(len(mods)):
        assert torch.equal(ys[m], ref[m]), m
        y1 = cts.apply(x, aid, cof, dev(mods[m].W), dev(mods[m].U), dev(mods[m].Vt), dev(mods[m].Sigma))
        torch.cuda.synchronize()
        assert torch.equal(singles[m], y1), m
    oref = oracle_mod.apply_multi(w0.x, w0.adapter_id, w0.cluster_of, [m.W for m in mods], [m.U for m in mods],
                                  Vt, [m.Sigma for m in mods])
    for m in range(len(mods)):
        assert row_rel_err(host(ys[m]), oref[m]) <= TOL[w0.dtype], m


def test_apply_multi_sorted_many_calls_one_sort(oracle_mod):
    """As a decoder step: one sort, then several layers' calls on the same
    bucketing (other inputs each), interleaved with a different batch's
    sort on another buffer."""
    kw = dict(cfg=145, T=512, d_in=256, d_outs=(256, 128), r=32, n=200, K=10)
    w0, mods, Vt = _modules(kw)
    other = wl.synthetic("other_ids", cfg=146, T=512, d_in=64, d_out=64, r=8, n=200, K=10, with_lora=False)
    x, aid, cof = dev(w0.x), dev(w0.adapter_id), dev(w0.cluster_of)
    say("apply_multi_sorted: one sort, four calls")
    perm, _, bk = cts.sort_by_cluster(aid, cof, w0.n, w0.K, bucketing=True)
    cts.sort_by_cluster(dev(other.adapter_id), cof, w0.n, w0.K, bucketing=True)
    outs = [cts.apply_multi_sorted(perm, bk, x, [dev(m.W) for m in mods], [dev(m.U) for m in mods], dev(Vt),
                                   [dev(m.Sigma) for m in mods]) for _ in range(4)]
    torch.cuda.synchronize()
    for ys in outs[1:]:
        for a, b in zip(ys, outs[0]):
            assert torch.equal(a, b)
    oref = oracle_mod.apply_multi(w0.x, w0.adapter_id, w0.cluster_of, [m.W for m in mods], [m.U for m in mods],
                                  Vt, [m.Sigma for m in mods])
    for m in range(len(mods)):
        assert row_rel_err(host(outs[0][m]), oref[m]) <= TOL["bf16"], m


@pytest.mark.parametrize("name", sorted(CASES))
def test_apply_multi_packed(name):
    """cts_apply_multi_packed: the modules' outputs as column slices of one
    packed y with padded rows, from the ids and from a shared bucketing; each
    slice bit for bit cts_apply_multi's output for that module, the padding
    columns untouched."""
    w0, mods, Vt = _modules(CASES[name])
    x, aid, cof = dev(w0.x), dev(w0.adapter_id), dev(w0.cluster_of)
    Ws, Us, Ss = [dev(m.W) for m in mods], [dev(m.U) for m in mods], [dev(m.Sigma) for m in mods]
    d_out = [m.d_out for m in mods]
    ldy = sum(d_out) + 16
    odt = x.dtype
    say("apply_multi_packed %s (M=%d, ldy=%d)" % (name, len(mods), ldy))
    ref = cts.apply_multi(x, aid, cof, Ws, Us, dev(Vt), Ss)
    y_ids = torch.full((w0.T, ldy), 7.0, dtype=odt, device="cuda")
    cts.apply_multi_packed(x, Ws, Us, dev(Vt), Ss, adapter_id=aid, cluster_of=cof, out=y_ids)
    perm, _, bk = cts.sort_by_cluster(aid, cof, w0.n, w0.K, bucketing=True)
    y_srt = torch.full((w0.T, ldy), 7.0, dtype=odt, device="cuda")
    cts.apply_multi_packed(x, Ws, Us, dev(Vt), Ss, perm=perm, bucketing=bk, out=y_srt)
    torch.cuda.synchronize()
    for y in (y_ids, y_srt):
        c = 0
        for m, dm in enumerate(d_out):
            assert torch.equal(y[:, c:c + dm], ref[m]), m
            c += dm
        assert bool((y[:, c:] == 7.0).all())


def test_apply_multi_packed_pieces(oracle_mod):
    """A packed output over a batch of 9000 tokens (two pieces)."""
    w0, mods, Vt = _modules(dict(cfg=147, T=9000, d_in=128, d_outs=(64, 32), r=16, n=30, K=3, ids="zipf"))
    x, aid, cof = dev(w0.x), dev(w0.adapter_id), dev(w0.cluster_of)
    say("apply_multi_packed over 9000 tokens")
    y = cts.apply_multi_packed(x, [dev(m.W) for m in mods], [dev(m.U) for m in mods], dev(Vt),
                               [dev(m.Sigma) for m in mods], adapter_id=aid, cluster_of=cof)
    torch.cuda.synchronize()
    oref = oracle_mod.apply_multi(w0.x, w0.adapter_id, w0.cluster_of, [m.W for m in mods], [m.U for m in mods],
                                  Vt, [m.Sigma for m in mods])
    yh = host(y)
    assert row_rel_err(yh[:, :64], oref[0]) <= TOL["bf16"]
    assert row_rel_err(yh[:, 64:], oref[1]) <= TOL["bf16"]
