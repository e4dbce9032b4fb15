"""GPU parity on the 32-layer decoder stack's own inputs: the tensors the
benchmark times (workloads.stack_*, drawn on the device from per-projection
seeds), layers 0, 15 and 31, all seven projections, run through the same
calls as the benchmark's step (one cts_sort_by_cluster for the batch, then
q/k/v and gate/up through cts_apply_multi_sorted with their V_k^T stacked
along r, o and down through it with one module), and 64 of the 512 tokens
compared with the fp64 oracle per projection.  The calls that sort for
themselves (cts_apply_multi, cts_apply) give the same bits."""
import numpy as np
import pytest
import torch

import paper_2407_00066_amd as cts
from paper_2407_00066_amd import workloads as wl

from _gpu_helpers import TOL, dev, host, row_rel_err, say

pytestmark = pytest.mark.gpu

GROUPS = (("q", "k", "v"), ("o",), ("gate", "up"), ("down",))


def _bits(t: torch.Tensor) -> np.ndarray:
    """bf16 tensor -> uint16 bit patterns on the host (the oracle widens them)."""
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def _tokens(oracle_mod, aid, cof, count=64):
    """64 tokens: both sides of every multiple of 64 in the cluster-sorted
    order (tile edges of every tile shape), the first cluster boundaries,
    then random positions up to `count`."""
    T = len(aid)
    perm, offs = oracle_mod.sort_by_cluster(aid, cof, wl.STACK["n"], wl.STACK["K"])
    pos = [0, T - 1] + [p for b in range(64, T, 64) for p in (b - 1, b)]
    pos += [q for o in offs[1:9] for q in (int(o) - 1, int(o))]
    rs = np.random.default_rng(512)
    toks = list(dict.fromkeys(int(perm[j]) for j in pos if 0 <= j < T))[:count]
    while len(toks) < count:
        t = int(rs.integers(0, T))
        if t not in toks:
            toks.append(t)
    return np.array(sorted(toks), np.int64)


@pytest.mark.parametrize("layer", [0, 15, 31])
def test_stack_bench_inputs_sampled(oracle_mod, layer):
    aid_h, cof_h = wl.stack_ids()
    aid, cof = dev(aid_h), dev(cof_h)
    xs = {4096: wl.stack_x(torch, "cuda", 4096), 14336: wl.stack_x(torch, "cuda", 14336)}
    x_o = wl.stack_x_o(torch, "cuda")
    d_in = {nm: di for nm, di, _ in wl.STACK_PROJ}
    mods = {nm: wl.stack_module(torch, "cuda", layer, nm) for nm, _, _ in wl.STACK_PROJ}
    xin = {nm: (x_o if nm == "o" else xs[d_in[nm]]) for nm in mods}
    say("stack layer %d: the benchmark's calls" % layer)
    n, K = wl.STACK["n"], wl.STACK["K"]
    perm = torch.empty(len(aid_h), dtype=torch.int32, device="cuda")
    offs = torch.empty(K + 1, dtype=torch.int32, device="cuda")
    bk = torch.empty(cts.bucketing_size(len(aid_h), n, K), dtype=torch.uint8, device="cuda")
    cts.sort_by_cluster(aid, cof, n, K, perm=perm, offsets=offs, bucketing=bk)
    ys, ys_own = {}, {}
    for grp in GROUPS:
        x = xin[grp[0]]
        Vt = torch.cat([mods[nm][2] for nm in grp], dim=1).contiguous()
        Ws, Us, Ss = ([mods[nm][i] for nm in grp] for i in (0, 1, 3))
        ys.update(zip(grp, cts.apply_multi_sorted(perm, bk, x, Ws, Us, Vt, Ss)))
        if len(grp) == 1:
            ys_own[grp[0]] = cts.apply(x, aid, cof, Ws[0], Us[0], Vt, Ss[0])
        else:
            ys_own.update(zip(grp, cts.apply_multi(x, aid, cof, Ws, Us, Vt, Ss)))
    torch.cuda.synchronize()
    for nm in ys:
        assert torch.equal(ys[nm], ys_own[nm]), nm
    toks = _tokens(oracle_mod, aid_h, cof_h)
    assert len(toks) == 64
    for nm, _, _ in wl.STACK_PROJ:
        W, U, Vt, S = (_bits(t) for t in mods[nm])
        ref = oracle_mod.apply(_bits(xin[nm]), aid_h, cof_h, W, U, Vt, S, tokens=toks)
        yh = host(ys[nm])
        assert np.isfinite(yh).all(), nm
        err = row_rel_err(yh[toks], ref)
        assert err <= TOL["bf16"], (nm, err)
