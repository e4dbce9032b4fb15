"""GPU parity of the diagonal-Sigma variant (cts_apply_diag; Sec. 3.1, eq.
JD-Diag) against the fp64 oracle's apply_diag, through the C ABI.  Same
tolerances as the full-Sigma path: per-token inf-norm relative error <= 1e-5
(fp32 inputs) or 2e-2 (bf16 inputs, fp32 accumulation)."""
import numpy as np
import pytest
import torch

import paper_2407_00066_amd as cts
from paper_2407_00066_amd import workloads as wl

from _gpu_helpers import TOL, dev, host, row_rel_err, say
from test_gpu_parity import SMALL, _sample_tokens

pytestmark = pytest.mark.gpu

DIAG_SMALL = ["tiny_fp32", "f32_ragged", "bf16_ragged", "bf16_large_tiles", "bf16_T1",
              "bf16_decode_split4", "bf16_ring_ragged", "bf16_wide_split", "bf16_mid_tiles",
              "bf16_empty_clusters"]


@pytest.fixture(scope="module")
def cases():
    out = {}
    for name in DIAG_SMALL:
        kw = dict(SMALL[name])
        w = wl.synthetic(name, **kw)
        out[name] = (w, wl.sigma_diagonals(kw["cfg"], w.n, w.r, w.dtype))
    return out


def _args(w, sig):
    return (dev(w.x), dev(w.adapter_id), dev(w.cluster_of), dev(w.W), dev(w.U), dev(w.Vt), dev(sig))


@pytest.mark.parametrize("name", DIAG_SMALL)
def test_apply_diag_small(oracle_mod, cases, name):
    w, sig = cases[name]
    say("apply_diag %s T=%d d_in=%d d_out=%d r=%d n=%d K=%d" % (name, w.T, w.d_in, w.d_out, w.r, w.n, w.K))
    y = cts.apply_diag(*_args(w, sig))
    torch.cuda.synchronize()
    ref = oracle_mod.apply_diag(w.x, w.adapter_id, w.cluster_of, w.W, w.U, w.Vt, sig)
    err = row_rel_err(host(y), ref)
    assert err <= TOL[w.dtype], err


def test_zero_diag_is_exactly_base_layer(cases):
    """sigma_i = 0 and Sigma_i = 0 both add exactly nothing: identical bits."""
    w, sig = cases["bf16_ragged"]
    say("apply_diag zero sigma bitwise")
    y_d = cts.apply_diag(*_args(w, np.zeros_like(sig)))
    y_f = cts.apply(dev(w.x), dev(w.adapter_id), dev(w.cluster_of), dev(w.W), dev(w.U), dev(w.Vt),
                    dev(np.zeros_like(w.Sigma)))
    torch.cuda.synchronize()
    assert torch.equal(y_d, y_f)


def test_diag_matches_full_path_with_diagonal_sigma(cases):
    """The same layer through cts_apply with Sigma_i = diag(sigma_i)."""
    w, sig = cases["bf16_large_tiles"]
    say("apply_diag vs apply with diagonal Sigma")
    sig32 = wl.bf16_bits_to_f32(sig)
    full = np.zeros((w.n, w.r, w.r), np.float32)
    for i in range(w.n):
        np.fill_diagonal(full[i], sig32[i])
    y_d = cts.apply_diag(*_args(w, sig))
    y_f = cts.apply(dev(w.x), dev(w.adapter_id), dev(w.cluster_of), dev(w.W), dev(w.U), dev(w.Vt),
                    dev(wl.f32_to_bf16_bits(full)))
    torch.cuda.synchronize()
    assert row_rel_err(host(y_d), host(y_f).astype(np.float64)) <= 1e-2


@pytest.mark.parametrize("name", ["decode_q", "prefill_mix"])
def test_apply_diag_full_size_sampled(oracle_mod, name):
    w = wl.make(name)
    sig = wl.sigma_diagonals(wl.CONFIGS[name]["cfg"], w.n, w.r, w.dtype)
    toks = _sample_tokens(w, oracle_mod)
    say("apply_diag %s (full size), %d sampled tokens" % (name, len(toks)))
    y = cts.apply_diag(*_args(w, sig))
    torch.cuda.synchronize()
    yh = host(y)
    assert np.isfinite(yh).all()
    ref = oracle_mod.apply_diag(w.x, w.adapter_id, w.cluster_of, w.W, w.U, w.Vt, sig, tokens=toks)
    assert row_rel_err(yh[toks], ref) <= TOL["bf16"]
