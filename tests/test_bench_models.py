"""The benchmark's byte and flop models (CPU): the figures its roofline lines
divide by, pinned to values worked out by hand from the layer's definition
(y = W x + U_k Sigma_i V_k^T x, bf16 operands, each tensor read once)."""
import os
import sys
import types

import numpy as np
import pytest

sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
import bench  # noqa: E402


def _w(T, d_in, d_out, r, dtype="bf16"):
    return types.SimpleNamespace(T=T, d_in=d_in, d_out=d_out, r=r, dtype=dtype)


# (T, d_in, d_out, r, touched clusters) -> (flops, bytes) of the fused GEMM:
#   flops 2 T d_in d_out + 2 T r d_out
#   bytes 2 (W + X + Y + touched U_k + Z')
GEMM_CASES = {
    # 4096 tokens of a 4096 x 4096 projection, 17 touched rank-64 clusters:
    # 137 438 953 472 + 2 147 483 648 flops; 3 x 33 554 432 (W, X, Y)
    # + 8 912 896 (U) + 524 288 (Z') bytes
    "prefill_mix": ((4096, 4096, 4096, 64, 17), (139_586_437_120, 110_100_480)),
    # 64 tokens, one cluster: 2 147 483 648 + 33 554 432 flops;
    # 33 554 432 (W) + 2 x 524 288 (X, Y) + 524 288 (U) + 8 192 (Z') bytes
    "decode_q": ((64, 4096, 4096, 64, 1), (2_181_038_080, 35_135_488)),
    # 256 tokens into 14336 features, 45 touched rank-128 clusters
    "mlp_up": ((256, 4096, 14336, 128, 45),
               (2 * 256 * 4096 * 14336 + 2 * 256 * 128 * 14336,
                2 * (14336 * 4096 + 256 * 4096 + 256 * 14336 + 45 * 14336 * 128 + 256 * 128))),
}


@pytest.mark.parametrize("name", list(GEMM_CASES))
def test_fused_gemm_model(name):
    (T, d_in, d_out, r, touched), (flops, nbytes) = GEMM_CASES[name]
    f, b = bench.main_kernel_model(_w(T, d_in, d_out, r), touched)
    assert f == flops
    assert b == nbytes


def test_fused_gemm_model_with_full_ranks_matches_uniform():
    """A rank per cluster equal to r everywhere gives the uniform model."""
    rs = np.random.default_rng(7)
    T, n, K, r = 300, 40, 6, 32
    w = _w(T, 256, 192, r)
    w.adapter_id = rs.integers(0, n, T)
    w.cluster_of = rs.integers(0, K, n)
    touched = len(set(w.cluster_of[w.adapter_id].tolist()))
    ranks = np.full(K, r)
    assert bench.main_kernel_model(w, touched, ranks) == bench.main_kernel_model(w, touched)
    # halving one touched cluster's rank removes its share of U_k and of the U_k Z' flops
    k0 = int(w.cluster_of[w.adapter_id[0]])
    ranks[k0] = r // 2
    f1, b1 = bench.main_kernel_model(w, touched, ranks)
    f0, b0 = bench.main_kernel_model(w, touched)
    t0 = int((w.cluster_of[w.adapter_id] == k0).sum())
    assert f0 - f1 == 2.0 * t0 * (r // 2) * w.d_out
    assert b0 - b1 == 2 * ((r // 2) * w.d_out + t0 * (r // 2))


def test_layer_model_decode():
    """Whole layer: W X + U_k Sigma_i V_k^T X, each touched basis and Sigma_i once."""
    T, d_in, d_out, r, touched, distinct = 64, 4096, 4096, 64, 1, 48
    f, b = bench.layer_model(T, d_in, d_out, r, 2, touched, distinct)
    assert f == 2 * 64 * 4096 * 4096 + 2 * 64 * (4096 * 64 + 64 * 64 + 4096 * 64)
    assert b == 2 * (4096 * 4096 + 64 * 4096 + 64 * 4096 + 64 * (4096 + 4096) + 48 * 64 * 64)
    # diagonal Sigma_i: r entries per adapter
    f2, b2 = bench.layer_model(T, d_in, d_out, r, 2, touched, distinct, sigma_elems=r)
    assert f - f2 == 2 * T * (r * r - r)
    assert b - b2 == 2 * distinct * (r * r - r)


def test_roofline_bound_and_fraction():
    # prefill: 139.6 GF over 110 MB is past the ridge (2.5 PF / 8 TB/s = 312 flop/B)
    f, b = GEMM_CASES["prefill_mix"][1]
    roof = bench.roofline_of(f, b, 111.1e-6, "bf16")
    assert roof["bound"] == "mfma" and roof["unit"] == "TFLOP/s" and roof["peak"] == 2500.0
    assert roof["frac"] == pytest.approx(f / 111.1e-6 / 1e12 / 2500.0, abs=1e-4)
    # decode: 2.18 GF over 35 MB is HBM-bound
    f, b = GEMM_CASES["decode_q"][1]
    roof = bench.roofline_of(f, b, 10.87e-6, "bf16")
    assert roof["bound"] == "hbm" and roof["unit"] == "GB/s" and roof["peak"] == 8000.0
    assert roof["frac"] == pytest.approx(b / 10.87e-6 / 1e9 / 8000.0, abs=1e-4)
    # fp32 inputs take the fp32 matrix-core peak
    roof = bench.roofline_of(1e12, 1e3, 1.0, "f32")
    assert roof["bound"] == "mfma" and roof["peak"] == 157.3
