"""Seeded synthetic inputs for the batched multi-adapter linear layer.

This module draws random numbers and lays them out; it holds none of the
method's arithmetic.  Both the GPU tests/benchmark and the CPU oracle tests
take their inputs from here, and from nowhere else.

Recipe (one independent numpy PCG64 stream per tensor):
  seed = 240700066 + 1000 * config_index + stream_id
Gaussians are drawn in float64, scaled to the stated variance ("N(0, s)" means
variance s), then cast to float32, or cast to float32 and rounded to nearest
even bfloat16.  bfloat16 arrays are returned as uint16 bit patterns.
Shared bases U_k, V_k are the Q factors of a float64 QR of a Gaussian matrix.
Clusters are a seeded balanced assignment: a permutation of the adapters cut
into K groups of n/K.  "Zipf(s)" is the finite law P(rank k) ~ k^-s over
k = 1..n, rank k meaning adapter k-1.

The shapes mirror the paper's serving setting: Mistral-7B-sized layers,
rank-16 LoRAs, up to ~1000 adapters, random adapters per request, and the
compression settings it reports (JD-Full, 25 clusters at ~1000 LoRAs).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

SEED_BASE = 240700066

# stream ids
_S_W, _S_U, _S_V, _S_SIG, _S_X, _S_IDS, _S_CLU, _S_A, _S_B, _S_LEN, _S_SEQ, _S_SDIAG, _S_RANK = range(1, 14)


def _rng(cfg: int, stream: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(SEED_BASE + 1000 * cfg + stream))


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round float32 to the nearest bfloat16 (ties to even); returns uint16 bits."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    rounded = u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return (rounded >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _cast(a64: np.ndarray, dtype: str) -> np.ndarray:
    a32 = a64.astype(np.float32)
    return a32 if dtype == "f32" else f32_to_bf16_bits(a32)


def _gauss(rng: np.random.Generator, shape, var: float, dtype: str, chunk_rows: int = 64) -> np.ndarray:
    """N(0, var) of the given shape, drawn row-block by row-block along axis 0
    (the values equal one big draw; chunking only bounds the float64 temporary)."""
    out = np.empty(shape, np.float32 if dtype == "f32" else np.uint16)
    std = float(np.sqrt(var))
    for i in range(0, shape[0], chunk_rows):
        j = min(shape[0], i + chunk_rows)
        out[i:j] = _cast(rng.standard_normal((j - i,) + tuple(shape[1:])) * std, dtype)
    return out


def _orthonormal(rng: np.random.Generator, K: int, rows: int, r: int) -> np.ndarray:
    """K independent rows x r matrices with orthonormal columns (float64)."""
    out = np.empty((K, rows, r), np.float64)
    for k in range(K):
        q, _ = np.linalg.qr(rng.standard_normal((rows, r)))
        out[k] = q
    return out


def balanced_clusters(rng: np.random.Generator, n: int, K: int) -> np.ndarray:
    """cluster_of[n]: a random permutation of adapters cut into K groups of n//K
    (the first n % K groups get one extra)."""
    perm = rng.permutation(n)
    cluster_of = np.empty(n, np.int32)
    sizes = [n // K + (1 if g < n % K else 0) for g in range(K)]
    pos = 0
    for g, s in enumerate(sizes):
        cluster_of[perm[pos:pos + s]] = g
        pos += s
    return cluster_of


def zipf_ids(rng: np.random.Generator, n: int, size: int, s: float = 1.1) -> np.ndarray:
    p = np.arange(1, n + 1, dtype=np.float64) ** (-s)
    p /= p.sum()
    return rng.choice(n, size=size, p=p).astype(np.int32)


def prefill_lengths(rng: np.random.Generator, n_seq: int, total: int, lo: int, hi: int) -> np.ndarray:
    """n_seq lengths drawn uniformly from {lo..hi}, rescaled to sum to `total`:
    scale by total/sum, floor, clamp to [lo, hi], then add (or remove) one
    token per sequence in sequence order, staying inside [lo, hi]."""
    raw = rng.integers(lo, hi + 1, size=n_seq).astype(np.float64)
    lens = np.clip(np.floor(raw * total / raw.sum()).astype(np.int64), lo, hi)
    i = 0
    while lens.sum() != total:
        step = 1 if lens.sum() < total else -1
        if lo <= lens[i] + step <= hi:
            lens[i] += step
        i = (i + 1) % n_seq
    return lens


@dataclass
class Workload:
    """One batch of one multi-adapter linear layer.

    Layouts: x[T][d_in], W[d_out][d_in], U[K][d_out][r], Vt[K][r][d_in] (= V_k^T),
    Sigma[n][r][r] (applied as z' = Sigma_i z), A[n][r_l][d_in], B[n][d_out][r_l],
    adapter_id[T], cluster_of[n].  Float arrays are float32 (dtype "f32") or
    bfloat16 bits in uint16 (dtype "bf16").
    """
    name: str
    dtype: str
    T: int
    d_in: int
    d_out: int
    r: int
    n: int
    K: int
    r_l: int
    x: np.ndarray
    W: np.ndarray
    U: np.ndarray
    Vt: np.ndarray
    Sigma: np.ndarray
    adapter_id: np.ndarray
    cluster_of: np.ndarray
    A: np.ndarray | None = None
    B: np.ndarray | None = None
    meta: dict = field(default_factory=dict)


def synthetic(name: str, cfg: int, *, T: int, d_in: int, d_out: int, r: int, n: int, K: int,
              r_l: int = 16, dtype: str = "bf16", ids: str = "uniform", w_var: float | None = None,
              sigma_var: float | None = None, a_var: float | None = None, b_var: float | None = None,
              x_var: float = 1.0, with_lora: bool = True, n_seq: int = 32,
              seq_len: tuple[int, int] = (32, 256)) -> Workload:
    """General seeded workload.  ids: "uniform" (per token), "zipf" (Zipf(1.1)
    per token), or "prefill" (n_seq sequences of lengths U{seq_len} rescaled to
    T, one Zipf(1.1) adapter per sequence, tokens contiguous per sequence)."""
    w_var = 1.0 / d_in if w_var is None else w_var
    sigma_var = 1.0 / r if sigma_var is None else sigma_var
    a_var = 1.0 / d_in if a_var is None else a_var
    b_var = 1.0 / (64.0 * r_l) if b_var is None else b_var

    W = _gauss(_rng(cfg, _S_W), (d_out, d_in), w_var, dtype)
    U = _cast(_orthonormal(_rng(cfg, _S_U), K, d_out, r), dtype)
    Vt = _cast(np.ascontiguousarray(_orthonormal(_rng(cfg, _S_V), K, d_in, r).transpose(0, 2, 1)), dtype)
    Sigma = _gauss(_rng(cfg, _S_SIG), (n, r, r), sigma_var, dtype)
    x = _gauss(_rng(cfg, _S_X), (T, d_in), x_var, dtype)
    cluster_of = balanced_clusters(_rng(cfg, _S_CLU), n, K)
    meta = {}
    rid = _rng(cfg, _S_IDS)
    if ids == "uniform":
        adapter_id = rid.integers(0, n, size=T).astype(np.int32)
    elif ids == "zipf":
        adapter_id = zipf_ids(rid, n, T)
    elif ids == "prefill":
        lens = prefill_lengths(_rng(cfg, _S_LEN), n_seq, T, seq_len[0], seq_len[1])
        seq_ad = zipf_ids(_rng(cfg, _S_SEQ), n, n_seq)
        adapter_id = np.repeat(seq_ad, lens).astype(np.int32)
        meta["seq_lens"] = lens
        meta["seq_adapters"] = seq_ad
    else:
        raise ValueError(ids)
    A = B = None
    if with_lora:
        A = _gauss(_rng(cfg, _S_A), (n, r_l, d_in), a_var, dtype, chunk_rows=8)
        B = _gauss(_rng(cfg, _S_B), (n, d_out, r_l), b_var, dtype, chunk_rows=8)
    return Workload(name, dtype, T, d_in, d_out, r, n, K, r_l, x, W, U, Vt, Sigma,
                    adapter_id, cluster_of, A, B, meta)


# The named workloads.  The index is the seed's config index.
CONFIGS = {
    # d=256 fp32; 8 rank-4 LoRAs ~N(0,1/16); one r=16 cluster; 32 uniform tokens.
    "tiny_fp32": dict(cfg=0, T=32, d_in=256, d_out=256, r=16, n=8, K=1, r_l=4, dtype="f32",
                      ids="uniform", sigma_var=1.0 / 16, a_var=1.0 / 16, b_var=1.0 / 16),
    # 7B-shaped q_proj decode: d=4096, 100 LoRAs, one r=64 cluster, 64 uniform tokens.
    "decode_q": dict(cfg=1, T=64, d_in=4096, d_out=4096, r=64, n=100, K=1, ids="uniform"),
    # Prefill mix: 1000 LoRAs in 25 clusters (r=64), 32 sequences, 4096 tokens.
    "prefill_mix": dict(cfg=2, T=4096, d_in=4096, d_out=4096, r=64, n=1000, K=25, ids="prefill"),
    # MLP gate/up: 4096 -> 14336, 1000 LoRAs in 50 clusters (r=128), 256 Zipf tokens.
    "mlp_up": dict(cfg=3, T=256, d_in=4096, d_out=14336, r=128, n=1000, K=50, ids="zipf"),
}

# The 32-layer 7B-shaped decoder stack: every linear projection of a layer,
# 1000 LoRAs in 50 clusters (r=64) per projection, 512 uniform decode tokens.
STACK_LAYERS = 32
STACK_PROJ = (("q", 4096, 4096), ("k", 4096, 1024), ("v", 4096, 1024), ("o", 4096, 4096),
              ("gate", 4096, 14336), ("up", 4096, 14336), ("down", 14336, 4096))
STACK = dict(T=512, r=64, n=1000, K=50, ids="uniform")
# one parity workload per distinct projection shape of the stack
for _i, (_name, _din, _dout) in enumerate((("q", 4096, 4096), ("kv", 4096, 1024),
                                            ("gate", 4096, 14336), ("down", 14336, 4096))):
    CONFIGS["stack_" + _name] = dict(cfg=10 + _i, d_in=_din, d_out=_dout, with_lora=False, **STACK)


def sigma_diagonals(cfg: int, n: int, r: int, dtype: str, var: float = 1.0) -> np.ndarray:
    """Diagonal Sigma_i (Sec. 3.1, JD-Diag) as [n][r], entries ~N(0, var): with
    var = 1 the scaled z'_q = sigma_i[q] z_q keeps the magnitude of z, as the
    full Sigma_i ~N(0, 1/r) does."""
    return _gauss(_rng(cfg, _S_SDIAG), (n, r), var, dtype)


def mixed_ranks(cfg: int, count: int, r_max: int, lo: int = 16) -> np.ndarray:
    """A rank per cluster (Sec. 3.2) or per uncompressed LoRA (App. H: ranks
    drawn uniformly between 16 and 64): multiples of 8, uniform in [lo, r_max]."""
    lo = min(lo, r_max)
    return (8 * _rng(cfg, _S_RANK).integers(lo // 8, r_max // 8 + 1, size=count)).astype(np.int32)


def make(name: str, **overrides) -> Workload:
    spec = dict(CONFIGS[name])
    spec.update(overrides)
    return synthetic(name, **spec)


# ---- the 32-layer stack's tensors, generated on the device ----------------
# The stack holds ~32 GB of weights, so its tensors are drawn on the GPU with
# torch's generator, each from a seed of its own (layer, projection, tensor),
# so that any projection can be regenerated alone: the benchmark and the
# parity test of its inputs draw the same values.  Variances: W ~N(0,1/d_in),
# U ~N(0,1/d_out), V_k^T ~N(0,1/d_in) (Gaussian bases, not orthonormalized:
# the layer's cost does not depend on it), Sigma ~N(0,1/r), x ~N(0,1).
_STACK_SEED = SEED_BASE + 500_000
STACK_TENSORS = ("W", "U", "Vt", "Sigma")


def stack_ids():
    """(adapter_id[T], cluster_of[n]) of the stack batch: uniform ids, one
    balanced cluster map shared by all projections."""
    rs = np.random.default_rng(SEED_BASE + 501)
    aid = rs.integers(0, STACK["n"], STACK["T"]).astype(np.int32)
    cof = balanced_clusters(rs, STACK["n"], STACK["K"])
    return aid, cof


def _stack_draw(torch, device, seed, shape, var):
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return (torch.randn(shape, generator=g, device=device) * float(np.sqrt(var))).to(torch.bfloat16)


def stack_x(torch, device, d_in: int):
    """The stack's input rows for projections reading d_in features: q/k/v
    and gate/up share x[T][4096]; o gets its own x[T][4096] (index 1); down
    x[T][14336]."""
    return _stack_draw(torch, device, _STACK_SEED + d_in, (STACK["T"], d_in), 1.0)


def stack_x_o(torch, device):
    return _stack_draw(torch, device, _STACK_SEED + 1, (STACK["T"], 4096), 1.0)


def stack_module(torch, device, layer: int, proj: str):
    """(W, U, Vt, Sigma) of one projection of the stack (bf16, on device)."""
    names = [p[0] for p in STACK_PROJ]
    pi = names.index(proj)
    _, d_in, d_out = STACK_PROJ[pi]
    T, r, n, K = STACK["T"], STACK["r"], STACK["n"], STACK["K"]
    shapes = {"W": ((d_out, d_in), 1.0 / d_in), "U": ((K, d_out, r), 1.0 / d_out),
              "Vt": ((K, r, d_in), 1.0 / d_in), "Sigma": ((n, r, r), 1.0 / r)}
    out = []
    for ti, t in enumerate(STACK_TENSORS):
        shape, var = shapes[t]
        out.append(_stack_draw(torch, device, _STACK_SEED + 100_000 + 1000 * layer + 10 * pi + ti, shape, var))
    return tuple(out)


def stack_lora(torch, device, layer: int, proj: str, r_l: int = 16):
    """(A, B) of one projection's uncompressed rank-16 LoRAs for the
    comparison path (bf16, on device): A ~N(0,1/d_in), B ~N(0,1/(64 r_l)),
    so the adapter term is about 1/8 of the base term, as for the shared
    bases."""
    names = [p[0] for p in STACK_PROJ]
    pi = names.index(proj)
    _, d_in, d_out = STACK_PROJ[pi]
    n = STACK["n"]
    seed = _STACK_SEED + 200_000 + 1000 * layer + 10 * pi
    return (_stack_draw(torch, device, seed, (n, r_l, d_in), 1.0 / d_in),
            _stack_draw(torch, device, seed + 1, (n, d_out, r_l), 1.0 / (64 * r_l)))
