"""Seeded synthetic inputs for the affinity path (shared by the kernels' tests and the oracle).

This module only draws random numbers and rounds them to the storage dtype.  It
holds none of the affinity arithmetic: no RMS, no SiLU, no projection onto
W_gate / W_up, no aggregation.  The one matrix product here, ``x = x_pre + z·W_Oᵀ``,
builds the synthetic residual that enters the FFN pre-norm (the paper's x in the
affinity-score definition of Section 3 is that residual, which already contains the
attention output), so it is part of the data-generating process, not the method.

Workloads are shaped like the paper's models (Section 4): a Qwen3-0.6B-shaped layer
(d=1024, I=3072, 16 query / 8 KV heads of 128), its 28-layer model, a
Danube3-500M-shaped model (d=1536, I=4096, 16/8 heads of 96) and an 8B-class layer
stack (d=4096, I=14336, 32/8 heads of 128), plus a tiny fp32 layer for fast checks.
The calibration set of the paper (64 x 1024 FineWeb-Edu tokens through the real
models) is not available; these seeded stand-ins take its shapes and token count.

Two generators share one recipe:

* ``host_*``: numpy, fp64, bit-reproducible on any machine (tests, oracle parity);
* ``device_*``: torch on a GPU device, fp32, for workloads too large to build on the
  host (multi-layer benchmarks).  Same distributions, different random streams.

bf16 tensors are carried on the host as ``np.uint16`` bit patterns; ``to_f64`` turns
any stored array into the exact fp64 values the GPU reads.
"""
from __future__ import annotations

import dataclasses

import numpy as np

SEED_ROOT = 260913846  # arXiv id of the paper, used as the root of every seed


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    key: int               # workload id inside the seed
    n_layers: int
    d_model: int
    n_neurons: int         # I, FFN width
    n_q_heads: int         # H
    n_kv_groups: int       # G
    head_dim: int          # dh
    tokens: int            # calibration tokens per layer
    chunk: int             # tokens per accumulate call when streaming
    shards: tuple          # L values (logical devices)
    dtype: str             # "bf16" or "f32"
    weight_std: float
    n_outliers: int        # residual channels scaled up (massive activations)
    outlier_scale: float
    heads_dist: str        # "normal" or "student4"
    gamma_std: float = 0.1
    rms_eps: float = 1e-6

    @property
    def attn_width(self) -> int:
        return self.n_q_heads * self.head_dim


WORKLOADS = {
    "tiny": Workload("tiny", 0, 1, 64, 128, 8, 4, 16, 512, 512, (2,), "f32",
                     0.05, 0, 1.0, "normal"),
    "qwen3-0.6b-layer": Workload("qwen3-0.6b-layer", 1, 1, 1024, 3072, 16, 8, 128,
                                 65536, 65536, (2,), "bf16", 0.02, 4, 50.0, "normal"),
    "qwen3-0.6b-model": Workload("qwen3-0.6b-model", 2, 28, 1024, 3072, 16, 8, 128,
                                 262144, 16384, (4,), "bf16", 0.02, 4, 50.0, "normal"),
    "danube3-500m": Workload("danube3-500m", 3, 16, 1536, 4096, 16, 8, 96,
                             131072, 16384, (2, 4), "bf16", 0.02, 8, 30.0, "student4"),
    "8b-class-4layer": Workload("8b-class-4layer", 4, 4, 4096, 14336, 32, 8, 128,
                                131072, 16384, (4,), "bf16", 0.02, 4, 50.0, "normal"),
}


def shaped(base: Workload, **kw) -> Workload:
    """A workload with the same distributions and some shape fields replaced."""
    return dataclasses.replace(base, **kw)


# ----------------------------------------------------------------------------- rounding
def round_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round to bf16 (round-to-nearest-even from the fp32 value); returns uint16 bits."""
    f = np.ascontiguousarray(a, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16).astype(np.uint16)
    nan = np.isnan(f)
    if nan.any():
        r[nan] = 0x7FC0
    return r


def bf16_bits_to_f64(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def store(a64: np.ndarray, dtype: str) -> np.ndarray:
    """fp64 values -> storage array of the workload dtype (uint16 bits or float32)."""
    if dtype == "bf16":
        return round_to_bf16_bits(a64)
    if dtype == "f32":
        return np.ascontiguousarray(a64, dtype=np.float32)
    raise ValueError(f"unknown dtype {dtype!r}")


def to_f64(stored: np.ndarray) -> np.ndarray:
    """Exact fp64 values of a stored array."""
    if stored.dtype == np.uint16:
        return bf16_bits_to_f64(stored)
    return np.asarray(stored, dtype=np.float64)


# ----------------------------------------------------------------------------- host path
def _rng(wl: Workload, layer: int, stream: int, part: int) -> np.random.Generator:
    """Independent stream per (workload, layer, stream, part); stream 0 = weights."""
    return np.random.Generator(np.random.PCG64(
        np.random.SeedSequence([SEED_ROOT, wl.key, layer, stream, part])))


@dataclasses.dataclass
class LayerWeights:
    w_o: np.ndarray      # [d, H*dh]  (o_proj.weight layout)
    gamma: np.ndarray    # [d]        FFN pre-norm gain
    w_gate: np.ndarray   # [I, d]
    w_up: np.ndarray     # [I, d]
    w_down: np.ndarray   # [d, I]
    outliers: np.ndarray  # residual channels scaled up for this layer (int64)


def host_weights(wl: Workload, layer: int) -> LayerWeights:
    d, I, HD = wl.d_model, wl.n_neurons, wl.attn_width
    g = _rng(wl, layer, 0, 0)
    s = wl.weight_std
    w_o = g.standard_normal((d, HD)) * s
    gamma = 1.0 + g.standard_normal(d) * wl.gamma_std
    w_gate = g.standard_normal((I, d)) * s
    w_up = g.standard_normal((I, d)) * s
    w_down = g.standard_normal((d, I)) * s
    outl = np.sort(g.choice(d, size=wl.n_outliers, replace=False)) if wl.n_outliers else np.zeros(0, np.int64)
    return LayerWeights(store(w_o, wl.dtype), store(gamma, wl.dtype), store(w_gate, wl.dtype),
                        store(w_up, wl.dtype), store(w_down, wl.dtype), outl.astype(np.int64))


@dataclasses.dataclass
class AttnWeights:
    """Attention-side weights of a layer, used by the down edge into that layer."""
    w_q: np.ndarray      # [H*dh, d]  (q_proj.weight layout)
    w_k: np.ndarray      # [G*dh, d]
    w_v: np.ndarray      # [G*dh, d]
    gamma: np.ndarray    # [d]        attention pre-norm gain


def host_attn_weights(wl: Workload, layer: int) -> AttnWeights:
    """Seeded q/k/v projections and attention pre-norm gain of a layer (own stream)."""
    d, HD, GD = wl.d_model, wl.attn_width, wl.n_kv_groups * wl.head_dim
    g = _rng(wl, layer, 0, 1)
    s = wl.weight_std
    w_q = g.standard_normal((HD, d)) * s
    w_k = g.standard_normal((GD, d)) * s
    w_v = g.standard_normal((GD, d)) * s
    gamma = 1.0 + g.standard_normal(d) * wl.gamma_std
    return AttnWeights(store(w_q, wl.dtype), store(w_k, wl.dtype), store(w_v, wl.dtype),
                       store(gamma, wl.dtype))


def _heads(g: np.random.Generator, wl: Workload, n: int) -> np.ndarray:
    shape = (n, wl.n_q_heads, wl.head_dim)
    if wl.heads_dist == "normal":
        return g.standard_normal(shape)
    if wl.heads_dist == "student4":
        return g.standard_t(4.0, size=shape)
    raise ValueError(wl.heads_dist)


def host_tokens(wl: Workload, layer: int, weights: LayerWeights, n_tokens: int,
                chunk: int = 0, with_pre: bool = False) -> tuple:
    """(x [T,d], attn [T,H,dh]) in storage dtype for chunk ``chunk`` of a layer.

    x is the residual entering the FFN pre-norm: x_pre (the residual entering the
    layer's attention pre-norm) plus the attention output.  With ``with_pre`` the stored
    x_pre is returned as a third element; the down edge of layer i-1 reads it as the
    residual entering layer i.  Rows are drawn sequentially, so a smaller ``n_tokens``
    gives a prefix of a larger draw from the same chunk.
    """
    d = wl.d_model
    gx = _rng(wl, layer, 1, chunk)
    gz = _rng(wl, layer, 2, chunk)
    x_pre = gx.standard_normal((n_tokens, d))
    if wl.n_outliers:
        x_pre[:, weights.outliers] *= wl.outlier_scale
    z = store(_heads(gz, wl, n_tokens), wl.dtype)
    z64 = to_f64(z).reshape(n_tokens, wl.attn_width)
    x = x_pre + z64 @ to_f64(weights.w_o).T
    if with_pre:
        return store(x, wl.dtype), z, store(x_pre, wl.dtype)
    return store(x, wl.dtype), z


# ----------------------------------------------------------------------------- device path
def device_weights(wl: Workload, layer: int, device) -> dict:
    """Same recipe as ``host_weights`` with torch's generator on ``device``."""
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed(int(np.random.SeedSequence([SEED_ROOT, wl.key, layer, 0, 0]).generate_state(1)[0]))
    dt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    d, I, HD = wl.d_model, wl.n_neurons, wl.attn_width
    s = wl.weight_std

    def nrm(*shape):
        return torch.randn(*shape, generator=gen, device=device, dtype=torch.float32)

    out = {
        "w_o": (nrm(d, HD) * s).to(dt),
        "gamma": (1.0 + nrm(d) * wl.gamma_std).to(dt),
        "w_gate": (nrm(I, d) * s).to(dt),
        "w_up": (nrm(I, d) * s).to(dt),
        "w_down": (nrm(d, I) * s).to(dt),
    }
    perm = torch.randperm(d, generator=gen, device=device)
    out["outliers"] = torch.sort(perm[: wl.n_outliers]).values
    return out


def device_attn_weights(wl: Workload, layer: int, device) -> dict:
    """Same recipe as ``host_attn_weights`` with torch's generator on ``device``."""
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed(int(np.random.SeedSequence([SEED_ROOT, wl.key, layer, 0, 1]).generate_state(1)[0]))
    dt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    d, HD, GD = wl.d_model, wl.attn_width, wl.n_kv_groups * wl.head_dim
    s = wl.weight_std

    def nrm(*shape):
        return torch.randn(*shape, generator=gen, device=device, dtype=torch.float32)

    return {"w_q": (nrm(HD, d) * s).to(dt), "w_k": (nrm(GD, d) * s).to(dt),
            "w_v": (nrm(GD, d) * s).to(dt), "gamma": (1.0 + nrm(d) * wl.gamma_std).to(dt)}


def device_tokens(wl: Workload, layer: int, weights: dict, n_tokens: int, chunk: int, device,
                  with_pre: bool = False):
    """(x [T,d], attn [T,H,dh]) on ``device``, same recipe as ``host_tokens``."""
    import torch
    gen = torch.Generator(device=device)
    gen.manual_seed(int(np.random.SeedSequence([SEED_ROOT, wl.key, layer, 1, chunk]).generate_state(1)[0]))
    dt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    x_pre = torch.randn(n_tokens, wl.d_model, generator=gen, device=device, dtype=torch.float32)
    if wl.n_outliers:
        x_pre[:, weights["outliers"]] *= wl.outlier_scale
    shape = (n_tokens, wl.n_q_heads, wl.head_dim)
    if wl.heads_dist == "normal":
        z = torch.randn(*shape, generator=gen, device=device, dtype=torch.float32)
    else:
        # Student-t with 4 degrees of freedom: N(0,1) / sqrt(chi2_4 / 4), chi2_4 = -2 log(U1 U2)
        nrm = torch.randn(*shape, generator=gen, device=device, dtype=torch.float32)
        u = torch.rand(2, *shape, generator=gen, device=device, dtype=torch.float32).clamp_min_(1e-30)
        chi2 = -2.0 * torch.log(u[0] * u[1])
        z = nrm / torch.sqrt(chi2 / 4.0)
    z = z.to(dt)
    x = x_pre + (z.reshape(n_tokens, -1).float() @ weights["w_o"].float().t())
    if with_pre:
        return x.to(dt).contiguous(), z.contiguous(), x_pre.to(dt).contiguous()
    return x.to(dt).contiguous(), z.contiguous()

