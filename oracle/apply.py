"""CPU oracle for applying a layout to a decoder layer's weights (test infrastructure only).

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s ``cpu_baseline`` leg may
import this module.  It shares no code with the HIP library.

Section 3, "The layout as a free variable": the layout (h_i, nu_i) of a layer becomes an
ordering of its KV groups and of its neurons (device 0's in increasing original index,
then device 1's, ...).  Every weight indexed by a group (the query rows of its query
heads, its key and value rows, the matching output-projection columns) and every weight
indexed by a neuron (gate and up rows, down-projection columns) is reordered with it, so
each device's shard is a contiguous slice.  Rotary embeddings, per-head norms and the
SwiGLU product work head by head or neuron by neuron, which is why the reordered layer
computes the same function.

Reading (listed in the design notes): device l's shard holds its groups and neurons in
increasing original index, and the shards follow each other in device order.
"""
from __future__ import annotations

import numpy as np


def layout_orders(h, nu, L: int):
    """(group_order [G], neuron_order [I]): new position -> original index."""
    h = np.asarray(h)
    nu = np.asarray(nu)
    group_order = np.concatenate([np.flatnonzero(h == l) for l in range(L)])
    neuron_order = np.concatenate([np.flatnonzero(nu == l) for l in range(L)])
    return group_order, neuron_order


def _blocks(order, size):
    """Row (or column) indices of whole blocks of `size` taken in `order`."""
    return np.concatenate([np.arange(b * size, (b + 1) * size) for b in order])


def apply_layout(w: dict, h, nu, n_q_heads: int, n_kv_groups: int, head_dim: int, L: int) -> dict:
    """Permuted copies of w_q [H*dh, d], w_k / w_v [G*dh, d], w_o [d, H*dh],
    w_gate / w_up [I, d], w_down [d, I]; other entries are copied unchanged."""
    go, no = layout_orders(h, nu, L)
    hpg = n_q_heads // n_kv_groups
    q_rows = _blocks(go, hpg * head_dim)   # a group's query heads are consecutive rows
    kv_rows = _blocks(go, head_dim)
    out = dict(w)
    out["w_q"] = w["w_q"][q_rows]
    out["w_k"] = w["w_k"][kv_rows]
    out["w_v"] = w["w_v"][kv_rows]
    out["w_o"] = w["w_o"][:, q_rows]
    out["w_gate"] = w["w_gate"][no]
    out["w_up"] = w["w_up"][no]
    out["w_down"] = w["w_down"][:, no]
    return out


def _rms_norm(x, gain, eps):
    return gain * x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)


def _rope(x, base=10000.0):
    """Rotary embedding on [T, heads, dh] (pairs (j, j + dh/2), position = row index)."""
    T, _, dh = x.shape
    half = dh // 2
    inv = base ** (-np.arange(half) / half)
    ang = np.arange(T)[:, None] * inv[None, :]
    c, s = np.cos(ang)[:, None, :], np.sin(ang)[:, None, :]
    a, b = x[..., :half], x[..., half:]
    return np.concatenate([a * c - b * s, a * s + b * c], axis=-1)


def decoder_layer(x, w: dict, n_q_heads: int, n_kv_groups: int, head_dim: int, eps: float):
    """One pre-norm decoder layer in fp64: GQA attention with per-head q/k norms and rotary
    embedding under a causal mask, then a SwiGLU FFN; both with residuals.  x [T, d]."""
    T, _ = x.shape
    H, G, dh = n_q_heads, n_kv_groups, head_dim
    n = _rms_norm(x, w["gamma_attn"], eps)
    q = (n @ w["w_q"].T).reshape(T, H, dh)
    k = (n @ w["w_k"].T).reshape(T, G, dh)
    v = (n @ w["w_v"].T).reshape(T, G, dh)
    q = _rope(_rms_norm(q, w["q_norm"], eps))
    k = _rope(_rms_norm(k, w["k_norm"], eps))
    mask = np.triu(np.full((T, T), -np.inf), 1)
    heads = np.empty((T, H, dh))
    for hh in range(H):
        g = hh // (H // G)
        s = q[:, hh, :] @ k[:, g, :].T / np.sqrt(dh) + mask
        p = np.exp(s - s.max(axis=1, keepdims=True))
        p /= p.sum(axis=1, keepdims=True)
        heads[:, hh, :] = p @ v[:, g, :]
    x1 = x + heads.reshape(T, H * dh) @ w["w_o"].T
    n2 = _rms_norm(x1, w["gamma"], eps)
    g_ = n2 @ w["w_gate"].T
    act = g_ / (1.0 + np.exp(-g_)) * (n2 @ w["w_up"].T)
    return x1 + act @ w["w_down"].T
