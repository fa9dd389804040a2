"""fp64 CPU oracle for the down-edge affinity S_down (test infrastructure only).

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this module.  It shares no code with the HIP library.

What is computed (Section 3, "Affinity scores", down edge):

* neuron k of layer i writes alpha_k w^d_k into the residual stream, with
  alpha_k = silu(g_k) u_k its activation at the layer's operating point and w^d_k column
  k of W_down [d, I];
* that write reaches the q/k/v projections of KV group g of layer i+1 through the
  attention pre-norm of layer i+1 (gain gamma', rms r' of the residual entering it) as
  (alpha_k / r') b_gk with b_gk = W^{qkv}_g (gamma' * w^d_k);
* S_down[k, g] = E_t[alpha_k^2 / r'^2] ||b_gk||^2.

Readings where the paper is silent (each listed in the design notes):

* W^{qkv}_g stacks the q rows of group g's query heads, then its k rows and its v rows
  (``q_proj``/``k_proj``/``v_proj`` weight layouts; consecutive query heads share a
  group, as on the up edge);
* r' = sqrt(mean_j x'_j^2 + eps') with x' the residual entering layer i+1's attention
  pre-norm and eps' an input; r' is held fixed (as r is on the up edge);
* the raw token sum replaces E_t, as for S_up.

Two forms: ``down_affinity_literal`` pushes every neuron's write through the next
layer's projection token by token; ``down_affinity`` uses the factorisation above
(a token statistic times a weight-only norm), which is what makes full sizes affordable.
"""
from __future__ import annotations

import numpy as np

from oracle.affinity import operating_point, rms, silu


def qkv_rows(n_q_heads: int, n_kv_groups: int, head_dim: int, g: int):
    """Row indices of group g in q_proj.weight and in k_proj/v_proj.weight."""
    if n_q_heads % n_kv_groups:
        raise ValueError("H must be a multiple of G")
    hpg = n_q_heads // n_kv_groups
    q = np.arange(g * hpg * head_dim, (g + 1) * hpg * head_dim)
    kv = np.arange(g * head_dim, (g + 1) * head_dim)
    return q, kv


def group_projection(w_q, w_k, w_v, n_q_heads, n_kv_groups, g):
    """W^{qkv}_g: the stacked q, k and v rows of KV group g, [(H/G + 2) dh, d]."""
    head_dim = w_k.shape[0] // n_kv_groups
    q, kv = qkv_rows(n_q_heads, n_kv_groups, head_dim, g)
    return np.concatenate([w_q[q], w_k[kv], w_v[kv]], axis=0)


def activations(x, gamma, w_gate, w_up, eps):
    """alpha [T, I] = silu(g) u at the unmodified residual x."""
    _, g, u = operating_point(x, gamma, w_gate, w_up, eps)
    return silu(g) * u


def down_token_stat(x, gamma, w_gate, w_up, eps, x_next, eps_next):
    """s[k] = sum_t alpha_k(t)^2 / r'_t^2."""
    alpha = activations(x, gamma, w_gate, w_up, eps)
    r_next = rms(x_next, eps_next)
    return np.sum((alpha / r_next[:, None]) ** 2, axis=0)


def down_weight_norms(w_q, w_k, w_v, gamma_next, w_down, n_q_heads, n_kv_groups):
    """B[g, k] = ||W^{qkv}_g (gamma' * w^d_k)||^2, [G, I]."""
    m = gamma_next[:, None] * w_down  # [d, I]: gamma' * w^d_k in column k
    out = np.empty((n_kv_groups, w_down.shape[1]))
    for g in range(n_kv_groups):
        b = group_projection(w_q, w_k, w_v, n_q_heads, n_kv_groups, g) @ m
        out[g] = np.sum(b * b, axis=0)
    return out


def down_affinity(x, gamma, w_gate, w_up, eps, x_next, eps_next, w_q, w_k, w_v, gamma_next,
                  w_down, n_q_heads, n_kv_groups):
    """S_down [I, G] = s[k] B[g, k] (raw token sum)."""
    s = down_token_stat(x, gamma, w_gate, w_up, eps, x_next, eps_next)
    B = down_weight_norms(w_q, w_k, w_v, gamma_next, w_down, n_q_heads, n_kv_groups)
    return s[:, None] * B.T


def down_affinity_literal(x, gamma, w_gate, w_up, eps, x_next, eps_next, w_q, w_k, w_v,
                          gamma_next, w_down, n_q_heads, n_kv_groups):
    """The same quantity token by token: the residual change of neuron k's write, through
    the frozen pre-norm and group g's projection, squared and summed over tokens."""
    alpha = activations(x, gamma, w_gate, w_up, eps)
    r_next = rms(x_next, eps_next)
    T, I = alpha.shape
    out = np.zeros((I, n_kv_groups))
    for g in range(n_kv_groups):
        wg = group_projection(w_q, w_k, w_v, n_q_heads, n_kv_groups, g)
        for t in range(T):
            write = w_down * alpha[t][None, :]              # [d, I]: column k = alpha_k w^d_k
            normed = gamma_next[:, None] * write / r_next[t]
            contrib = wg @ normed                            # [(H/G+2) dh, I]
            out[:, g] += np.sum(contrib * contrib, axis=0)
    return out
