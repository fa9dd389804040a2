"""fp64 CPU oracle for the first-order head-to-neuron affinity (test infrastructure only).

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this module.  It shares no code with the HIP library and
imports nothing from the product package; callers pass the same rounded input bytes
the GPU reads, upcast to fp64.

What is computed (Section 3, "Affinity scores"):

* x is the residual entering the FFN pre-norm, r = rms(x), gamma the norm gain;
* head h's piece of the normalised FFN input is p_h = gamma * (a_h W_o^(h)) / r;
* neuron k has pre-activations g_k = w^g_k . (gamma * x / r), u_k = w^u_k . (...);
* the first-order change of silu(g_k) u_k when head h's piece is removed is
  Delta_hk = silu'(g_k) u_k (p_h . w^g_k) + silu(g_k) (p_h . w^u_k)   (unnumbered eq.);
* the FO up score is E_t[Delta_hk^2] ||w^d_k||^2, summed over the query heads of
  each KV group.

Readings where the paper is silent (each listed in the design notes):

* r = sqrt(mean_j x_j^2 + eps), eps an input (the norm's epsilon is not given);
* silu'(g) = sigma(g) (1 + g (1 - sigma(g))), the derivative of g sigma(g);
* r, g and u are taken from the unmodified x (the FO score ignores the rms change);
* query head h belongs to KV group floor(h / (H/G)) (consecutive heads share a group);
* W_o is stored as ``o_proj.weight`` [d, H*dh], so a_h W_o^(h) = W_o[:, h*dh:(h+1)*dh] a_h;
* w^d_k is column k of W_down [d, I];
* the oracle returns the raw token sum A = sum_t (...) rather than the mean E_t; the
  1/T factor cancels in the unit-mass normalisation of the objective.

The ADD score of the same section, E_t[(p_h . w^g_k)^2 + (p_h . w^u_k)^2] summed over
the query heads of each KV group, ignores the operating point and the neuron's write
(no ||w^d_k||^2 factor): ``affinity_add_literal`` and ``affinity_add_folded``.

Two forms:

* ``affinity_literal`` materialises every p_h in model space, exactly as written;
* ``affinity_folded`` re-associates p_h . w_k = a_h (W_o^(h) diag(gamma) w_k) / r,
  which is the same quantity up to rounding order and affordable at full size.
"""
from __future__ import annotations

import numpy as np


def rms(x: np.ndarray, eps: float) -> np.ndarray:
    """r_t = sqrt(mean_j x_tj^2 + eps) for every row of x [T, d]."""
    return np.sqrt(np.mean(x * x, axis=1) + eps)


def sigmoid(g: np.ndarray) -> np.ndarray:
    return 1.0 / (1.0 + np.exp(-g))


def silu(g: np.ndarray) -> np.ndarray:
    return g * sigmoid(g)


def silu_prime(g: np.ndarray) -> np.ndarray:
    s = sigmoid(g)
    return s * (1.0 + g * (1.0 - s))


def group_of_head(n_q_heads: int, n_kv_groups: int) -> np.ndarray:
    """KV group of each query head: consecutive query heads share a group."""
    if n_q_heads % n_kv_groups:
        raise ValueError("H must be a multiple of G")
    return np.arange(n_q_heads) // (n_q_heads // n_kv_groups)


def operating_point(x, gamma, w_gate, w_up, eps):
    """(r [T], g [T,I], u [T,I]) at the unmodified residual x [T,d]."""
    r = rms(x, eps)
    n = gamma[None, :] * x / r[:, None]
    return r, n @ w_gate.T, n @ w_up.T


def head_pieces(x, attn, w_o, gamma, eps):
    """p_h = gamma * (a_h W_o^(h)) / r for every token and head: [T, H, d]."""
    T, H, dh = attn.shape
    r = rms(x, eps)
    out = np.empty((T, H, x.shape[1]))
    for h in range(H):
        out[:, h, :] = attn[:, h, :] @ w_o[:, h * dh:(h + 1) * dh].T
    return gamma[None, None, :] * out / r[:, None, None]


def damage_literal(x, attn, w_o, gamma, w_gate, w_up, eps):
    """Delta [T, H, I]: first-order change of silu(g_k) u_k when p_h is removed."""
    _, g, u = operating_point(x, gamma, w_gate, w_up, eps)
    p = head_pieces(x, attn, w_o, gamma, eps)
    pg = p @ w_gate.T          # p_h . w^g_k   [T, H, I]
    pu = p @ w_up.T            # p_h . w^u_k
    return silu_prime(g)[:, None, :] * u[:, None, :] * pg + silu(g)[:, None, :] * pu


def _aggregate(delta_sq_sum_per_head, w_down, n_kv_groups):
    """sum over the query heads of each group, times ||w^d_k||^2."""
    H = delta_sq_sum_per_head.shape[0]
    grp = group_of_head(H, n_kv_groups)
    A = np.zeros((n_kv_groups, delta_sq_sum_per_head.shape[1]))
    for h in range(H):
        A[grp[h]] += delta_sq_sum_per_head[h]
    col_norm_sq = np.sum(w_down * w_down, axis=0)   # ||column k of W_down||^2
    return A * col_norm_sq[None, :]


def affinity_literal(x, attn, w_o, gamma, w_gate, w_up, w_down, n_kv_groups, eps,
                     block: int = 128):
    """Raw FO up affinity A [G, I] (sum over tokens), materialising every p_h."""
    T, H, _ = attn.shape
    acc = np.zeros((H, w_gate.shape[0]))
    for t0 in range(0, T, block):
        sl = slice(t0, min(T, t0 + block))
        dlt = damage_literal(x[sl], attn[sl], w_o, gamma, w_gate, w_up, eps)
        acc += np.sum(dlt * dlt, axis=0)
    return _aggregate(acc, w_down, n_kv_groups)


def fold(w_o, gamma, w, n_q_heads):
    """F_h = W_o^(h) diag(gamma) w^T for every head: [H, dh, I] (w is [I, d])."""
    d, HD = w_o.shape
    dh = HD // n_q_heads
    wg = w * gamma[None, :]                       # [I, d]
    return np.stack([w_o[:, h * dh:(h + 1) * dh].T @ wg.T for h in range(n_q_heads)])


def affinity_folded(x, attn, w_o, gamma, w_gate, w_up, w_down, n_kv_groups, eps,
                    block: int = 1024, neurons=None):
    """Raw FO up affinity A [G, I] via the fold; ``neurons`` restricts the columns."""
    T, H, _ = attn.shape
    if neurons is not None:
        neurons = np.asarray(neurons)
        w_gate, w_up, w_down = w_gate[neurons], w_up[neurons], w_down[:, neurons]
    fg = fold(w_o, gamma, w_gate, H)
    fu = fold(w_o, gamma, w_up, H)
    acc = np.zeros((H, w_gate.shape[0]))
    for t0 in range(0, T, block):
        sl = slice(t0, min(T, t0 + block))
        r, g, u = operating_point(x[sl], gamma, w_gate, w_up, eps)
        c1 = silu_prime(g) * u / r[:, None]
        c2 = silu(g) / r[:, None]
        for h in range(H):
            dlt = c1 * (attn[sl, h, :] @ fg[h]) + c2 * (attn[sl, h, :] @ fu[h])
            acc[h] += np.sum(dlt * dlt, axis=0)
    return _aggregate(acc, w_down, n_kv_groups)



def _group_sum(per_head, n_kv_groups):
    """sum over the query heads of each group: [H, I] -> [G, I]."""
    grp = group_of_head(per_head.shape[0], n_kv_groups)
    out = np.zeros((n_kv_groups, per_head.shape[1]))
    for h in range(per_head.shape[0]):
        out[grp[h]] += per_head[h]
    return out


def affinity_add_literal(x, attn, w_o, gamma, w_gate, w_up, n_kv_groups, eps, block: int = 128):
    """Raw ADD up affinity [G, I]: sum_t (p_h . w^g_k)^2 + (p_h . w^u_k)^2 per group."""
    T, H, _ = attn.shape
    acc = np.zeros((H, w_gate.shape[0]))
    for t0 in range(0, T, block):
        sl = slice(t0, min(T, t0 + block))
        p = head_pieces(x[sl], attn[sl], w_o, gamma, eps)
        acc += np.sum((p @ w_gate.T) ** 2 + (p @ w_up.T) ** 2, axis=0)
    return _group_sum(acc, n_kv_groups)


def affinity_add_folded(x, attn, w_o, gamma, w_gate, w_up, n_kv_groups, eps, block: int = 1024,
                        neurons=None):
    """Raw ADD up affinity via the fold; ``neurons`` restricts the columns."""
    T, H, _ = attn.shape
    if neurons is not None:
        neurons = np.asarray(neurons)
        w_gate, w_up = w_gate[neurons], w_up[neurons]
    fg = fold(w_o, gamma, w_gate, H)
    fu = fold(w_o, gamma, w_up, H)
    acc = np.zeros((H, w_gate.shape[0]))
    for t0 in range(0, T, block):
        sl = slice(t0, min(T, t0 + block))
        r = rms(x[sl], eps)[:, None]
        for h in range(H):
            acc[h] += np.sum((attn[sl, h, :] @ fg[h] / r) ** 2 + (attn[sl, h, :] @ fu[h] / r) ** 2, axis=0)
    return _group_sum(acc, n_kv_groups)
