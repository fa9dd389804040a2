"""Pins of the fp64 down-edge oracle against what the paper and the mathematics fix.

Section 3 defines S_down[k, g] as the mean squared effect of neuron k's residual write
alpha_k w^d_k on the q/k/v projections of KV group g of the next layer, through that
layer's pre-norm (gain gamma', rms r' held fixed).  The pins:

* the effect computed by removing the write from the next layer's residual and
  projecting both residuals with torch (heads split by reshaping, not by row indices);
* a closed form: one group whose projection is the identity gives ||w^d_k||^2;
* invariances the definition implies (column scale of W_down, scale of W_up, scale of
  the next residual with eps' = 0, neuron and group permutations, token additivity);
* the factorised form against the token-by-token one.
"""
import numpy as np
import pytest
import torch

from oracle import down as orc
from paper_2609_13846_amd import synth

TINY = synth.shaped(synth.WORKLOADS["tiny"], tokens=24)


def _data(wl=TINY, T=None):
    f = synth.to_f64
    w = synth.host_weights(wl, 0)
    x, _, _ = synth.host_tokens(wl, 0, w, T or wl.tokens, with_pre=True)
    wn = synth.host_weights(wl, 1)
    _, _, x_next = synth.host_tokens(wl, 1, wn, T or wl.tokens, with_pre=True)
    an = synth.host_attn_weights(wl, 1)
    return dict(x=f(x), gamma=f(w.gamma), w_gate=f(w.w_gate), w_up=f(w.w_up), eps=wl.rms_eps,
                x_next=f(x_next), eps_next=wl.rms_eps, w_q=f(an.w_q), w_k=f(an.w_k),
                w_v=f(an.w_v), gamma_next=f(an.gamma), w_down=f(w.w_down),
                n_q_heads=wl.n_q_heads, n_kv_groups=wl.n_kv_groups)


def _S(d, **over):
    kw = dict(d)
    kw.update(over)
    return orc.down_affinity(**kw)


@pytest.fixture(scope="module")
def tiny():
    return _data()


def _removal_effect(d):
    """sum_t ||qkv_g(x') - qkv_g(x' - alpha_k w^d_k)||^2 with r' frozen, via torch."""
    t = {k: torch.tensor(v) for k, v in d.items() if isinstance(v, np.ndarray)}
    H, G = d["n_q_heads"], d["n_kv_groups"]
    dh = t["w_k"].shape[0] // G
    x = t["x"]
    r = torch.sqrt(torch.mean(x * x, dim=1, keepdim=True) + d["eps"])
    n = t["gamma"] * x / r
    alpha = torch.nn.functional.silu(n @ t["w_gate"].T) * (n @ t["w_up"].T)     # [T, I]
    xn = t["x_next"]
    rn = torch.sqrt(torch.mean(xn * xn, dim=1, keepdim=True) + d["eps_next"])  # frozen

    def qkv(resid):
        nn = t["gamma_next"] * resid / rn
        q = (nn @ t["w_q"].T).reshape(-1, G, H // G, dh).reshape(-1, G, (H // G) * dh)
        k = (nn @ t["w_k"].T).reshape(-1, G, dh)
        v = (nn @ t["w_v"].T).reshape(-1, G, dh)
        return torch.cat([q, k, v], dim=2)                                     # [T, G, rows]

    base = qkv(xn)
    I = alpha.shape[1]
    out = np.zeros((I, G))
    for kk in range(I):
        removed = xn - alpha[:, kk:kk + 1] * t["w_down"][:, kk][None, :]
        diff = base - qkv(removed)
        out[kk] = (diff * diff).sum(dim=(0, 2)).numpy()
    return out


def test_equals_removal_through_next_projection(tiny):
    np.testing.assert_allclose(_S(tiny), _removal_effect(tiny), rtol=1e-9)


def test_factorised_equals_token_by_token(tiny):
    np.testing.assert_allclose(orc.down_affinity(**tiny), orc.down_affinity_literal(**tiny),
                               rtol=1e-12)


def test_identity_projection_gives_column_norm(tiny):
    """One group, one head with dh = d, q_proj = I, k = v = 0, gamma' = 1:
    b_k = w^d_k, so S[k] = sum_t alpha_k^2 / r'^2 * ||w^d_k||^2."""
    d = tiny["x"].shape[1]
    eye = np.eye(d)
    zero = np.zeros((d, d))
    S = _S(tiny, w_q=eye, w_k=zero, w_v=zero, gamma_next=np.ones(d), n_q_heads=1, n_kv_groups=1)
    t = {k: torch.tensor(v) for k, v in tiny.items() if isinstance(v, np.ndarray)}
    r = torch.sqrt(torch.mean(t["x"] ** 2, dim=1, keepdim=True) + tiny["eps"])
    n = t["gamma"] * t["x"] / r
    alpha = torch.nn.functional.silu(n @ t["w_gate"].T) * (n @ t["w_up"].T)
    rn = torch.sqrt(torch.mean(t["x_next"] ** 2, dim=1, keepdim=True) + tiny["eps_next"])
    ref = ((alpha / rn) ** 2).sum(0) * (t["w_down"] ** 2).sum(0)
    np.testing.assert_allclose(S[:, 0], ref.numpy(), rtol=1e-12)


def test_down_column_scale(tiny):
    k, c = 5, 3.0
    wd = tiny["w_down"].copy()
    wd[:, k] *= c
    S0, S1 = _S(tiny), _S(tiny, w_down=wd)
    np.testing.assert_allclose(S1[k], c * c * S0[k], rtol=1e-12)
    np.testing.assert_array_equal(np.delete(S1, k, axis=0), np.delete(S0, k, axis=0))


def test_up_scale_scales_activation(tiny):
    np.testing.assert_allclose(_S(tiny, w_up=2.0 * tiny["w_up"]), 4.0 * _S(tiny), rtol=1e-12)


def test_next_residual_scale_without_eps(tiny):
    S0 = _S(tiny, eps_next=0.0)
    S1 = _S(tiny, eps_next=0.0, x_next=4.0 * tiny["x_next"])
    np.testing.assert_allclose(S1, S0 / 16.0, rtol=1e-12)


def test_neuron_permutation_permutes_rows(tiny):
    I = tiny["w_gate"].shape[0]
    perm = np.random.default_rng(1).permutation(I)
    S0 = _S(tiny)
    S1 = _S(tiny, w_gate=tiny["w_gate"][perm], w_up=tiny["w_up"][perm], w_down=tiny["w_down"][:, perm])
    np.testing.assert_allclose(S1, S0[perm], rtol=1e-12)


def test_next_group_permutation_permutes_columns(tiny):
    H, G = tiny["n_q_heads"], tiny["n_kv_groups"]
    dh = tiny["w_k"].shape[0] // G
    hpg = H // G
    gperm = np.array([3, 1, 0, 2])
    q_rows = np.concatenate([np.arange(g * hpg * dh, (g + 1) * hpg * dh) for g in gperm])
    kv_rows = np.concatenate([np.arange(g * dh, (g + 1) * dh) for g in gperm])
    S0 = _S(tiny)
    S1 = _S(tiny, w_q=tiny["w_q"][q_rows], w_k=tiny["w_k"][kv_rows], w_v=tiny["w_v"][kv_rows])
    np.testing.assert_allclose(S1, S0[:, gperm], rtol=1e-12)


def test_token_chunks_add(tiny):
    S = _S(tiny)
    parts = [_S(tiny, x=tiny["x"][q], x_next=tiny["x_next"][q]) for q in (slice(0, 10), slice(10, None))]
    np.testing.assert_allclose(parts[0] + parts[1], S, rtol=1e-12)


def test_silent_neuron_has_no_down_edge(tiny):
    """A neuron whose up row is zero never activates (u = 0), so its row is zero."""
    wu = tiny["w_up"].copy()
    wu[7] = 0.0
    S = _S(tiny, w_up=wu)
    assert np.all(S[7] == 0.0) and np.all(np.delete(S, 7, axis=0) > 0.0)
