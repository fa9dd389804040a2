"""Pins of the layout-application oracle (Section 3, "The layout as a free variable").

* the permuted layer computes the same function (fp64 decoder layer with GQA attention,
  per-head q/k norms, rotary embedding and a SwiGLU FFN), as the paper states;
* device l's contiguous shard holds exactly the groups (with their query heads) and the
  neurons that the layout puts on l, in increasing original index (built by explicit
  loops here);
* the contiguous layout changes nothing; an inconsistent permutation breaks invariance.
"""
import numpy as np
import pytest

from oracle import apply as ap
from oracle import layout as lay
from paper_2609_13846_amd import synth

WL = synth.shaped(synth.WORKLOADS["tiny"], n_neurons=64)


def layer_weights(wl=WL, seed=0):
    f = synth.to_f64
    w = synth.host_weights(wl, 0)
    an = synth.host_attn_weights(wl, 0)
    rng = np.random.default_rng(seed)
    return {"w_q": f(an.w_q), "w_k": f(an.w_k), "w_v": f(an.w_v), "w_o": f(w.w_o),
            "gamma_attn": f(an.gamma), "q_norm": 1.0 + 0.1 * rng.standard_normal(wl.head_dim),
            "k_norm": 1.0 + 0.1 * rng.standard_normal(wl.head_dim), "gamma": f(w.gamma),
            "w_gate": f(w.w_gate), "w_up": f(w.w_up), "w_down": f(w.w_down)}


def tokens(wl=WL, T=12):
    return np.random.default_rng(3).standard_normal((T, wl.d_model))


def _fwd(w, x, wl=WL):
    return ap.decoder_layer(x, w, wl.n_q_heads, wl.n_kv_groups, wl.head_dim, wl.rms_eps)


@pytest.mark.parametrize("L,seed", [(2, 1000), (4, 1001), (2, 7)])
def test_permuted_layer_computes_the_same_function(L, seed):
    w = layer_weights()
    x = tokens()
    hs, nus = lay.random_layout(1, WL.n_kv_groups, WL.n_neurons, L, seed)
    wp = ap.apply_layout(w, hs[0], nus[0], WL.n_q_heads, WL.n_kv_groups, WL.head_dim, L)
    y0, y1 = _fwd(w, x), _fwd(wp, x)
    np.testing.assert_allclose(y1, y0, rtol=1e-12, atol=1e-12 * np.abs(y0).max())
    assert not np.array_equal(wp["w_q"], w["w_q"])


def test_shards_hold_the_assigned_groups_and_neurons():
    w = layer_weights()
    H, G, dh, I, L = WL.n_q_heads, WL.n_kv_groups, WL.head_dim, WL.n_neurons, 2
    h = np.array([1, 0, 1, 0])
    nu = np.array([(k * 7) % 2 for k in range(I)])
    wp = ap.apply_layout(w, h, nu, H, G, dh, L)
    hpg = H // G
    pos = 0
    for l in range(L):
        for g in range(G):
            if h[g] != l:
                continue
            for hh in range(hpg):
                src = (g * hpg + hh) * dh
                dst = (pos * hpg + hh) * dh
                np.testing.assert_array_equal(wp["w_q"][dst:dst + dh], w["w_q"][src:src + dh])
                np.testing.assert_array_equal(wp["w_o"][:, dst:dst + dh], w["w_o"][:, src:src + dh])
            np.testing.assert_array_equal(wp["w_k"][pos * dh:(pos + 1) * dh], w["w_k"][g * dh:(g + 1) * dh])
            np.testing.assert_array_equal(wp["w_v"][pos * dh:(pos + 1) * dh], w["w_v"][g * dh:(g + 1) * dh])
            pos += 1
    pos = 0
    for l in range(L):
        for k in range(I):
            if nu[k] == l:
                np.testing.assert_array_equal(wp["w_gate"][pos], w["w_gate"][k])
                np.testing.assert_array_equal(wp["w_up"][pos], w["w_up"][k])
                np.testing.assert_array_equal(wp["w_down"][:, pos], w["w_down"][:, k])
                pos += 1


def test_contiguous_layout_changes_nothing():
    w = layer_weights()
    h = np.array(lay.contiguous_heads(WL.n_kv_groups, 2))
    nu = lay.contiguous_neurons(WL.n_neurons, 2)
    wp = ap.apply_layout(w, h, nu, WL.n_q_heads, WL.n_kv_groups, WL.head_dim, 2)
    for k in w:
        np.testing.assert_array_equal(wp[k], w[k])


def test_inconsistent_permutation_changes_the_function():
    """Moving the q rows without the o columns (or gate rows without down columns) is
    not a symmetry: the invariance test above would catch either mistake."""
    w = layer_weights()
    x = tokens()
    hs, nus = lay.random_layout(1, WL.n_kv_groups, WL.n_neurons, 2, 5)
    wp = ap.apply_layout(w, hs[0], nus[0], WL.n_q_heads, WL.n_kv_groups, WL.head_dim, 2)
    bad = dict(wp, w_o=w["w_o"])
    assert np.abs(_fwd(bad, x) - _fwd(w, x)).max() > 1e-3
    bad = dict(wp, w_down=w["w_down"])
    assert np.abs(_fwd(bad, x) - _fwd(w, x)).max() > 1e-3


def test_single_token_attention_returns_its_value():
    """T = 1: softmax over one position is 1, so the attention output is v of the group."""
    w = layer_weights()
    x = tokens(T=1)
    H, G, dh = WL.n_q_heads, WL.n_kv_groups, WL.head_dim
    n = w["gamma_attn"] * x / np.sqrt(np.mean(x * x) + WL.rms_eps)
    v = (n @ w["w_v"].T).reshape(G, dh)
    heads = np.concatenate([v[hh // (H // G)] for hh in range(H)])[None, :]
    x1 = x + heads @ w["w_o"].T
    n2 = w["gamma"] * x1 / np.sqrt(np.mean(x1 * x1) + WL.rms_eps)
    gg = n2 @ w["w_gate"].T
    ref = x1 + (gg / (1 + np.exp(-gg)) * (n2 @ w["w_up"].T)) @ w["w_down"].T
    np.testing.assert_allclose(_fwd(w, x), ref, rtol=1e-12)
