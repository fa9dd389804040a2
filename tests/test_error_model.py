"""Pins of the rounding-error model used by the GPU parity tests (tests/error_model.py).

The model must (a) contain every rounding it names: an fp64 emulation that applies
exactly those roundings (bf16 W' and F_h, fp16 damage coefficients; bf16 gamma' * w^d on
the down edge) stays inside the bound on every entry, and (b) not be vacuous: measured in
units of the predicted sigma, the emulated errors have an rms of order one.  The
derivatives of silu it uses are checked against finite differences.  The emulation is
only a check of the model; the GPU tests compare the library with the exact oracle.
"""
import numpy as np
import pytest

from oracle import affinity as orc
from oracle import down as dwn
from paper_2609_13846_amd import synth
from tests import error_model as em


def _bf16(v):
    return synth.bf16_bits_to_f64(synth.round_to_bf16_bits(np.asarray(v, np.float32)))


def _fp16(v):
    m, e = np.frexp(v)
    return np.ldexp(np.round(m * 2.0 ** 11) / 2.0 ** 11, e)


def test_silu_derivatives_match_finite_differences():
    g = np.linspace(-12, 12, 97)
    h = 1e-5
    sl, d1, d2, d3 = em._silu_derivatives(g)
    f = lambda v: em._silu_derivatives(v)
    assert np.allclose(sl, orc.silu(g))
    assert np.allclose(d1, (orc.silu(g + h) - orc.silu(g - h)) / (2 * h), atol=1e-8)
    assert np.allclose(d2, (f(g + h)[1] - f(g - h)[1]) / (2 * h), atol=1e-8)
    assert np.allclose(d3, (f(g + h)[2] - f(g - h)[2]) / (2 * h), atol=1e-8)


def _emulated_up(x, attn, w_o, gamma, w_gate, w_up, w_down, G, eps):
    T, H, dh = attn.shape
    r = orc.rms(x, eps)
    Wg, Wu = _bf16(w_gate * gamma[None, :]), _bf16(w_up * gamma[None, :])
    g, u = (x @ Wg.T) / r[:, None], (x @ Wu.T) / r[:, None]
    c1 = _fp16(orc.silu_prime(g) * u / r[:, None])
    c2 = _fp16(orc.silu(g) / r[:, None])
    acc = np.zeros((H, w_gate.shape[0]))
    for h in range(H):
        Wo = w_o[:, h * dh:(h + 1) * dh]
        Fg, Fu = _bf16(Wo.T @ Wg.T), _bf16(Wo.T @ Wu.T)
        D = c1 * (attn[:, h] @ Fg) + c2 * (attn[:, h] @ Fu)
        acc[h] = np.sum(D * D, axis=0)
    return orc._aggregate(acc, w_down, G)


@pytest.mark.parametrize("name,T", [("qwen3-0.6b-layer", 1), ("qwen3-0.6b-layer", 5), ("danube3-500m", 2)])
def test_up_model_bounds_the_emulated_rounding(name, T):
    wl = synth.shaped(synth.WORKLOADS[name], n_neurons=384)
    w = synth.host_weights(wl, 0)
    x, a = synth.host_tokens(wl, 0, w, T)
    f = synth.to_f64
    args = (f(x), f(a), f(w.w_o), f(w.gamma), f(w.w_gate), f(w.w_up), f(w.w_down), wl.n_kv_groups,
            wl.rms_eps)
    A, sig, sec = em.up_affinity_error(*args)
    A_ref = orc.affinity_folded(*args)
    np.testing.assert_allclose(A, A_ref, rtol=1e-10)
    A_emu = _emulated_up(*args)
    em.check_entrywise(A_emu, A, sig, sec, label="emulated up")
    big = A > 1e-3 * A.max()
    z = (A_emu - A)[big] / sig[big]
    assert 0.2 < np.sqrt(np.mean(z * z)) < 1.5, np.sqrt(np.mean(z * z))


def test_down_models_bound_the_emulated_rounding():
    wl = synth.shaped(synth.WORKLOADS["qwen3-0.6b-layer"], n_neurons=512)
    w = synth.host_weights(wl, 0)
    x, a, _ = synth.host_tokens(wl, 0, w, 40, with_pre=True)
    wn = synth.host_weights(wl, 1)
    _, _, x_next = synth.host_tokens(wl, 1, wn, 40, with_pre=True)
    an = synth.host_attn_weights(wl, 1)
    f = synth.to_f64
    X, Xn, gam = f(x), f(x_next), f(w.gamma)
    s, sig, sec = em.down_stat_error(X, gam, f(w.w_gate), f(w.w_up), wl.rms_eps, Xn, wl.rms_eps)
    np.testing.assert_allclose(s, dwn.down_token_stat(X, gam, f(w.w_gate), f(w.w_up), wl.rms_eps, Xn,
                                                      wl.rms_eps), rtol=1e-10)
    r, rn = orc.rms(X, wl.rms_eps), orc.rms(Xn, wl.rms_eps)
    Wg, Wu = _bf16(f(w.w_gate) * gam), _bf16(f(w.w_up) * gam)
    g, u = X @ Wg.T / r[:, None], X @ Wu.T / r[:, None]
    s_emu = np.sum((orc.silu(g) * u / rn[:, None]) ** 2, axis=0)
    em.check_entrywise(s_emu[None], s[None], sig[None], sec[None], label="emulated s_down")
    z = (s_emu - s) / sig
    assert 0.2 < np.sqrt(np.mean(z * z)) < 1.5

    args = (f(an.w_q), f(an.w_k), f(an.w_v), f(an.gamma), f(w.w_down), wl.n_q_heads, wl.n_kv_groups)
    B, bsig, bsec = em.down_weight_error(*args)
    np.testing.assert_allclose(B, dwn.down_weight_norms(*args), rtol=1e-10)
    m = _bf16(f(an.gamma)[:, None] * f(w.w_down))
    B_emu = np.stack([np.sum((dwn.group_projection(*args[:3], wl.n_q_heads, wl.n_kv_groups, g) @ m) ** 2, axis=0)
                      for g in range(wl.n_kv_groups)])
    em.check_entrywise(B_emu, B, bsig, bsec, label="emulated B")
    z = (B_emu - B) / bsig
    assert 0.2 < np.sqrt(np.mean(z * z)) < 1.5
