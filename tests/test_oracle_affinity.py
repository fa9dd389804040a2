"""Pins of the fp64 affinity oracle against what the paper and the mathematics fix.

Section 3 ("Affinity scores") defines Delta_hk as the first-order change of neuron k's
output silu(g_k) u_k when head h's piece p_h of the normalised FFN input is removed,
with the rms held fixed.  That is a directional derivative, so the pins are:

* torch autograd's JVP of n -> silu(W_g n) * (W_u n) along p_h (a library routine,
  computed independently of the oracle's closed form);
* forward differences of the same map converging at first order (central: second);
* invariances the definition implies (head scale, head removal, W_down column scale,
  joint scale of x and a, permutations of groups and neurons, token additivity);
* the folded form against the literal one.
"""
import numpy as np
import pytest
import torch

from oracle import affinity as orc
from paper_2609_13846_amd import synth

TINY = synth.shaped(synth.WORKLOADS["tiny"], tokens=48)


def _data(wl=TINY, T=None, layer=0):
    w = synth.host_weights(wl, layer)
    x, a = synth.host_tokens(wl, layer, w, T or wl.tokens)
    f = synth.to_f64
    return dict(x=f(x), attn=f(a), w_o=f(w.w_o), gamma=f(w.gamma), w_gate=f(w.w_gate),
                w_up=f(w.w_up), w_down=f(w.w_down), n_kv_groups=wl.n_kv_groups, eps=wl.rms_eps)


def _A(d, **over):
    kw = dict(d)
    kw.update(over)
    return orc.affinity_literal(**kw)


@pytest.fixture(scope="module")
def tiny():
    return _data()


def _jvp_damage(d, t, h):
    """torch.func.jvp of the neuron outputs along p_h at token t (fp64, rms frozen)."""
    x = torch.tensor(d["x"][t])
    gam = torch.tensor(d["gamma"])
    wg = torch.tensor(d["w_gate"])
    wu = torch.tensor(d["w_up"])
    dh = d["attn"].shape[2]
    r = torch.sqrt(torch.mean(x * x) + d["eps"])
    n = gam * x / r
    a_h = torch.tensor(d["attn"][t, h])
    wo_h = torch.tensor(d["w_o"][:, h * dh:(h + 1) * dh])
    p = gam * (wo_h @ a_h) / r

    def neuron_out(v):
        return torch.nn.functional.silu(wg @ v) * (wu @ v)

    _, tangent = torch.func.jvp(neuron_out, (n,), (p,))
    return tangent.numpy(), neuron_out, n, p


def test_damage_equals_autograd_jvp(tiny):
    dlt = orc.damage_literal(tiny["x"], tiny["attn"], tiny["w_o"], tiny["gamma"],
                             tiny["w_gate"], tiny["w_up"], tiny["eps"])
    T, H, I = dlt.shape
    for t in range(0, T, 7):
        for h in range(H):
            ref, *_ = _jvp_damage(tiny, t, h)
            np.testing.assert_allclose(dlt[t, h], ref, rtol=1e-11, atol=1e-14 * np.abs(ref).max())


def test_forward_difference_converges_first_order(tiny):
    """(y(n) - y(n - eps p_h)) / eps -> Delta with error O(eps); central difference O(eps^2)."""
    dlt = orc.damage_literal(tiny["x"], tiny["attn"], tiny["w_o"], tiny["gamma"],
                             tiny["w_gate"], tiny["w_up"], tiny["eps"])
    t, h = 5, 3
    _, f, n, p = _jvp_damage(tiny, t, h)
    ref = dlt[t, h]
    errs, cerrs = [], []
    for e in [1e-1, 1e-2, 1e-3, 1e-4]:
        fd = ((f(n) - f(n - e * p)) / e).numpy()
        cd = ((f(n + e * p) - f(n - e * p)) / (2 * e)).numpy()
        errs.append(np.linalg.norm(fd - ref))
        cerrs.append(np.linalg.norm(cd - ref))
    slopes = np.diff(np.log10(errs))
    assert np.all(np.abs(slopes + 1.0) < 0.1), slopes           # first order
    cslopes = np.diff(np.log10(cerrs[:3]))
    assert np.all(np.abs(cslopes + 2.0) < 0.2), cslopes         # second order
    assert errs[-1] < 1e-3 * np.linalg.norm(ref)


def test_rms_change_is_second_effect(tiny):
    """Removing eps*(a_h W_o) from x itself (rms recomputed) has a different first-order
    limit than Delta: the FO score deliberately ignores the rms change.  The gap is
    recorded, not bounded, except that it must be finite and smaller than Delta."""
    t, h = 3, 1
    dh = tiny["attn"].shape[2]
    x = tiny["x"][t:t + 1]
    head_out = tiny["attn"][t, h] @ tiny["w_o"][:, h * dh:(h + 1) * dh].T
    e = 1e-6

    def y(xx):
        _, g, u = orc.operating_point(xx, tiny["gamma"], tiny["w_gate"], tiny["w_up"], tiny["eps"])
        return orc.silu(g) * u

    fd = ((y(x) - y(x - e * head_out[None, :])) / e)[0]
    dlt = orc.damage_literal(tiny["x"][t:t + 1], tiny["attn"][t:t + 1], tiny["w_o"], tiny["gamma"],
                             tiny["w_gate"], tiny["w_up"], tiny["eps"])[0, h]
    gap = np.linalg.norm(fd - dlt) / np.linalg.norm(dlt)
    assert np.isfinite(gap) and gap < 1.0


def test_single_head_affinity_equals_jvp_square_sum(tiny):
    """Only head h active: row grp(h) is ||w^d_k||^2 sum_t JVP_k^2, all other rows are 0."""
    H = tiny["attn"].shape[1]
    hpg = H // tiny["n_kv_groups"]
    for h in (0, H - 1, 3):
        a = np.zeros_like(tiny["attn"])
        a[:, h] = tiny["attn"][:, h]
        A = _A(tiny, attn=a)
        dd = dict(tiny, attn=a)
        s = sum(_jvp_damage(dd, t, h)[0] ** 2 for t in range(a.shape[0]))
        wd = torch.tensor(tiny["w_down"])
        ref = s * (torch.linalg.vector_norm(wd, dim=0) ** 2).numpy()
        g = h // hpg
        np.testing.assert_allclose(A[g], ref, rtol=1e-10)
        assert np.all(np.delete(A, g, axis=0) == 0.0)


def test_group_sums_its_query_heads(tiny):
    H = tiny["attn"].shape[1]
    G = tiny["n_kv_groups"]
    rows = []
    for h in range(H):
        a = np.zeros_like(tiny["attn"])
        a[:, h] = tiny["attn"][:, h]
        rows.append(_A(tiny, attn=a).sum(axis=0))
    A = _A(tiny)
    for g in range(G):
        np.testing.assert_allclose(A[g], sum(rows[h] for h in range(H) if h // (H // G) == g), rtol=1e-12)


@pytest.mark.parametrize("c", [2.0, 0.5, 3.0])
def test_head_scale_is_quadratic_and_local(tiny, c):
    """a_h -> c a_h (x fixed): Delta_h -> c Delta_h, so only h's term scales by c^2."""
    H = tiny["attn"].shape[1]
    G = tiny["n_kv_groups"]
    h = 2
    a0 = np.zeros_like(tiny["attn"])
    a0[:, h] = tiny["attn"][:, h]
    only_h = _A(tiny, attn=a0)
    a = tiny["attn"].copy()
    a[:, h] *= c
    diff = _A(tiny, attn=a) - _A(tiny)
    np.testing.assert_allclose(diff, (c * c - 1.0) * only_h, rtol=1e-10, atol=1e-12 * only_h.max())
    assert np.all(diff[np.arange(G) != h // (H // G)] == 0.0)


def test_zero_head_removes_its_term(tiny):
    H = tiny["attn"].shape[1]
    a = tiny["attn"].copy()
    a[:, :] = 0.0
    assert np.all(_A(tiny, attn=a) == 0.0)


def test_down_column_scale(tiny):
    k, c = 17, 3.0
    wd = tiny["w_down"].copy()
    wd[:, k] *= c
    A0, A1 = _A(tiny), _A(tiny, w_down=wd)
    np.testing.assert_allclose(A1[:, k], c * c * A0[:, k], rtol=1e-12)
    np.testing.assert_array_equal(np.delete(A1, k, axis=1), np.delete(A0, k, axis=1))


def test_joint_scale_of_x_and_heads_without_eps(tiny):
    """eps = 0: x -> c x and a -> c a leave r-normalised quantities, hence A, unchanged."""
    A0 = _A(tiny, eps=0.0)
    A1 = _A(tiny, eps=0.0, x=2.5 * tiny["x"], attn=2.5 * tiny["attn"])
    np.testing.assert_allclose(A1, A0, rtol=1e-12)


def test_neuron_permutation_permutes_columns(tiny):
    I = tiny["w_gate"].shape[0]
    perm = np.random.default_rng(0).permutation(I)
    A0 = _A(tiny)
    A1 = _A(tiny, w_gate=tiny["w_gate"][perm], w_up=tiny["w_up"][perm], w_down=tiny["w_down"][:, perm])
    np.testing.assert_allclose(A1, A0[:, perm], rtol=1e-12)


def test_group_permutation_permutes_rows(tiny):
    T, H, dh = tiny["attn"].shape
    G = tiny["n_kv_groups"]
    hpg = H // G
    gperm = np.array([2, 0, 3, 1])
    hperm = np.concatenate([np.arange(g * hpg, (g + 1) * hpg) for g in gperm])
    cols = np.concatenate([np.arange(h * dh, (h + 1) * dh) for h in hperm])
    A0 = _A(tiny)
    A1 = _A(tiny, attn=tiny["attn"][:, hperm], w_o=tiny["w_o"][:, cols])
    np.testing.assert_allclose(A1, A0[gperm], rtol=1e-12)


def test_token_chunks_add(tiny):
    A = _A(tiny)
    s = slice(0, 19), slice(19, None)
    parts = [_A(tiny, x=tiny["x"][q], attn=tiny["attn"][q]) for q in s]
    np.testing.assert_allclose(parts[0] + parts[1], A, rtol=1e-12)


def test_folded_equals_literal(tiny):
    kw = {k: v for k, v in tiny.items()}
    np.testing.assert_allclose(orc.affinity_folded(**kw), orc.affinity_literal(**kw), rtol=1e-12)


def test_folded_equals_literal_qwen_shaped_prefix():
    wl = synth.WORKLOADS["qwen3-0.6b-layer"]
    d = _data(wl, T=24)
    lit = orc.affinity_literal(**d, block=8)
    fol = orc.affinity_folded(**d)
    np.testing.assert_allclose(fol, lit, rtol=1e-12)
    sub = [0, 5, 3071, 1000]
    np.testing.assert_allclose(orc.affinity_folded(**d, neurons=sub), lit[:, sub], rtol=1e-12)


def test_silu_prime_is_derivative():
    g = np.linspace(-8, 8, 101)
    gt = torch.tensor(g, requires_grad=True)
    torch.nn.functional.silu(gt).sum().backward()
    np.testing.assert_allclose(orc.silu_prime(g), gt.grad.numpy(), rtol=1e-13, atol=1e-15)



# ----------------------------------------------------------------------------- ADD score
def _preact_removal_add(d):
    """sum_t (g(n) - g(n - p_h))^2 + (u(n) - u(n - p_h))^2 per head, via torch: [H, I]."""
    x = torch.tensor(d["x"])
    gam = torch.tensor(d["gamma"])
    wg, wu = torch.tensor(d["w_gate"]), torch.tensor(d["w_up"])
    wo = torch.tensor(d["w_o"])
    attn = torch.tensor(d["attn"])
    T, H, dh = attn.shape
    r = torch.sqrt(torch.mean(x * x, dim=1, keepdim=True) + d["eps"])
    n = gam * x / r
    out = np.zeros((H, wg.shape[0]))
    for h in range(H):
        piece = gam * (attn[:, h, :] @ wo[:, h * dh:(h + 1) * dh].T) / r
        dg = n @ wg.T - (n - piece) @ wg.T
        du = n @ wu.T - (n - piece) @ wu.T
        out[h] = (dg * dg + du * du).sum(0).numpy()
    return out


def test_add_equals_preactivation_removal(tiny):
    per_head = _preact_removal_add(tiny)
    H = per_head.shape[0]
    G = tiny["n_kv_groups"]
    ref = np.stack([per_head[[h for h in range(H) if h // (H // G) == g]].sum(0) for g in range(G)])
    add = orc.affinity_add_literal(tiny["x"], tiny["attn"], tiny["w_o"], tiny["gamma"],
                                   tiny["w_gate"], tiny["w_up"], G, tiny["eps"])
    np.testing.assert_allclose(add, ref, rtol=1e-9)


def test_add_folded_equals_literal(tiny):
    kw = {k: v for k, v in tiny.items() if k != "w_down"}
    np.testing.assert_allclose(orc.affinity_add_folded(**kw), orc.affinity_add_literal(**kw),
                               rtol=1e-12)
    sub = [0, 9, 127]
    np.testing.assert_allclose(orc.affinity_add_folded(**kw, neurons=sub),
                               orc.affinity_add_literal(**kw)[:, sub], rtol=1e-12)


def test_add_ignores_operating_point_and_write(tiny):
    """ADD depends on x only through r: the pre-activation levels and W_down do not enter."""
    kw = {k: v for k, v in tiny.items() if k != "w_down"}
    base = orc.affinity_add_literal(**kw)
    # flip the sign of x: r is unchanged, g and u flip, ADD must not move
    flipped = orc.affinity_add_literal(**dict(kw, x=-tiny["x"]))
    np.testing.assert_allclose(flipped, base, rtol=1e-12)


def test_add_head_scale_is_quadratic_and_local(tiny):
    kw = {k: v for k, v in tiny.items() if k != "w_down"}
    H = tiny["attn"].shape[1]
    G = tiny["n_kv_groups"]
    a = tiny["attn"].copy()
    a[:, 5] *= 3.0
    only = tiny["attn"] * 0.0
    only[:, 5] = tiny["attn"][:, 5]
    diff = orc.affinity_add_literal(**dict(kw, attn=a)) - orc.affinity_add_literal(**kw)
    np.testing.assert_allclose(diff, 8.0 * orc.affinity_add_literal(**dict(kw, attn=only)),
                               rtol=1e-10, atol=1e-14)
    assert np.all(diff[np.arange(G) != 5 // (H // G)] == 0.0)
