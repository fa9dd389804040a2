"""First-order rounding-error model of the GPU affinity (test infrastructure).

The library reads the same bf16 inputs as the oracle, but it keeps some derived operands
at lower precision than the oracle's fp64:

* W' = gamma * W, the gate and up rows of the operating point, rounded to bf16;
* the folded per-head weights F_h = W_o^(h) W'^T, rounded to bf16;
* the damage coefficients c1 = silu'(g) u / r and c2 = silu(g) / r, kept in fp16;
* on the down edge, gamma' * w^d_k rounded to bf16 before the next layer's projection.

Each such rounding is modelled as an independent relative error of rms at most u/sqrt(3),
u = 2^-8 for bf16's 8 significant bits and 2^-11 for fp16's 11: round-to-nearest leaves
an absolute error uniform within half a unit in the last place, and a unit in the last
place is at most 2u times the value.  The sums themselves (fp32 MFMA accumulation over a
few thousand terms, fp64 across tokens and splits) add errors orders of magnitude
smaller and are neglected.

The functions here propagate those roundings through the definitions of Section 3
("Affinity scores") in fp64, from the inputs alone: they never see what the library
computed.  Per entry they return the oracle's value, the standard deviation sigma of
the first-order error, and a bound on the second-order terms.  A correct GPU result then
lies within a few sigma of the oracle.  kappa = sigma / (rho_bf16 * value) is the entry's
condition number: about 1 when nothing cancels, large where a pre-activation is near zero,
where the two damage terms cancel, or where a single token dominates the sum.
"""
from __future__ import annotations

import numpy as np

from oracle import affinity as orc

RHO_BF16 = 2.0 ** -8 / np.sqrt(3.0)
RHO_FP16 = 2.0 ** -11 / np.sqrt(3.0)
N_SIGMA = 6.0      # a correct entry lies within this many sigma (plus the second-order bound)
N_SECOND = 4.0     # multiple of the second-order bound allowed on top
# An entry is held to the target's relative bar when N_HOLD sigma (plus the second-order
# bound) fits inside it.  sigma is an upper bound: emulating the roundings gives errors of
# rms 0.70-0.76 sigma, so N_HOLD model sigmas are about 5.5 actual standard deviations,
# a tail below 1e-7 per entry.
N_HOLD = 4.0


def _silu_derivatives(g):
    s = orc.sigmoid(g)
    q = s * (1.0 - s)
    d1 = s * (1.0 + g * (1.0 - s))                                    # silu'
    d2 = q * (2.0 + g * (1.0 - 2.0 * s))                              # silu''
    d3 = q * ((1.0 - 2.0 * s) * (3.0 + g * (1.0 - 2.0 * s)) - 2.0 * g * q)   # silu'''
    return g * s, d1, d2, d3


def up_affinity_error(x, attn, w_o, gamma, w_gate, w_up, w_down, n_kv_groups, eps):
    """(A [G, I], sigma [G, I], second [G, I]) of the FO up affinity on a few tokens.

    Sources: W'_gate, W'_up (shared by all tokens and heads), the folded F_h (shared by all
    tokens), and c1, c2 (one pair per token and neuron).  Memory is O(T H I), so T should
    stay small (tens of tokens).
    """
    T, H, dh = attn.shape
    hpg = H // n_kv_groups
    r = orc.rms(x, eps)
    xr = x / r[:, None]                                   # [T, d]
    Wg = w_gate * gamma[None, :]                          # exact gamma * W, [I, d]
    Wu = w_up * gamma[None, :]
    g, u = xr @ Wg.T, xr @ Wu.T                           # [T, I]
    sl, d1, d2, d3 = _silu_derivatives(g)
    ri = (1.0 / r)[:, None]
    c1, c2 = d1 * u * ri, sl * ri                          # [T, I]
    c1_g, c1_u, c2_g = d2 * u * ri, d1 * ri, d1 * ri       # first derivatives
    c1_gg, c1_gu, c2_gg = d3 * u * ri, d2 * ri, d2 * ri    # second derivatives
    O = np.stack([attn[:, h, :] @ w_o[:, h * dh:(h + 1) * dh].T for h in range(H)], axis=1)  # [T,H,d]
    Pg, Pu = O @ Wg.T, O @ Wu.T                           # r p_h . w_k, [T, H, I]
    D = c1[:, None, :] * Pg + c2[:, None, :] * Pu         # Delta
    Fg = orc.fold(w_o, gamma, w_gate, H)                  # [H, dh, I]
    Fu = orc.fold(w_o, gamma, w_up, H)
    nd = np.sum(w_down * w_down, axis=0)                  # [I]
    dDg = c1_g[:, None, :] * Pg + c2_g[:, None, :] * Pu   # dDelta/dg
    dDu = c1_u[:, None, :] * Pg                           # dDelta/du

    # Variances of the perturbations of g, u, Pg, Pu per token (and head) for the
    # second-order bound.
    Wg2, Wu2 = Wg * Wg, Wu * Wu
    var_g = RHO_BF16 ** 2 * (xr * xr) @ Wg2.T             # [T, I]
    var_u = RHO_BF16 ** 2 * (xr * xr) @ Wu2.T
    a2 = attn * attn
    var_Pg = RHO_BF16 ** 2 * ((O * O) @ Wg2.T + np.stack([a2[:, h] @ (Fg[h] ** 2) for h in range(H)], 1))
    var_Pu = RHO_BF16 ** 2 * ((O * O) @ Wu2.T + np.stack([a2[:, h] @ (Fu[h] ** 2) for h in range(H)], 1))
    # Var(first-order dDelta) per (t, h, k): each source's coefficient squared.
    xo_g = np.einsum("td,thd,kd->thk", xr, O, Wg2)
    xo_u = np.einsum("td,thd,kd->thk", xr, O, Wu2)
    oo_g, oo_u = (O * O) @ Wg2.T, (O * O) @ Wu2.T
    xx_g, xx_u = (xr * xr) @ Wg2.T, (xr * xr) @ Wu2.T
    c1h, c2h = c1[:, None, :], c2[:, None, :]
    var_D = RHO_BF16 ** 2 * (
        dDg ** 2 * xx_g[:, None, :] + 2 * dDg * c1h * xo_g + c1h ** 2 * oo_g
        + dDu ** 2 * xx_u[:, None, :] + 2 * dDu * c2h * xo_u + c2h ** 2 * oo_u
        + c1h ** 2 * np.stack([a2[:, h] @ (Fg[h] ** 2) for h in range(H)], 1)
        + c2h ** 2 * np.stack([a2[:, h] @ (Fu[h] ** 2) for h in range(H)], 1)
    ) + RHO_FP16 ** 2 * ((c1h * Pg) ** 2 + (c2h * Pu) ** 2)
    sd_c1 = np.sqrt(c1_g ** 2 * var_g + c1_u ** 2 * var_u + RHO_FP16 ** 2 * c1 ** 2)[:, None, :]
    sd_c2 = np.sqrt(c2_g ** 2 * var_g + RHO_FP16 ** 2 * c2 ** 2)[:, None, :]
    curv = 0.5 * np.abs(c1_gg[:, None, :] * Pg + c2_gg[:, None, :] * Pu) * var_g[:, None, :] \
        + np.abs(c1_gu[:, None, :] * Pg) * np.sqrt(var_g * var_u)[:, None, :]
    second_th = var_D + 2.0 * np.abs(D) * (sd_c1 * np.sqrt(var_Pg) + sd_c2 * np.sqrt(var_Pu) + curv)

    G, I = n_kv_groups, w_gate.shape[0]
    A = np.zeros((G, I))
    sig2 = np.zeros((G, I))
    second = np.zeros((G, I))
    for grp in range(G):
        hs = range(grp * hpg, (grp + 1) * hpg)
        A[grp] = nd * sum(np.sum(D[:, h] ** 2, axis=0) for h in hs)
        second[grp] = nd * sum(np.sum(second_th[:, h], axis=0) for h in hs)
        # W'_gate and W'_up: one rounding per (k, j), shared by every token and head
        Mg = sum((2 * D[:, h] * dDg[:, h]).T @ xr + (2 * D[:, h] * c1).T @ O[:, h] for h in hs)
        Mu = sum((2 * D[:, h] * dDu[:, h]).T @ xr + (2 * D[:, h] * c2).T @ O[:, h] for h in hs)
        v = RHO_BF16 ** 2 * (np.sum((Wg * Mg) ** 2, axis=1) + np.sum((Wu * Mu) ** 2, axis=1))
        # F_h: one rounding per (h, e, k), shared by every token
        for h in hs:
            v += RHO_BF16 ** 2 * np.sum((attn[:, h].T @ (2 * D[:, h] * c1) * Fg[h]) ** 2, axis=0)
            v += RHO_BF16 ** 2 * np.sum((attn[:, h].T @ (2 * D[:, h] * c2) * Fu[h]) ** 2, axis=0)
        # c1, c2: one rounding per (t, k), shared by the group's heads
        z1 = sum(2 * D[:, h] * c1 * Pg[:, h] for h in hs)
        z2 = sum(2 * D[:, h] * c2 * Pu[:, h] for h in hs)
        v += RHO_FP16 ** 2 * np.sum(z1 ** 2 + z2 ** 2, axis=0)
        sig2[grp] = nd * nd * v
    return A, np.sqrt(sig2), second


def down_stat_error(x, gamma, w_gate, w_up, eps, x_next, eps_next):
    """(s [I], sigma [I], second [I]) of the down-edge token statistic
    s[k] = sum_t alpha_k^2 / r'^2, alpha = silu(g) u, with W' rounded to bf16."""
    r = orc.rms(x, eps)
    rn = orc.rms(x_next, eps_next)
    xr = x / r[:, None]
    Wg, Wu = w_gate * gamma[None, :], w_up * gamma[None, :]
    g, u = xr @ Wg.T, xr @ Wu.T
    sl, d1, d2, _ = _silu_derivatives(g)
    w = (1.0 / rn ** 2)[:, None]
    al = sl * u
    s = np.sum(al * al * w, axis=0)
    a_g, a_u, a_gg, a_gu = d1 * u, sl, d2 * u, d1          # derivatives of alpha
    # first order: coefficients of the roundings of W'_gate and W'_up, shared by all tokens
    Mg = (2 * al * a_g * w).T @ xr                        # [I, d]
    Mu = (2 * al * a_u * w).T @ xr
    sig2 = RHO_BF16 ** 2 * (np.sum((Wg * Mg) ** 2, axis=1) + np.sum((Wu * Mu) ** 2, axis=1))
    var_g = RHO_BF16 ** 2 * (xr * xr) @ (Wg * Wg).T
    var_u = RHO_BF16 ** 2 * (xr * xr) @ (Wu * Wu).T
    var_a = a_g ** 2 * var_g + a_u ** 2 * var_u
    curv = 0.5 * np.abs(a_gg) * var_g + np.abs(a_gu) * np.sqrt(var_g * var_u)
    second = np.sum((var_a + 2 * np.abs(al) * curv) * w, axis=0)
    return s, np.sqrt(sig2), second


def down_weight_error(w_q, w_k, w_v, gamma_next, w_down, n_q_heads, n_kv_groups):
    """(B [G, I], sigma [G, I], second [G, I]) of B[g, k] = ||W^qkv_g (gamma' * w^d_k)||^2
    with gamma' * w^d_k rounded to bf16 (one rounding per (j, k), shared by every group)."""
    from oracle import down as dwn
    m = gamma_next[:, None] * w_down                      # [d, I]
    G = n_kv_groups
    B = np.empty((G, w_down.shape[1]))
    sig = np.empty_like(B)
    second = np.empty_like(B)
    for grp in range(G):
        Wq = dwn.group_projection(w_q, w_k, w_v, n_q_heads, n_kv_groups, grp)   # [R, d]
        b = Wq @ m                                        # [R, I]
        B[grp] = np.sum(b * b, axis=0)
        coef = m * (2.0 * Wq.T @ b)                       # dB/d(relative error of m_jk)
        sig[grp] = RHO_BF16 * np.sqrt(np.sum(coef * coef, axis=0))
        second[grp] = RHO_BF16 ** 2 * np.sum((Wq * Wq) @ (m * m), axis=0)
    return B, sig, second


def check_entrywise(got, ref, sigma, second, rel=1e-2, thresh=1e-3, label=""):
    """Entrywise parity under the rounding model.

    * Every entry lies within N_SIGMA sigma + N_SECOND second of the oracle.
    * Entries above thresh * max are held to relative error rel (the target's bar)
      unless N_HOLD sigma + N_SECOND second exceeds rel, i.e. unless the condition number
      kappa > rel / (N_HOLD rho_bf16) = 1.1 to first order; those are exempted and counted.
    * Entries below thresh * max are held to rel * thresh * max absolute, with the same
      exemption when their bound exceeds that.

    Returns a dict: the largest relative error over the held entries, how many entries
    were held and how many exempted."""
    got = np.asarray(got, dtype=np.float64)
    assert got.shape == ref.shape and np.all(np.isfinite(got))
    err = np.abs(got - ref)
    bound = N_SIGMA * sigma + N_SECOND * second
    top = ref.max()
    bad = err > bound + 1e-6 * top
    assert not bad.any(), (f"{label}: {int(bad.sum())} entries outside the rounding model, worst "
                           f"|err|/bound = {np.max(err[bad] / (bound[bad] + 1e-6 * top)):.2f}")
    big = ref > thresh * top
    hold = N_HOLD * sigma + N_SECOND * second
    held = big & (hold <= rel * ref)
    rel_err = err[held] / ref[held]
    assert rel_err.size == 0 or rel_err.max() <= rel, f"{label}: max rel err {rel_err.max():.3e}"
    small_held = ~big & (hold <= rel * thresh * top)
    assert err[small_held].max(initial=0.0) <= rel * thresh * top, f"{label}: small entry"
    z = err[big] / np.maximum(sigma[big], 1e-300)
    return {"max_rel_err_held": float(rel_err.max(initial=0.0)), "held": int(held.sum() + small_held.sum()),
            "exempt": int(ref.size - held.sum() - small_held.sum()), "entries": int(ref.size),
            "max_rel_err_all": float((err[big] / ref[big]).max(initial=0.0)),
            "max_sigmas": float(z.max(initial=0.0))}
