"""The oracle's pins must fail when a plausible mistake is planted in the oracle.

Each case patches one oracle function with a wrong variant (a dropped factor, a wrong
index, a non-exact solver) and checks that the pin meant to guard it now fails.
"""
import numpy as np
import pytest

from oracle import affinity as orc
from oracle import layout as lay
from tests import test_oracle_affinity as pa
from tests import test_oracle_layout as pl


@pytest.fixture(scope="module")
def tiny():
    return pa._data()


def test_wrong_silu_derivative_is_caught(tiny, monkeypatch):
    def bad(g):
        s = orc.sigmoid(g)
        return s * (1.0 + g * s)
    monkeypatch.setattr(orc, "silu_prime", bad)
    with pytest.raises(AssertionError):
        pa.test_damage_equals_autograd_jvp(tiny)


def test_dropped_gain_in_head_piece_is_caught(tiny, monkeypatch):
    orig = orc.head_pieces

    def bad(x, attn, w_o, gamma, eps):
        return orig(x, attn, w_o, np.ones_like(gamma), eps)
    monkeypatch.setattr(orc, "head_pieces", bad)
    with pytest.raises(AssertionError):
        pa.test_damage_equals_autograd_jvp(tiny)


def test_wrong_group_mapping_is_caught(tiny, monkeypatch):
    monkeypatch.setattr(orc, "group_of_head", lambda H, G: np.arange(H) % G)
    with pytest.raises(AssertionError):
        pa.test_single_head_affinity_equals_jvp_square_sum(tiny)


def test_unsquared_down_norm_is_caught(tiny, monkeypatch):
    orig = orc._aggregate

    def bad(s, w_down, G):
        return orig(s, np.sqrt(np.abs(w_down)) * np.sign(w_down), G)   # ||w||, not ||w||^2
    monkeypatch.setattr(orc, "_aggregate", bad)
    with pytest.raises(AssertionError):
        pa.test_down_column_scale(tiny)


def test_mean_instead_of_token_sum_is_caught(tiny, monkeypatch):
    orig = orc.affinity_literal

    def bad(x, attn, *a, **k):
        return orig(x, attn, *a, **k) / x.shape[0]
    monkeypatch.setattr(orc, "affinity_literal", bad)
    with pytest.raises(AssertionError):
        pa.test_token_chunks_add(tiny)


def test_heuristic_assignment_is_caught(monkeypatch):
    def greedy(M):
        I, L = M.shape
        nu = np.empty(I, dtype=np.int64)
        cap = [I // L] * L
        for k in range(I):
            for l in np.argsort(-M[k], kind="stable"):
                if cap[l]:
                    nu[k] = l
                    cap[l] -= 1
                    break
        return nu
    monkeypatch.setattr(lay, "optimal_assignment", greedy)
    with pytest.raises(AssertionError):
        for I, L, seed in [(8, 2, 1), (8, 4, 2), (9, 3, 4)]:
            pl.test_assign_brute_force(I, L, seed)


def test_wrong_tie_break_is_caught(monkeypatch):
    monkeypatch.setattr(lay, "best_partition", lambda s, minimise=False: int(np.argmax(s[::-1]) * -1 + len(s) - 1))
    with pytest.raises(AssertionError):
        pl.test_head_step_brute_force_and_ties()


# ----------------------------------------------------------------------------- down edge
from oracle import down as dwn  # noqa: E402
from tests import test_oracle_down as pd  # noqa: E402


@pytest.fixture(scope="module")
def tiny_down():
    return pd._data()


def test_down_gain_dropped_is_caught(tiny_down, monkeypatch):
    orig = dwn.down_weight_norms

    def bad(w_q, w_k, w_v, gamma_next, w_down, H, G):
        return orig(w_q, w_k, w_v, np.ones_like(gamma_next), w_down, H, G)
    monkeypatch.setattr(dwn, "down_weight_norms", bad)
    with pytest.raises(AssertionError):
        pd.test_equals_removal_through_next_projection(tiny_down)


def test_down_wrong_rms_is_caught(tiny_down, monkeypatch):
    orig = dwn.down_token_stat

    def bad(x, gamma, w_gate, w_up, eps, x_next, eps_next):  # this layer's r instead of r'
        return orig(x, gamma, w_gate, w_up, eps, x, eps)
    monkeypatch.setattr(dwn, "down_token_stat", bad)
    with pytest.raises(AssertionError):
        pd.test_equals_removal_through_next_projection(tiny_down)


def test_down_wrong_group_rows_are_caught(tiny_down, monkeypatch):
    def bad(H, G, dh, g):  # strided query heads instead of consecutive ones
        q = np.concatenate([np.arange(h * dh, (h + 1) * dh) for h in range(g, H, G)])
        return q, np.arange(g * dh, (g + 1) * dh)
    monkeypatch.setattr(dwn, "qkv_rows", bad)
    with pytest.raises(AssertionError):
        pd.test_equals_removal_through_next_projection(tiny_down)


def test_down_value_rows_dropped_are_caught(tiny_down, monkeypatch):
    def bad(w_q, w_k, w_v, H, G, g):
        dh = w_k.shape[0] // G
        q, kv = dwn.qkv_rows(H, G, dh, g)
        return np.concatenate([w_q[q], w_k[kv]], axis=0)
    monkeypatch.setattr(dwn, "group_projection", bad)
    with pytest.raises(AssertionError):
        pd.test_equals_removal_through_next_projection(tiny_down)


# ----------------------------------------------------------------------------- ADD, random, optimum
def test_add_dropping_up_term_is_caught(tiny, monkeypatch):
    def bad(x, attn, w_o, gamma, w_gate, w_up, n_kv_groups, eps, block=128):
        T, H, _ = attn.shape
        acc = np.zeros((H, w_gate.shape[0]))
        p = orc.head_pieces(x, attn, w_o, gamma, eps)
        acc += np.sum((p @ w_gate.T) ** 2, axis=0)
        return orc._group_sum(acc, n_kv_groups)
    monkeypatch.setattr(orc, "affinity_add_literal", bad)
    with pytest.raises(AssertionError):
        pa.test_add_equals_preactivation_removal(tiny)


def test_sattolo_shuffle_is_caught(monkeypatch):
    def bad(labels, seed, counter):  # i in [0, j): only cyclic permutations
        a = list(labels)
        for j in range(len(a) - 1, 0, -1):
            r = lay.splitmix64(seed, counter)
            counter += 1
            i = (r * j) >> 64
            a[j], a[i] = a[i], a[j]
        return a, counter
    monkeypatch.setattr(lay, "_shuffle", bad)
    with pytest.raises(AssertionError):
        pl.test_random_layout_marginals_are_uniform()


def test_wrong_splitmix_constant_is_caught(monkeypatch):
    monkeypatch.setattr(lay, "SPLITMIX_GAMMA", 0x9E3779B97F4A7C13)
    with pytest.raises(AssertionError):
        pl.test_splitmix64_published_outputs()


def test_optimum_over_contiguous_heads_only_is_caught(monkeypatch):
    monkeypatch.setattr(lay, "unlabelled_partitions", lambda G, L: [lay.contiguous_heads(G, L)])
    with pytest.raises(AssertionError):
        pl.test_layer_optimum_equals_brute_force(4, 8, 2, 31)


# ---- the paper's approximate neuron assignment
from oracle import dual_ascent as da  # noqa: E402
from tests import test_oracle_dual_ascent as pda  # noqa: E402


def test_one_sided_swap_gain_is_caught(monkeypatch):
    def bad(M, nu):
        _, L = M.shape
        nu = np.array(nu, dtype=np.int64)
        for a in range(L):
            for b in range(a + 1, L):
                on_a, on_b = np.flatnonzero(nu == a), np.flatnonzero(nu == b)
                to_b = M[on_a, b] - M[on_a, a]
                i = int(np.argmax(to_b))
                if to_b[i] > 0:   # ignores what the partner loses
                    j = int(np.argmin(M[on_b, b] - M[on_b, a]))
                    nu[on_a[i]], nu[on_b[j]] = b, a
        return nu
    monkeypatch.setattr(da, "pairwise_swaps", bad)
    with pytest.raises(AssertionError):
        pda.test_swaps_from_the_contiguous_layout_end_at_a_local_optimum(24, 3, 11)


def test_costliest_fix_up_move_is_caught(monkeypatch):
    def bad(M, nu):
        I, L = M.shape
        cap = I // L
        nu = np.array(nu, dtype=np.int64)
        load = np.bincount(nu, minlength=L)
        while np.any(load > cap):
            movable = np.flatnonzero(load[nu] > cap)
            targets = np.flatnonzero(load < cap)
            loss = M[movable, nu[movable]][:, None] - M[np.ix_(movable, targets)]
            flat = int(np.argmax(loss))
            k, b = movable[flat // len(targets)], targets[flat % len(targets)]
            load[nu[k]] -= 1
            load[b] += 1
            nu[k] = b
        return nu
    monkeypatch.setattr(da, "fix_up", bad)
    with pytest.raises(AssertionError):
        pda.test_fix_up_moves_the_cheapest_excess()


def test_offsets_moving_the_wrong_way_are_caught(monkeypatch):
    orig = da.dual_offsets

    def bad(M, iterations=da.ITERATIONS, decay=da.DECAY):
        lam, _ = orig(M, iterations, decay)
        lam = -lam
        return lam, np.argmax(M.astype(np.float64) - lam[None, :], axis=1)
    monkeypatch.setattr(da, "dual_offsets", bad)
    M = np.zeros((12, 3), dtype=np.int64)
    M[:, 0] = 10          # every neuron prefers device 0: the offsets must push them away
    lam, _ = da.dual_offsets(M)
    assert lam[0] < 0     # wrong direction: device 0 got cheaper


# ---- chain coupling of eq. (objective) and of the two block steps
def test_neuron_gain_down_term_keyed_to_own_heads_is_caught(monkeypatch):
    orig = lay.neuron_gain

    def bad(Q_up, h, L, Q_down=None, h_next=None):   # down edge against h_i, not h_{i+1}
        return orig(Q_up, h, L, Q_down, h if Q_down is not None else None)
    monkeypatch.setattr(lay, "neuron_gain", bad)
    with pytest.raises(AssertionError):
        pl.test_neuron_block_is_the_brute_force_optimum_of_the_chain(3, 4, 8, 2, 51)


def test_head_gain_down_term_keyed_to_own_neurons_is_caught(monkeypatch):
    orig = lay.head_gain

    def bad(Q_up, nu, L, Q_down_prev=None, nu_prev=None):   # nu_i, not nu_{i-1}
        return orig(Q_up, nu, L, Q_down_prev, nu if Q_down_prev is not None else None)
    monkeypatch.setattr(lay, "head_gain", bad)
    with pytest.raises(AssertionError):
        pl.test_head_block_is_the_brute_force_optimum_of_the_chain(3, 4, 8, 2, 61)


def test_objective_down_edge_keyed_to_own_heads_is_caught(monkeypatch):
    def bad(Q_up, Q_down, hs, nus):
        J = 0
        for i in range(len(Q_up)):
            h, nu = np.asarray(hs[i]), np.asarray(nus[i])
            J += int(Q_up[i][h[:, None] == nu[None, :]].sum())
            if Q_down is not None and i + 1 < len(Q_up):
                J += int(Q_down[i][nu[:, None] == h[None, :]].sum())   # h_i, not h_{i+1}
        return J
    monkeypatch.setattr(lay, "objective", bad)
    with pytest.raises(AssertionError):
        pl.test_objective_equals_explicit_chain_sum(3, 4, 8, 2)
    with pytest.raises(AssertionError):
        pl.test_single_down_entry_counts_with_the_next_layers_group()
