"""CPU oracle for the layout objective and its optimiser (test infrastructure only).

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s ``cpu_baseline`` leg may
import this module.  It shares no code with the HIP library.  All arithmetic on scores
is exact (Python integers or int64 below 2^62), so results do not depend on the order
of any summation.

Section 3 of the paper, "Objective" and "Optimiser":

* every affinity matrix is normalised to unit mass; J (eq. ``objective``) is the total
  co-located normalised affinity over the N up edges (KV groups of layer i -> neurons
  of layer i) and the N-1 down edges (neurons of layer i -> KV groups of layer i+1);
* h_i maps the G KV groups and nu_i the I neurons of layer i to the L devices, each
  balanced (G/L groups and I/L neurons per device);
* neuron step: given h_i and h_{i+1}, the gain M_kl of putting neuron k on device l is
  the normalised up affinity of k to the groups on l plus its normalised down
  affinity to the next layer's groups on l; the best balanced nu_i is a linear
  assignment with I/L slots per device;
* head step: given nu_{i-1} and nu_i, score every labelled balanced partition of the
  G groups and keep the best;
* coordinate ascent: from the contiguous head assignment, alternate the two steps
  over all layers until J stops increasing.

Readings (the paper does not fix these; each is listed in the design notes):

* unit mass in exact arithmetic: ``encode`` maps a raw fp32 matrix to integers that sum
  to 2^48 up to truncation (one unit per entry at most), J_int is the integer sum of
  co-located codes and J = J_int / 2^48;
* ties: the best partition is the one of lowest lexicographic rank; the neuron
  assignment is the lexicographically smallest optimal nu;
* a sweep is the neuron block over all layers, then the head block over all layers;
  the ascent stops at the first sweep whose J_int does not exceed the previous one.

The neuron step finds an optimum by cycle cancelling on the L-device exchange graph
(an assignment is optimal exactly when no cycle of single-neuron moves gains), then
picks the lexicographically smallest optimum among the assignments that use only
tight edges of a dual solution derived from it.
"""
from __future__ import annotations

import itertools
import math

import numpy as np

FRAC_BITS = 48   # codes sum to 2^48 (unit mass)
MANT_BITS = 40   # the largest entry is scaled into [2^40, 2^41) before truncation


# ----------------------------------------------------------------------------- encoding
def encode(A) -> np.ndarray:
    """Unit-mass fixed-point code of a non-negative fp32 matrix, exact.

    E = floor(log2 max A); q_i = floor(A_i 2^(40-E)) (exact for fp32 inputs);
    Q_i = floor(q_i 2^48 / sum q).  Returns int64 codes with the input's shape.
    """
    a = np.asarray(A, dtype=np.float32)
    flat = [float(v) for v in a.ravel()]
    if any(not math.isfinite(v) or v < 0 for v in flat):
        raise ValueError("affinity must be finite and non-negative")
    amax = max(flat) if flat else 0.0
    if amax <= 0.0:
        raise ValueError("degenerate affinity (all zero)")
    E = math.frexp(amax)[1] - 1                    # amax in [2^E, 2^(E+1))
    q = [math.floor(math.ldexp(v, MANT_BITS - E)) for v in flat]
    S = sum(q)
    Q = [(qi << FRAC_BITS) // S for qi in q]
    return np.array(Q, dtype=np.int64).reshape(a.shape)


# ----------------------------------------------------------------------------- partitions
def partitions(G: int, L: int) -> list:
    """Every labelled balanced h in {0..L-1}^G (G/L groups per device), lexicographic."""
    if L <= 0 or G % L:
        raise ValueError("G must be a multiple of L")
    per = G // L
    return [h for h in itertools.product(range(L), repeat=G)
            if all(h.count(l) == per for l in range(L))]


def contiguous_heads(G: int, L: int) -> tuple:
    return tuple(g // (G // L) for g in range(G))


def contiguous_neurons(I: int, L: int) -> np.ndarray:
    return np.arange(I) // (I // L)


def head_gain(Q_up, nu, L, Q_down_prev=None, nu_prev=None) -> np.ndarray:
    """C[g, l]: co-located mass gained by putting KV group g of layer i on device l.

    Up edge of layer i: sum of Q_up[g, k] over the neurons k of layer i on l.  Down edge
    from layer i-1: sum of Q_down_prev[k, g] over the neurons k of layer i-1 on l.
    """
    G = Q_up.shape[0]
    C = np.zeros((G, L), dtype=np.int64)
    for l in range(L):
        C[:, l] = Q_up[:, np.asarray(nu) == l].sum(axis=1)
        if Q_down_prev is not None:
            C[:, l] += Q_down_prev[np.asarray(nu_prev) == l, :].sum(axis=0)
    return C


def partition_scores(C: np.ndarray, parts: list) -> np.ndarray:
    G = C.shape[0]
    return np.array([sum(int(C[g, h[g]]) for g in range(G)) for h in parts], dtype=np.int64)


def best_partition(scores: np.ndarray, minimise: bool = False) -> int:
    """Rank of the best score; the lowest rank wins ties."""
    best = 0
    for p in range(1, len(scores)):
        if (scores[p] < scores[best]) if minimise else (scores[p] > scores[best]):
            best = p
    return best


# ----------------------------------------------------------------------------- neuron step
def neuron_gain(Q_up, h, L, Q_down=None, h_next=None) -> np.ndarray:
    """M[k, l] = sum_{g: h(g)=l} Q_up[g, k] + sum_{g: h_next(g)=l} Q_down[k, g]."""
    G, I = Q_up.shape
    M = np.zeros((I, L), dtype=np.int64)
    h = np.asarray(h)
    for l in range(L):
        M[:, l] = Q_up[h == l, :].sum(axis=0)
        if Q_down is not None:
            M[:, l] += Q_down[:, np.asarray(h_next) == l].sum(axis=1)
    return M


def _exchange_graph(M, nu, L):
    """w[a][b] = best gain of moving one neuron from device a to device b, and who."""
    w = [[None] * L for _ in range(L)]
    who = [[-1] * L for _ in range(L)]
    for a in range(L):
        idx = np.nonzero(nu == a)[0]
        if idx.size == 0:
            continue
        for b in range(L):
            if a == b:
                continue
            gain = M[idx, b] - M[idx, a]
            j = int(np.argmax(gain))
            w[a][b] = int(gain[j])
            who[a][b] = int(idx[j])
    return w, who


def _simple_cycles(L):
    for n in range(2, L + 1):
        for cyc in itertools.permutations(range(L), n):
            if cyc[0] == min(cyc):
                yield cyc


def optimal_assignment(M: np.ndarray) -> np.ndarray:
    """An optimal balanced assignment by cycle cancelling, from the contiguous one."""
    I, L = M.shape
    nu = contiguous_neurons(I, L).copy()
    cycles = list(_simple_cycles(L))
    while True:
        w, who = _exchange_graph(M, nu, L)
        best, best_gain = None, 0
        for cyc in cycles:
            edges = [(cyc[i], cyc[(i + 1) % len(cyc)]) for i in range(len(cyc))]
            if any(w[a][b] is None for a, b in edges):
                continue
            gain = sum(w[a][b] for a, b in edges)
            if gain > best_gain:
                best, best_gain = edges, gain
        if best is None:
            return nu
        moves = [(who[a][b], b) for a, b in best]
        for k, b in moves:
            nu[k] = b


def dual_prices(M: np.ndarray, nu: np.ndarray) -> list:
    """Device prices lambda with M[k,nu(k)] - lambda_nu(k) >= M[k,l] - lambda_l for all k, l.

    Longest-path distances in the exchange graph (weights w[a][b]); they exist because an
    optimal assignment has no gaining cycle.
    """
    I, L = M.shape
    w, _ = _exchange_graph(M, nu, L)
    lam = [0] * L
    for _ in range(L):
        for a in range(L):
            for b in range(L):
                if a != b and w[a][b] is not None and lam[a] + w[a][b] > lam[b]:
                    lam[b] = lam[a] + w[a][b]
    return lam


def _hall_ok(cnt_by_mask, cap, L):
    """Can every remaining neuron (counted by tight-device mask) be placed within cap?"""
    for S in range(1, 1 << L):
        need = sum(c for m, c in cnt_by_mask.items() if m & ~S == 0)
        have = sum(cap[l] for l in range(L) if S >> l & 1)
        if need > have:
            return False
    return True


def canonical_assignment(M: np.ndarray, nu_opt: np.ndarray) -> np.ndarray:
    """Lexicographically smallest optimal balanced assignment.

    With prices lambda from an optimal assignment, the optimal assignments are exactly the
    balanced ones that put every neuron k on a device of its tight set
    argmax_l (M[k,l] - lambda_l) (complementary slackness).  Greedily give each neuron, in
    index order, the smallest tight device that still leaves a feasible completion.
    """
    I, L = M.shape
    lam = dual_prices(M, nu_opt)
    red = M - np.array(lam, dtype=np.int64)[None, :]
    top = red.max(axis=1)
    masks = [sum(1 << l for l in range(L) if red[k, l] == top[k]) for k in range(I)]
    cnt = {}
    for m in masks:
        cnt[m] = cnt.get(m, 0) + 1
    cap = [I // L] * L
    nu = np.empty(I, dtype=np.int64)
    for k in range(I):
        cnt[masks[k]] -= 1
        for l in range(L):
            if not (masks[k] >> l & 1) or cap[l] == 0:
                continue
            cap[l] -= 1
            if _hall_ok(cnt, cap, L):
                nu[k] = l
                break
            cap[l] += 1
        else:
            raise AssertionError("no feasible tight completion (dual not optimal)")
    return nu


def balanced_assign(M: np.ndarray, minimise: bool = False):
    """(canonical nu [I], value) maximising (or minimising) sum_k M[k, nu(k)]."""
    M = np.asarray(M, dtype=np.int64)
    I, L = M.shape
    if L <= 0 or I % L:
        raise ValueError("I must be a multiple of L")
    Mx = -M if minimise else M
    nu = canonical_assignment(Mx, optimal_assignment(Mx))
    return nu, int(M[np.arange(I), nu].sum())


# ----------------------------------------------------------------------------- objective
def objective(Q_up: list, Q_down: list, hs: list, nus: list) -> int:
    """J_int (eq. ``objective``): co-located codes over N up and N-1 down edges."""
    N = len(Q_up)
    J = 0
    for i in range(N):
        h = np.asarray(hs[i])
        nu = np.asarray(nus[i])
        J += int(Q_up[i][h[:, None] == nu[None, :]].sum())
        if Q_down is not None and i + 1 < N:
            hn = np.asarray(hs[i + 1])
            J += int(Q_down[i][nu[:, None] == hn[None, :]].sum())
    return J


def coordinate_ascent(Q_up: list, Q_down, L: int, max_sweeps: int = 64,
                      freeze_heads: bool = False, freeze_neurons: bool = False,
                      minimise: bool = False, layer_mask=None, neuron_step=None):
    """Alternate the neuron and head blocks from contiguous layouts (Section 3, Optimiser).

    Returns (hs, nus, J_int, sweeps).  ``layer_mask[i]`` false keeps layer i contiguous;
    ``freeze_*`` keep that block contiguous; ``minimise`` minimises J instead.
    ``neuron_step(M, minimise) -> nu`` replaces the exact neuron step (default: the
    canonical optimum of ``balanced_assign``).
    """
    N = len(Q_up)
    G, I = Q_up[0].shape
    parts = partitions(G, L)
    hs = [contiguous_heads(G, L) for _ in range(N)]
    nus = [contiguous_neurons(I, L) for _ in range(N)]
    moves = [True] * N if layer_mask is None else [bool(m) for m in layer_mask]
    J_prev = None
    sweeps = 0
    while sweeps < max_sweeps:
        sweeps += 1
        if not freeze_neurons:
            for i in range(N):
                if not moves[i]:
                    continue
                down = Q_down[i] if (Q_down is not None and i + 1 < N) else None
                M = neuron_gain(Q_up[i], hs[i], L, down, hs[i + 1] if down is not None else None)
                if neuron_step is None:
                    nus[i], _ = balanced_assign(M, minimise)
                else:
                    nus[i] = np.asarray(neuron_step(M, minimise))
        if not freeze_heads:
            for i in range(N):
                if not moves[i]:
                    continue
                prev = Q_down[i - 1] if (Q_down is not None and i > 0) else None
                C = head_gain(Q_up[i], nus[i], L, prev, nus[i - 1] if prev is not None else None)
                hs[i] = parts[best_partition(partition_scores(C, parts), minimise)]
        J = objective(Q_up, Q_down, hs, nus)
        better = J_prev is None or ((J < J_prev) if minimise else (J > J_prev))
        if not better:
            break
        J_prev = J
    return hs, nus, objective(Q_up, Q_down, hs, nus), sweeps


# ----------------------------------------------------------------------------- random layouts
SPLITMIX_GAMMA = 0x9E3779B97F4A7C15
_M64 = (1 << 64) - 1


def splitmix64(seed: int, n: int) -> int:
    """Output n (from 0) of SplitMix64 started from state ``seed``: the state advances by
    the golden-ratio increment and each state is mixed by two xor-shift-multiply rounds
    and a final xor-shift (Steele, Lea and Flood, OOPSLA 2014)."""
    z = (seed + (n + 1) * SPLITMIX_GAMMA) & _M64
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & _M64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & _M64
    return z ^ (z >> 31)


def _shuffle(labels, seed: int, counter: int):
    """Fisher-Yates from the last position down; position j swaps with
    floor(r (j + 1) / 2^64) for the next generator output r.  Returns (labels, counter)."""
    a = list(labels)
    for j in range(len(a) - 1, 0, -1):
        r = splitmix64(seed, counter)
        counter += 1
        i = (r * (j + 1)) >> 64
        a[j], a[i] = a[i], a[j]
    return a, counter


def random_layout(N: int, G: int, I: int, L: int, seed: int):
    """Seeded balanced layouts (the random baseline of Section 4): for each layer in turn,
    the contiguous h is shuffled, then the contiguous nu, drawing from one generator."""
    hs, nus = [], []
    c = 0
    for _ in range(N):
        h, c = _shuffle(contiguous_heads(G, L), seed, c)
        nu, c = _shuffle(contiguous_neurons(I, L), seed, c)
        hs.append(np.array(h, dtype=np.int64))
        nus.append(np.array(nu, dtype=np.int64))
    return hs, nus


# ----------------------------------------------------------------------------- exact optimum
def unlabelled_partitions(G: int, L: int) -> list:
    """One labelled representative per balanced partition up to device relabelling: the
    ones whose labels first appear in the order 0, 1, ..., L-1."""
    out = []
    for h in partitions(G, L):
        firsts = [h.index(l) for l in range(L)]
        if firsts == sorted(firsts):
            out.append(h)
    return out


def layer_optimum(Q_up: np.ndarray, L: int):
    """(h, nu, J_int) maximising one layer's co-located up mass exactly.

    With no neighbours, relabelling devices maps optima to optima, so it suffices to take
    every unlabelled head partition with its exact neuron assignment; the first partition
    (lexicographic) that attains the maximum is returned with its canonical assignment.
    """
    G, _ = Q_up.shape
    best = None
    for h in unlabelled_partitions(G, L):
        nu, val = balanced_assign(neuron_gain(Q_up, h, L))
        if best is None or val > best[2]:
            best = (tuple(h), nu, val)
    return best
