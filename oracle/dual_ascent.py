"""The paper's approximate neuron assignment (test infrastructure only).

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s ``cpu_baseline`` leg may
import this module.  It shares no code with the HIP library.

Section 3, "Optimiser", and the appendix's hyper-parameters: the balanced neuron
assignment (I/L slots per device) is solved by dual ascent on L device offsets, then a
fix-up that meets the capacities exactly, then pairwise swaps until no swap improves; the
dual ascent runs 300 iterations with a step that decays by 0.98 per iteration.  The exact
solver (``layout.balanced_assign``) is what the library's coordinate ascent uses; this
heuristic is kept to measure how far the paper's method is from the optimum.

Readings (the paper does not fix these; each is listed in the design notes):

* offsets start at zero; each iteration assigns every neuron to argmax_l (M_kl - lambda_l)
  (lowest l on ties), then raises the offset of every device by step * (n_l - I/L), where
  n_l is its load: overloaded devices become dearer;
* the first step is (max M - min M) / I, a full range of gains spread over the neurons;
  M is taken in fp64, exact while its entries stay below 2^53;
* fix-up: from the last iteration's assignment, move one neuron at a time from an
  overloaded device to an underloaded one, choosing the move that loses the least gain
  (smallest neuron index, then smallest device, on ties), until every device holds I/L;
* swaps: scan the device pairs (a, b), a < b, in order; for each, exchange the neuron of a
  that gains most by moving to b with the neuron of b that gains most by moving to a
  (smallest indices on ties) when the sum of the two gains is positive; repeat the scan
  until a whole scan exchanges nothing.

With L = 2 a balanced assignment that no swap improves is optimal (every improving cycle
of moves between two devices is a set of swaps), so the heuristic then returns the exact
optimum value.  Parity with the paper's own runs is unpinned: its first step size is not
given.
"""
from __future__ import annotations

import numpy as np

ITERATIONS = 300
DECAY = 0.98


def dual_offsets(M: np.ndarray, iterations: int = ITERATIONS, decay: float = DECAY) -> np.ndarray:
    """(lambda [L], nu [I]): offsets after the dual ascent and the assignment they induce."""
    I, L = M.shape
    cap = I // L
    gains = M.astype(np.float64)
    lam = np.zeros(L)
    step = (gains.max() - gains.min()) / I
    nu = np.argmax(gains - lam[None, :], axis=1)
    for _ in range(iterations):
        nu = np.argmax(gains - lam[None, :], axis=1)
        load = np.bincount(nu, minlength=L)
        for l in range(L):
            lam[l] = lam[l] + step * float(load[l] - cap)
        step = step * decay
    nu = np.argmax(gains - lam[None, :], axis=1)
    return lam, nu.astype(np.int64)


def fix_up(M: np.ndarray, nu: np.ndarray) -> np.ndarray:
    """Cheapest single moves from overloaded to underloaded devices until balanced."""
    I, L = M.shape
    cap = I // L
    nu = np.array(nu, dtype=np.int64)
    load = np.bincount(nu, minlength=L)
    while np.any(load > cap):
        movable = np.flatnonzero(load[nu] > cap)           # increasing neuron index
        targets = np.flatnonzero(load < cap)               # increasing device index
        loss = M[movable, nu[movable]][:, None] - M[np.ix_(movable, targets)]
        flat = int(np.argmin(loss))                        # first minimum: smallest k, then b
        k = movable[flat // len(targets)]
        b = targets[flat % len(targets)]
        load[nu[k]] -= 1
        load[b] += 1
        nu[k] = b
    return nu


def pairwise_swaps(M: np.ndarray, nu: np.ndarray) -> np.ndarray:
    """Best exchange per device pair, scanned in order, until a scan changes nothing."""
    _, L = M.shape
    nu = np.array(nu, dtype=np.int64)
    changed = True
    while changed:
        changed = False
        for a in range(L):
            for b in range(a + 1, L):
                on_a = np.flatnonzero(nu == a)
                on_b = np.flatnonzero(nu == b)
                if len(on_a) == 0 or len(on_b) == 0:
                    continue
                to_b = M[on_a, b] - M[on_a, a]
                to_a = M[on_b, a] - M[on_b, b]
                i = int(np.argmax(to_b))
                j = int(np.argmax(to_a))
                if int(to_b[i]) + int(to_a[j]) > 0:
                    nu[on_a[i]] = b
                    nu[on_b[j]] = a
                    changed = True
    return nu


def assign(M: np.ndarray, iterations: int = ITERATIONS, decay: float = DECAY):
    """(nu [I] int64, value): dual ascent, fix-up, pairwise swaps.  M is [I, L] int64."""
    M = np.asarray(M, dtype=np.int64)
    _, nu = dual_offsets(M, iterations, decay)
    nu = fix_up(M, nu)
    nu = pairwise_swaps(M, nu)
    return nu, int(M[np.arange(M.shape[0]), nu].sum())
