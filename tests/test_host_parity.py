"""Host-side library logic against the oracle, bit for bit: the unit-mass encoder, the
partition enumeration and the exact neuron assignment (these parts of the path run on
the host by design; no GPU is involved)."""
import numpy as np
import pytest

from oracle import dual_ascent as da
from oracle import layout as lay
from paper_2609_13846_amd import dtp


def rand_A(rng, shape, kind="gamma"):
    if kind == "gamma":
        return rng.gamma(0.4, size=shape).astype(np.float32) * np.float32(3e-3)
    if kind == "wide":
        return np.exp(rng.uniform(-60, 20, size=shape)).astype(np.float32)
    return rng.random(shape).astype(np.float32)


@pytest.mark.parametrize("shape,kind", [((4, 128), "gamma"), ((8, 3072), "gamma"),
                                        ((8, 4096), "wide"), ((3, 7), "uniform")])
def test_encode_bit_exact(shape, kind):
    rng = np.random.default_rng(sum(shape))
    A = rand_A(rng, shape, kind)
    A.ravel()[::13] = 0.0
    np.testing.assert_array_equal(dtp.dtp_encode_affinity(A), lay.encode(A))


@pytest.mark.parametrize("G,L", [(4, 2), (8, 2), (8, 4), (6, 3), (8, 8), (8, 1), (12, 4)])
def test_partitions_match_oracle(G, L):
    parts = lay.partitions(G, L) if (G, L) != (12, 4) else None
    P = dtp.dtp_partition_count(G, L)
    if parts is not None:
        assert P == len(parts)
        for r in list(range(min(P, 50))) + [P - 1, P // 2]:
            assert tuple(dtp.dtp_partition_unrank(G, L, r)) == parts[r]
    else:
        assert P == 369600
        prev = None
        for r in [0, 1, 2, 1000, P - 1]:
            h = tuple(dtp.dtp_partition_unrank(G, L, r))
            assert all(h.count(l) == G // L for l in range(L))
            assert prev is None or h > prev
            prev = h


CASES = [  # G, I, L, down, minimise
    (4, 8, 2, False, False), (4, 128, 2, False, False), (8, 3072, 2, False, False),
    (8, 64, 4, False, False), (8, 512, 4, True, False), (8, 3072, 4, False, False),
    (8, 3072, 4, True, False), (8, 96, 8, True, False), (6, 60, 3, True, False),
    (8, 256, 4, True, True), (8, 64, 1, True, False),
]


@pytest.mark.parametrize("G,I,L,down,minimise", CASES)
def test_balanced_assign_bit_exact(G, I, L, down, minimise):
    rng = np.random.default_rng(G * 1000 + I + L)
    Qu = lay.encode(rand_A(rng, (G, I)))
    Qd = lay.encode(rand_A(rng, (I, G))) if down else None
    h = rng.permutation(np.arange(G) // (G // L))
    hn = rng.permutation(np.arange(G) // (G // L)) if down else None
    nu, v = dtp.dtp_balanced_assign(G, I, L, Qu, h, Qd, hn, minimise)
    M = lay.neuron_gain(Qu, h, L, Qd, hn)
    onu, ov = lay.balanced_assign(M, minimise)
    assert v == ov
    np.testing.assert_array_equal(nu, onu)


@pytest.mark.parametrize("I,L", [(12, 4), (64, 4), (40, 2), (48, 8)])
def test_balanced_assign_ties_bit_exact(I, L):
    rng = np.random.default_rng(I * L)
    G = 8
    for trial in range(4):
        Qu = rng.integers(0, 3, size=(G, I)).astype(np.int64) << 40   # many equal gains
        h = rng.permutation(np.arange(G) // (G // L))
        nu, v = dtp.dtp_balanced_assign(G, I, L, Qu, h)
        onu, ov = lay.balanced_assign(lay.neuron_gain(Qu, h, L))
        assert v == ov
        np.testing.assert_array_equal(nu, onu)
    Z = np.zeros((G, I), np.int64)
    nu, v = dtp.dtp_balanced_assign(G, I, L, Z, np.arange(G) // (G // L))
    np.testing.assert_array_equal(nu, np.arange(I) // (I // L))


@pytest.mark.parametrize("G,I,L,down,minimise", CASES)
def test_dual_ascent_assign_bit_exact(G, I, L, down, minimise):
    """The paper's approximate neuron step, library against oracle, bit for bit."""
    rng = np.random.default_rng(G * 1000 + I + L + 7)
    Qu = lay.encode(rand_A(rng, (G, I)))
    Qd = lay.encode(rand_A(rng, (I, G))) if down else None
    h = rng.permutation(np.arange(G) // (G // L))
    hn = rng.permutation(np.arange(G) // (G // L)) if down else None
    nu, v = dtp.dtp_balanced_assign_dual_ascent(G, I, L, Qu, h, Qd, hn, minimise)
    M = lay.neuron_gain(Qu, h, L, Qd, hn)
    onu, ov = da.assign(-M if minimise else M)
    np.testing.assert_array_equal(nu, onu)
    assert v == (-ov if minimise else ov)
    assert v == int(M[np.arange(I), onu].sum())
    _, vopt = lay.balanced_assign(M, minimise)
    assert (v >= vopt) if minimise else (v <= vopt)
    if L == 2:
        assert v == vopt


@pytest.mark.parametrize("I,L", [(12, 4), (64, 4), (40, 2), (48, 8)])
def test_dual_ascent_ties_bit_exact(I, L):
    rng = np.random.default_rng(I * L + 1)
    G = 8
    for trial in range(4):
        Qu = rng.integers(0, 3, size=(G, I)).astype(np.int64) << 40   # many equal gains
        h = rng.permutation(np.arange(G) // (G // L))
        nu, v = dtp.dtp_balanced_assign_dual_ascent(G, I, L, Qu, h)
        onu, ov = da.assign(lay.neuron_gain(Qu, h, L))
        assert v == ov
        np.testing.assert_array_equal(nu, onu)


# ----------------------------------------------------------------------------- random layouts
@pytest.mark.parametrize("N,G,I,L,seed", [(1, 8, 64, 4, 1000), (3, 8, 3072, 2, 1007),
                                           (2, 4, 128, 2, 0), (2, 16, 96, 8, 2 ** 64 - 1)])
def test_random_layout_bit_exact(N, G, I, L, seed):
    h, nu = dtp.dtp_random_layout(N, G, I, L, seed)
    hs, nus = lay.random_layout(N, G, I, L, seed)
    np.testing.assert_array_equal(h, np.array(hs))
    np.testing.assert_array_equal(nu, np.array(nus))


# ----------------------------------------------------------------------------- objective
@pytest.mark.parametrize("down", [False, True])
def test_layout_objective_bit_exact(down):
    rng = np.random.default_rng(41)
    N, G, I, L = 3, 8, 256, 4
    Qu = [lay.encode(rand_A(rng, (G, I))) for _ in range(N)]
    Qd = [lay.encode(rand_A(rng, (I, G))) for _ in range(N - 1)] if down else None
    hs, nus = lay.random_layout(N, G, I, L, 5)
    J = dtp.dtp_layout_objective(N, G, I, L, np.stack(Qu), None if Qd is None else np.stack(Qd),
                                 np.array(hs), np.array(nus))
    assert J == lay.objective(Qu, Qd, hs, nus)


def test_layout_objective_rejects_unbalanced():
    G, I, L = 4, 8, 2
    Q = lay.encode(rand_A(np.random.default_rng(0), (G, I)))
    with pytest.raises(dtp.DtpError):
        dtp.dtp_layout_objective(1, G, I, L, Q, None, np.array([[0, 0, 0, 1]]), np.zeros((1, I)))


# ----------------------------------------------------------------------------- exact optimum
@pytest.mark.parametrize("G,I,L,seed", [(8, 64, 4, 51), (8, 128, 2, 52), (4, 16, 2, 53), (6, 24, 3, 54)])
def test_layer_optimum_bit_exact(G, I, L, seed):
    rng = np.random.default_rng(seed)
    Q = lay.encode(rand_A(rng, (G, I)))
    h, nu, J = dtp.dtp_layer_optimum(G, I, L, Q)
    rh, rnu, rJ = lay.layer_optimum(Q, L)
    assert J == rJ
    np.testing.assert_array_equal(h, np.array(rh))
    np.testing.assert_array_equal(nu, rnu)


# ----------------------------------------------------------------------------- layout orders
def test_layout_orders_match_oracle():
    from oracle import apply as ap
    for (G, I, L, seed) in [(8, 64, 4, 3), (4, 128, 2, 9), (16, 32, 8, 1)]:
        hs, nus = lay.random_layout(1, G, I, L, seed)
        go, no = dtp.dtp_layout_orders(G, I, L, hs[0], nus[0])
        rgo, rno = ap.layout_orders(hs[0], nus[0], L)
        np.testing.assert_array_equal(go, rgo)
        np.testing.assert_array_equal(no, rno)
    with pytest.raises(dtp.DtpError):
        dtp.dtp_layout_orders(4, 8, 2, np.array([0, 0, 0, 1]), np.zeros(8))
