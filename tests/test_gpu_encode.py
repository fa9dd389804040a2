"""The unit-mass fixed-point codes computed on the GPU against the oracle's, bit for bit
(Section 3, "Objective": every affinity matrix is normalised to unit mass).

The oracle computes the codes with Python integers; the device path reduces the maximum,
the first bad index and the 128-bit sum with integer atomics and divides with an fp64
estimate plus an exact correction, so any difference is a bug, not rounding.
"""
import sys

import numpy as np
import pytest
import torch

from oracle import layout as lay
from paper_2609_13846_amd import dtp

pytestmark = pytest.mark.gpu


def announce(msg):
    print(f"[gpu] {msg}", file=sys.stderr, flush=True)


def device_codes(A):
    a = torch.from_numpy(np.ascontiguousarray(A, dtype=np.float32)).cuda()
    q = torch.zeros(a.shape, dtype=torch.int64, device=a.device)
    dtp.dtp_encode_affinity_device(a, q)
    return q.cpu().numpy()


def _cases():
    rng = np.random.default_rng(2609)
    yield "one entry", np.array([3.5], np.float32)
    yield "ragged 255", (rng.gamma(0.4, size=255) * 1e-3).astype(np.float32)
    yield "qwen up edge 8x3072", (rng.gamma(0.4, size=(8, 3072)) * 1e-3).astype(np.float32)
    # entries from 1e-30 to 1e30: most truncate to zero, several are subnormal
    wide = np.exp(rng.uniform(np.log(1e-45), np.log(1e30), size=4099)).astype(np.float32)
    yield "wide range with subnormals", wide
    pw = np.ldexp(1.0, rng.integers(-60, 20, size=1000)).astype(np.float32)
    yield "powers of two", pw
    z = (rng.random(3000) * 7).astype(np.float32)
    z[::3] = 0.0
    z[1::7] = -0.0
    yield "zeros and negative zeros", z
    yield "all equal", np.full(4096 * 3 + 17, 0.25, np.float32)
    yield "2^20 + 3 entries", rng.random((1 << 20) + 3).astype(np.float32) ** 4


@pytest.mark.parametrize("name,A", list(_cases()), ids=[c[0] for c in _cases()])
def test_device_codes_equal_the_oracle(name, A):
    announce(f"device encode: {name}, n={A.size}")
    Q = device_codes(A)
    np.testing.assert_array_equal(Q, lay.encode(A))
    assert Q.sum() <= 1 << 48 and Q.sum() > (1 << 48) - A.size


def test_device_codes_equal_the_host_codes():
    announce("device encode against dtp_encode_affinity")
    rng = np.random.default_rng(7)
    A = (rng.gamma(0.2, size=(8, 14336)) * 1e-4).astype(np.float32)
    np.testing.assert_array_equal(device_codes(A), dtp.dtp_encode_affinity(A))


@pytest.mark.parametrize("bad,index", [(np.nan, 5), (np.inf, 4095), (-1e-20, 70000), (-np.inf, 0)])
def test_device_encode_rejects_bad_entries(bad, index):
    announce(f"device encode rejects {bad} at {index}")
    A = np.ones(70001, np.float32)
    A[index] = bad
    A[index + 1 if index + 1 < A.size else 0] = np.nan  # the first bad index is reported
    with pytest.raises(dtp.DtpError) as e:
        device_codes(A)
    assert e.value.status == dtp.DTP_ERR_DEGENERATE
    assert f"entry {min(index, index + 1 if index + 1 < A.size else 0)}" in str(e.value)


@pytest.mark.parametrize("A", [np.zeros(1000, np.float32), np.full(513, -0.0, np.float32)],
                         ids=["zeros", "negative zeros"])
def test_device_encode_rejects_all_zero(A):
    announce("device encode rejects an all-zero matrix")
    with pytest.raises(dtp.DtpError) as e:
        device_codes(A)
    assert e.value.status == dtp.DTP_ERR_DEGENERATE
    assert "all zero" in str(e.value)


def test_coordinate_ascent_rejects_degenerate_matrices():
    announce("coordinate ascent rejects a NaN up matrix and a negative down matrix")
    rng = np.random.default_rng(3)
    N, G, I, L = 3, 8, 256, 2
    up = torch.from_numpy(rng.random((N, G, I)).astype(np.float32)).cuda()
    down = torch.from_numpy(rng.random((N - 1, I, G)).astype(np.float32)).cuda()
    bad_up = up.clone()
    bad_up[2, 1, 7] = float("nan")
    with pytest.raises(dtp.DtpError) as e:
        dtp.dtp_coordinate_ascent(N, G, I, L, bad_up, A_down=down)
    assert e.value.status == dtp.DTP_ERR_DEGENERATE and "up affinity of layer 2" in str(e.value)
    bad_down = down.clone()
    bad_down[1].zero_()
    with pytest.raises(dtp.DtpError) as e:
        dtp.dtp_coordinate_ascent(N, G, I, L, up, A_down=bad_down)
    assert e.value.status == dtp.DTP_ERR_DEGENERATE and "down affinity of layer 1" in str(e.value)
    res = dtp.dtp_coordinate_ascent(N, G, I, L, up, A_down=down)
    assert res["sweeps"] >= 1
