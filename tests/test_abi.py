"""The C ABI: the library loads on a machine without a GPU, exports every declared
symbol, and rejects bad arguments on the host before any GPU work (no compute call on
the GPU is made here)."""
import ctypes

import numpy as np
import pytest

from paper_2609_13846_amd import dtp


def test_library_exports_every_declared_symbol():
    lib = dtp.lib()
    names = dtp.header_symbols()
    assert len(names) >= 14
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(dtp._SIGNATURES)


def test_status_strings():
    lib = dtp.lib()
    for code, name in [(0, "DTP_OK"), (-1, "DTP_ERR_INVALID_ARG"), (-2, "DTP_ERR_UNSUPPORTED"),
                       (-3, "DTP_ERR_DEGENERATE"), (-4, "DTP_ERR_NO_MEMORY"), (-5, "DTP_ERR_HIP")]:
        assert lib.dtp_status_string(code).decode() == name


def _expect(status, fn, *a, **k):
    with pytest.raises(dtp.DtpError) as e:
        fn(*a, **k)
    assert e.value.status == status, str(e.value)
    assert str(e.value)


@pytest.mark.parametrize("bad", [
    dict(d_model=0), dict(n_neurons=-1), dict(n_q_heads=6, n_kv_groups=4),
    dict(head_dim=24), dict(rms_eps=-1.0), dict(rms_eps=float("nan")),
    # d_model must be a multiple of 16 (rows are read in 16-element pieces)
    dict(d_model=72), dict(d_model=24), dict(d_model=8), dict(d_model=1000),
])
def test_layer_create_rejects_bad_shapes(bad):
    kw = dict(d_model=64, n_neurons=128, n_q_heads=8, n_kv_groups=4, head_dim=16, rms_eps=1e-6,
              dtype=dtp.DTP_BF16)
    kw.update(bad)
    _expect(dtp.DTP_ERR_INVALID_ARG, dtp.dtp_layer_create, **kw)


@pytest.mark.parametrize("bad", [dict(dtype=7), dict(n_kv_groups=64, n_q_heads=64)])
def test_layer_create_unsupported(bad):
    kw = dict(d_model=64, n_neurons=128, n_q_heads=8, n_kv_groups=4, head_dim=16, rms_eps=1e-6,
              dtype=dtp.DTP_BF16)
    kw.update(bad)
    _expect(dtp.DTP_ERR_UNSUPPORTED, dtp.dtp_layer_create, **kw)


def test_null_layer_arguments():
    lib = dtp.lib()
    assert lib.dtp_layer_create(None, None) == dtp.DTP_ERR_INVALID_ARG
    assert lib.dtp_layer_destroy(None) == dtp.DTP_OK
    assert lib.dtp_layer_set_weights(None, 1, 1, 1, 1, 1, None) == dtp.DTP_ERR_INVALID_ARG
    assert lib.dtp_affinity_accumulate(None, 1, 1, 10, 1, None) == dtp.DTP_ERR_INVALID_ARG
    assert lib.dtp_layer_profile(None, 1) == dtp.DTP_ERR_INVALID_ARG
    assert "NULL" in lib.dtp_last_error().decode()


def test_partition_count_and_unrank_arguments():
    assert dtp.dtp_partition_count(8, 4) == 2520
    assert dtp.dtp_partition_count(8, 3) == -1
    assert dtp.dtp_partition_count(65, 5) == -1
    assert dtp.dtp_partition_count(0, 1) == -1
    assert dtp.dtp_partition_count(64, 4) == -1   # beyond 2^62
    _expect(dtp.DTP_ERR_INVALID_ARG, dtp.dtp_partition_unrank, 8, 4, 2520)
    _expect(dtp.DTP_ERR_INVALID_ARG, dtp.dtp_partition_unrank, 8, 4, -1)
    _expect(dtp.DTP_ERR_INVALID_ARG, dtp.dtp_partition_unrank, 8, 3, 0)


def test_encode_arguments():
    _expect(dtp.DTP_ERR_DEGENERATE, dtp.dtp_encode_affinity, np.zeros(5, np.float32))
    _expect(dtp.DTP_ERR_DEGENERATE, dtp.dtp_encode_affinity, np.array([1, -1], np.float32))
    _expect(dtp.DTP_ERR_DEGENERATE, dtp.dtp_encode_affinity, np.array([1, np.inf], np.float32))
    _expect(dtp.DTP_ERR_DEGENERATE, dtp.dtp_encode_affinity, np.array([np.nan], np.float32))
    lib = dtp.lib()
    assert lib.dtp_encode_affinity(None, 4, None) == dtp.DTP_ERR_INVALID_ARG
    a = np.ones(4, np.float32)
    q = np.zeros(4, np.int64)
    assert lib.dtp_encode_affinity(a.ctypes.data, 0, q.ctypes.data) == dtp.DTP_ERR_INVALID_ARG


@pytest.mark.parametrize("fn", ["dtp_balanced_assign", "dtp_balanced_assign_dual_ascent"])
def test_balanced_assign_arguments(fn):
    Q = np.ones((8, 16), np.int64)
    h = np.arange(8) // 2
    assign = getattr(dtp, fn)
    _expect(dtp.DTP_ERR_INVALID_ARG, assign, 8, 15, 4, Q, h)          # I % L
    _expect(dtp.DTP_ERR_INVALID_ARG, assign, 8, 16, 3, Q, h)          # G % L
    _expect(dtp.DTP_ERR_INVALID_ARG, assign, 8, 16, 4, Q, np.zeros(8))  # unbalanced
    _expect(dtp.DTP_ERR_INVALID_ARG, assign, 8, 16, 4, Q, h + 4)      # not a device
    _expect(dtp.DTP_ERR_UNSUPPORTED, assign, 16, 16, 16, np.ones((16, 16), np.int64),
            np.arange(16))                                                                  # L > 8
    _expect(dtp.DTP_ERR_INVALID_ARG, assign, 8, 16, 4, Q, h, Q_down=Q.T.copy())
    lib = dtp.lib()
    v = ctypes.c_int64()
    assert getattr(lib, fn)(8, 16, 4, None, None, None, None, 0, None, ctypes.byref(v)) == \
        dtp.DTP_ERR_INVALID_ARG


def test_device_encode_arguments_checked_before_gpu():
    lib = dtp.lib()
    assert lib.dtp_encode_affinity_device(None, 5, 1, None) == dtp.DTP_ERR_INVALID_ARG
    assert lib.dtp_encode_affinity_device(1, 5, None, None) == dtp.DTP_ERR_INVALID_ARG
    assert lib.dtp_encode_affinity_device(1, 0, 1, None) == dtp.DTP_ERR_INVALID_ARG
    assert lib.dtp_encode_affinity_device(1, (1 << 30) + 1, 1, None) == dtp.DTP_ERR_INVALID_ARG


def test_partition_scores_and_ascent_arguments_checked_before_gpu():
    lib = dtp.lib()
    best = ctypes.c_int64()
    assert lib.dtp_partition_scores(8, 16, 3, 1, 1, None, None, 0, 1, ctypes.byref(best), None) == \
        dtp.DTP_ERR_INVALID_ARG
    assert lib.dtp_partition_scores(8, 16, 4, None, 1, None, None, 0, 1, ctypes.byref(best), None) == \
        dtp.DTP_ERR_INVALID_ARG
    assert lib.dtp_partition_scores(8, 16, 4, 1, 1, 1, None, 0, 1, ctypes.byref(best), None) == \
        dtp.DTP_ERR_INVALID_ARG
    _expect(dtp.DTP_ERR_INVALID_ARG, dtp.dtp_coordinate_ascent, 0, 8, 16, 4, 1)
    _expect(dtp.DTP_ERR_INVALID_ARG, dtp.dtp_coordinate_ascent, 2, 8, 18, 4, 1)
    _expect(dtp.DTP_ERR_INVALID_ARG, dtp.dtp_coordinate_ascent, 1, 8, 16, 4, 1, A_down=1)
    _expect(dtp.DTP_ERR_INVALID_ARG, dtp.dtp_coordinate_ascent, 2, 8, 16, 4, 1, max_sweeps=0)
    _expect(dtp.DTP_ERR_UNSUPPORTED, dtp.dtp_coordinate_ascent, 2, 32, 32, 16, 1)


# ----------------------------------------------------------------------------- binding checks
# The wrappers check every device argument before the library sees it: a contiguous torch
# tensor on the GPU, of the right dtype, with enough elements.  These checks run on the
# host, so CPU tensors and numpy arrays exercise them here without a GPU.
def test_device_argument_must_be_a_gpu_tensor():
    import torch
    with pytest.raises(TypeError, match="torch tensor"):
        dtp.dtp_coordinate_ascent(1, 8, 16, 4, np.ones((8, 16), np.float32))
    with pytest.raises(ValueError, match="on the GPU"):
        dtp.dtp_coordinate_ascent(1, 8, 16, 4, torch.ones(8, 16))
    with pytest.raises(ValueError, match="on the GPU"):
        dtp.dtp_down_affinity(16, 8, torch.ones(16), torch.ones(8, 16), torch.ones(16, 8))
    with pytest.raises(ValueError, match="on the GPU"):
        dtp.dtp_encode_affinity_device(torch.ones(4), torch.zeros(4, dtype=torch.int64))


def test_device_argument_dtype_and_size_checked():
    import torch
    t = torch.ones(10)
    with pytest.raises(ValueError, match="on the GPU"):
        dtp._dev(t, "A", ("float32",), 10)

    class FakeCuda(torch.Tensor):   # a CPU tensor that claims to be on the GPU
        @property
        def is_cuda(self):
            return True
    f32 = torch.ones(10).as_subclass(FakeCuda)
    assert dtp._dev(f32, "A", ("float32",), 10) == f32.data_ptr()
    with pytest.raises(ValueError, match="has 10 elements"):
        dtp._dev(f32, "A", ("float32",), 11)
    with pytest.raises(TypeError, match="dtype"):
        dtp._dev(f32, "A", ("bfloat16",), 10)
    with pytest.raises(ValueError, match="contiguous"):
        dtp._dev(torch.ones(4, 4).t().as_subclass(FakeCuda), "A", ("float32",), 16)
    assert dtp._dev(None, "A_down", ("float32",), 0, optional=True) is None
    with pytest.raises(ValueError, match="required"):
        dtp._dev(None, "A", ("float32",), 1)
    assert dtp._dev(12345, "A", ("float32",), 1) == 12345   # raw address: the library checks it


def test_layer_mask_must_have_one_entry_per_layer():
    with pytest.raises(ValueError, match="layer_mask has 3 elements, expected 4"):
        dtp.dtp_coordinate_ascent(4, 8, 16, 4, 1, layer_mask=[1, 0, 1])


def test_layer_wrappers_reject_unknown_handles():
    with pytest.raises(ValueError, match="layer handle"):
        dtp.dtp_affinity_accumulate(123456, 1, 1, 10, 1)


def test_noalloc_down_weights_refuses_more_than_its_scratch_before_any_gpu_work():
    """8 * 65536 * ceil(6 * 128 / 128) partial sums exceed the 2^20 of the fixed scratch:
    refused from the shapes alone (raw addresses, no GPU needed)."""
    lib = dtp.lib()
    st = lib.dtp_down_weights_noalloc(64, 65536, 32, 8, 128, dtp.DTP_BF16, 16, 16, 16, 16, 16, 16, None)
    assert st == dtp.DTP_ERR_UNSUPPORTED
    assert "allocation-free scratch" in lib.dtp_last_error().decode()
    # the allocating entry point has no such limit (it fails later, on the fake addresses)
    assert lib.dtp_down_weights(64, 65536, 32, 8, 128, dtp.DTP_BF16, 16, 16, 16, 16, 16, 16, None) != \
        dtp.DTP_ERR_UNSUPPORTED
