"""ctypes binding of libdtp.so (declared in include/dtp.h), one Python function per C entry point.

The functions carry the C names and only marshal arguments: device tensors are passed
as ``tensor.data_ptr()`` together with the current HIP stream, host arrays as numpy
buffers.  Every computation runs in the library.  A non-OK status raises ``DtpError``
with the library's message.  If ``libdtp.so`` has not been built, loading fails loudly:
there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
import re

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdtp.so")
HEADER = os.path.join(os.path.dirname(_HERE), "include", "dtp.h")

DTP_BF16 = 0
DTP_F32 = 1
DTP_OK, DTP_ERR_INVALID_ARG, DTP_ERR_UNSUPPORTED, DTP_ERR_DEGENERATE, DTP_ERR_NO_MEMORY, DTP_ERR_HIP = (
    0, -1, -2, -3, -4, -5)


class DtpError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(message)
        self.status = status


class dtp_layer_desc(ctypes.Structure):
    _fields_ = [("d_model", ctypes.c_int32), ("n_neurons", ctypes.c_int32),
                ("n_q_heads", ctypes.c_int32), ("n_kv_groups", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("rms_eps", ctypes.c_float),
                ("dtype", ctypes.c_int32)]


class dtp_ca_options(ctypes.Structure):
    _fields_ = [("max_sweeps", ctypes.c_int32), ("freeze_heads", ctypes.c_int32),
                ("freeze_neurons", ctypes.c_int32), ("minimise", ctypes.c_int32),
                ("layer_mask", ctypes.c_void_p), ("dual_ascent_neurons", ctypes.c_int32)]


_P = ctypes.c_void_p
_I32 = ctypes.c_int32
_I64 = ctypes.c_int64
_SIGNATURES = {
    "dtp_layer_create": (_I32, [ctypes.POINTER(dtp_layer_desc), ctypes.POINTER(_P)]),
    "dtp_layer_destroy": (_I32, [_P]),
    "dtp_layer_set_weights": (_I32, [_P, _P, _P, _P, _P, _P, _P]),
    "dtp_affinity_accumulate": (_I32, [_P, _P, _P, _I64, _P, _P]),
    "dtp_layout_orders": (_I32, [_I32, _I32, _I32, _P, _P, _P, _P]),
    "dtp_apply_layout": (_I32, [ctypes.POINTER(dtp_layer_desc), _I32, _P, _P, _P, _P, _P]),
    "dtp_affinity_accumulate_add": (_I32, [_P, _P, _P, _I64, _P, _P]),
    "dtp_random_layout": (_I32, [_I32, _I32, _I32, _I32, ctypes.c_uint64, _P, _P]),
    "dtp_layout_objective": (_I32, [_I32, _I32, _I32, _I32, _P, _P, _P, _P, ctypes.POINTER(_I64)]),
    "dtp_layer_optimum": (_I32, [_I32, _I32, _I32, _P, _P, _P, ctypes.POINTER(_I64)]),
    "dtp_affinity_accumulate_down": (_I32, [_P, _P, _P, _P, ctypes.c_float, _I64, _P, _P, _P]),
    "dtp_down_weights": (_I32, [_I32, _I32, _I32, _I32, _I32, _I32, _P, _P, _P, _P, _P, _P, _P]),
    "dtp_down_weights_noalloc": (_I32, [_I32, _I32, _I32, _I32, _I32, _I32, _P, _P, _P, _P, _P, _P, _P]),
    "dtp_down_affinity": (_I32, [_I32, _I32, _P, _P, _P, _P]),
    "dtp_layer_profile": (_I32, [_P, _I32]),
    "dtp_layer_profile_read": (_I32, [_P, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(_I64)]),
    "dtp_partition_count": (_I64, [_I32, _I32]),
    "dtp_partition_unrank": (_I32, [_I32, _I32, _I64, _P]),
    "dtp_encode_affinity": (_I32, [_P, _I64, _P]),
    "dtp_encode_affinity_device": (_I32, [_P, _I64, _P, _P]),
    "dtp_partition_scores": (_I32, [_I32, _I32, _I32, _P, _P, _P, _P, _I32, _P, ctypes.POINTER(_I64), _P]),
    "dtp_balanced_assign": (_I32, [_I32, _I32, _I32, _P, _P, _P, _P, _I32, _P, ctypes.POINTER(_I64)]),
    "dtp_balanced_assign_dual_ascent": (_I32, [_I32, _I32, _I32, _P, _P, _P, _P, _I32, _P,
                                               ctypes.POINTER(_I64)]),
    "dtp_coordinate_ascent": (_I32, [_I32, _I32, _I32, _I32, _P, _P, ctypes.POINTER(dtp_ca_options),
                                     _P, _P, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(_I64),
                                     ctypes.POINTER(_I32), _P]),
    "dtp_status_string": (ctypes.c_char_p, [_I32]),
    "dtp_last_error": (ctypes.c_char_p, []),
}

_lib = None


def lib() -> ctypes.CDLL:
    """The loaded library; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise DtpError(DTP_ERR_UNSUPPORTED, f"{LIB_PATH} is missing: build it with "
                           "`python -m paper_2609_13846_amd.build` (there is no fallback)")
        l = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _SIGNATURES.items():
            fn = getattr(l, name)
            fn.restype = res
            fn.argtypes = args
        _lib = l
    return _lib


def header_symbols() -> list:
    """Names of the functions include/dtp.h declares."""
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dtp_[a-z_]+)\s*\(", text)))


def _check(status: int):
    if status != DTP_OK:
        l = lib()
        raise DtpError(status, f"{l.dtp_status_string(status).decode()}: {l.dtp_last_error().decode()}")


def _ptr(x):
    """Address of a torch tensor, a numpy array, an int or None."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if isinstance(x, np.ndarray):
        if not x.flags["C_CONTIGUOUS"]:
            raise ValueError("numpy arrays must be C-contiguous")
        return x.ctypes.data
    if hasattr(x, "data_ptr"):
        if not x.is_contiguous():
            raise ValueError("tensors must be contiguous")
        return x.data_ptr()
    raise TypeError(f"cannot pass {type(x)!r} as a pointer")


def _dev(t, name, dtypes, numel, optional=False):
    """Address of a device argument after checking it: a contiguous torch tensor on the
    GPU, of one of ``dtypes`` (torch dtype names), with at least ``numel`` elements.  A
    plain int is taken as a raw device address (the library still checks that it is
    device memory large enough for the call)."""
    if t is None:
        if optional:
            return None
        raise ValueError(f"{name} is required")
    if isinstance(t, int):
        return t
    import torch
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor on the GPU, not {type(t).__name__}")
    if not t.is_cuda:
        raise ValueError(f"{name} must be on the GPU (got a tensor on {t.device})")
    if str(t.dtype).replace("torch.", "") not in dtypes:
        raise TypeError(f"{name} must have dtype {' or '.join(dtypes)}, not {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.numel() < numel:
        raise ValueError(f"{name} has {t.numel()} elements, the call needs {numel}")
    return t.data_ptr()


def _act_dtypes(dtype):
    return ("bfloat16",) if dtype == DTP_BF16 else ("float32",)


def _host(a, name, dtype, n):
    """A host array argument of exactly n elements (converted to ``dtype``)."""
    a = np.ascontiguousarray(a, dtype=dtype)
    if a.size != n:
        raise ValueError(f"{name} has {a.size} elements, expected {n}")
    return a


def _stream(stream):
    if stream is not None:
        return stream if isinstance(stream, int) else stream.cuda_stream
    import torch
    if torch.cuda.is_available() and torch.cuda.is_initialized():
        return torch.cuda.current_stream().cuda_stream
    return None


# ----------------------------------------------------------------------------- affinity
# Shapes of the layers created through this module, by handle: what each wrapper checks
# its device arguments against.
_LAYERS = {}


def dtp_layer_create(d_model, n_neurons, n_q_heads, n_kv_groups, head_dim, rms_eps, dtype):
    desc = dtp_layer_desc(d_model, n_neurons, n_q_heads, n_kv_groups, head_dim, rms_eps, dtype)
    h = _P()
    _check(lib().dtp_layer_create(ctypes.byref(desc), ctypes.byref(h)))
    _LAYERS[h.value] = (d_model, n_neurons, n_q_heads, n_kv_groups, head_dim, dtype)
    return h.value


def dtp_layer_destroy(layer):
    _check(lib().dtp_layer_destroy(layer))
    _LAYERS.pop(layer, None)


def _layer_shape(layer):
    if layer not in _LAYERS:
        raise ValueError("not a layer handle returned by dtp_layer_create (or already destroyed)")
    return _LAYERS[layer]


def dtp_layer_set_weights(layer, w_o, gamma, w_gate, w_up, w_down, stream=None):
    d, I, H, G, dh, dt = _layer_shape(layer)
    ad = _act_dtypes(dt)
    _check(lib().dtp_layer_set_weights(layer, _dev(w_o, "w_o", ad, d * H * dh), _dev(gamma, "gamma", ad, d),
                                       _dev(w_gate, "w_gate", ad, I * d), _dev(w_up, "w_up", ad, I * d),
                                       _dev(w_down, "w_down", ad, d * I), _stream(stream)))


def _tokens(layer, x, attn, n_tokens, A):
    d, I, H, G, dh, dt = _layer_shape(layer)
    n = int(n_tokens)
    ad = _act_dtypes(dt)
    return (_dev(x, "x", ad, n * d), _dev(attn, "attn", ad, n * H * dh), n,
            _dev(A, "A", ("float32",), G * I))


def dtp_affinity_accumulate(layer, x, attn, n_tokens, A, stream=None):
    _check(lib().dtp_affinity_accumulate(layer, *_tokens(layer, x, attn, n_tokens, A), _stream(stream)))


def dtp_affinity_accumulate_add(layer, x, attn, n_tokens, A, stream=None):
    _check(lib().dtp_affinity_accumulate_add(layer, *_tokens(layer, x, attn, n_tokens, A),
                                             _stream(stream)))


def dtp_affinity_accumulate_down(layer, x, attn, x_next, rms_eps_next, n_tokens, A, s_down,
                                 stream=None):
    d, I, H, G, dh, dt = _layer_shape(layer)
    px, pa, n, pA = _tokens(layer, x, attn, n_tokens, A)
    _check(lib().dtp_affinity_accumulate_down(layer, px, pa, _dev(x_next, "x_next", _act_dtypes(dt), n * d),
                                              float(rms_eps_next), n, pA,
                                              _dev(s_down, "s_down", ("float32",), I), _stream(stream)))


def dtp_down_weights(d_model, n_neurons, n_q_heads, n_kv_groups, head_dim, dtype, w_q, w_k, w_v,
                     gamma_next, w_down, B, stream=None):
    ad = _act_dtypes(dtype)
    d, I, HD, GD = d_model, n_neurons, n_q_heads * head_dim, n_kv_groups * head_dim
    _check(lib().dtp_down_weights(d_model, n_neurons, n_q_heads, n_kv_groups, head_dim, int(dtype),
                                  _dev(w_q, "w_q", ad, HD * d), _dev(w_k, "w_k", ad, GD * d),
                                  _dev(w_v, "w_v", ad, GD * d), _dev(gamma_next, "gamma_next", ad, d),
                                  _dev(w_down, "w_down", ad, d * I),
                                  _dev(B, "B", ("float32",), n_kv_groups * I), _stream(stream)))


def dtp_down_weights_noalloc(d_model, n_neurons, n_q_heads, n_kv_groups, head_dim, dtype, w_q, w_k,
                             w_v, gamma_next, w_down, B, stream=None):
    """dtp_down_weights without any device allocation (a fixed per-device scratch array)."""
    ad = _act_dtypes(dtype)
    d, I, HD, GD = d_model, n_neurons, n_q_heads * head_dim, n_kv_groups * head_dim
    _check(lib().dtp_down_weights_noalloc(
        d_model, n_neurons, n_q_heads, n_kv_groups, head_dim, int(dtype),
        _dev(w_q, "w_q", ad, HD * d), _dev(w_k, "w_k", ad, GD * d), _dev(w_v, "w_v", ad, GD * d),
        _dev(gamma_next, "gamma_next", ad, d), _dev(w_down, "w_down", ad, d * I),
        _dev(B, "B", ("float32",), n_kv_groups * I), _stream(stream)))


def dtp_down_affinity(n_neurons, n_kv_groups, s_down, B, A_down, stream=None):
    n = n_neurons * n_kv_groups
    f = ("float32",)
    _check(lib().dtp_down_affinity(n_neurons, n_kv_groups, _dev(s_down, "s_down", f, n_neurons),
                                   _dev(B, "B", f, n), _dev(A_down, "A_down", f, n), _stream(stream)))


def dtp_layer_profile(layer, enable):
    _check(lib().dtp_layer_profile(layer, int(bool(enable))))


def dtp_layer_profile_read(layer):
    ms = ctypes.c_double()
    n = _I64()
    _check(lib().dtp_layer_profile_read(layer, ctypes.byref(ms), ctypes.byref(n)))
    return ms.value, n.value


# ----------------------------------------------------------------------------- layout
def dtp_partition_count(G, L):
    return int(lib().dtp_partition_count(G, L))


def dtp_partition_unrank(G, L, rank):
    h = np.zeros(max(G, 1), dtype=np.int32)
    _check(lib().dtp_partition_unrank(G, L, int(rank), _ptr(h)))
    return h[:G]


def dtp_encode_affinity(A):
    a = np.ascontiguousarray(A, dtype=np.float32)
    q = np.zeros(a.shape, dtype=np.int64)
    _check(lib().dtp_encode_affinity(_ptr(a), a.size, _ptr(q)))
    return q


def dtp_encode_affinity_device(A, Q, stream=None):
    """A (fp32) and Q (int64, same number of elements) are device tensors; Q is written."""
    n = A.numel()
    _check(lib().dtp_encode_affinity_device(_dev(A, "A", ("float32",), n), n,
                                            _dev(Q, "Q", ("int64",), n), _stream(stream)))
    return Q


def dtp_partition_scores(G, I, L, Q_up, nu, Q_down_prev=None, nu_prev=None, minimise=False,
                         scores=None, stream=None):
    """Q_up, nu (and Q_down_prev, nu_prev) and scores are device tensors; returns best rank."""
    best = _I64()
    P = max(dtp_partition_count(G, L), 0)
    _check(lib().dtp_partition_scores(G, I, L, _dev(Q_up, "Q_up", ("int64",), G * I),
                                      _dev(nu, "nu", ("int32",), I),
                                      _dev(Q_down_prev, "Q_down_prev", ("int64",), I * G, True),
                                      _dev(nu_prev, "nu_prev", ("int32",), I, True),
                                      int(bool(minimise)), _dev(scores, "scores", ("int64",), P),
                                      ctypes.byref(best), _stream(stream)))
    return best.value


def _assign(fn, G, I, L, Q_up, h, Q_down, h_next, minimise):
    qu = np.ascontiguousarray(Q_up, dtype=np.int64)
    hh = np.ascontiguousarray(h, dtype=np.int32)
    qd = None if Q_down is None else np.ascontiguousarray(Q_down, dtype=np.int64)
    hn = None if h_next is None else np.ascontiguousarray(h_next, dtype=np.int32)
    nu = np.zeros(max(I, 1), dtype=np.int32)
    val = _I64()
    _check(fn(G, I, L, _ptr(qu), _ptr(hh), _ptr(qd), _ptr(hn), int(bool(minimise)), _ptr(nu),
              ctypes.byref(val)))
    return nu[:I], val.value


def dtp_balanced_assign(G, I, L, Q_up, h, Q_down=None, h_next=None, minimise=False):
    """Host arrays in, (nu int32 [I], value) out."""
    return _assign(lib().dtp_balanced_assign, G, I, L, Q_up, h, Q_down, h_next, minimise)


def dtp_balanced_assign_dual_ascent(G, I, L, Q_up, h, Q_down=None, h_next=None, minimise=False):
    """The paper's approximate neuron step: host arrays in, (nu int32 [I], value) out."""
    return _assign(lib().dtp_balanced_assign_dual_ascent, G, I, L, Q_up, h, Q_down, h_next,
                   minimise)


def dtp_coordinate_ascent(N, G, I, L, A_up, A_down=None, max_sweeps=64, freeze_heads=False,
                          freeze_neurons=False, minimise=False, layer_mask=None, stream=None,
                          dual_ascent_neurons=False):
    """A_up [N,G,I] (and A_down [N-1,I,G]) are device tensors; returns a dict of host results."""
    mask = None if layer_mask is None else _host(layer_mask, "layer_mask", np.uint8, N)
    opt = dtp_ca_options(max_sweeps, int(freeze_heads), int(freeze_neurons), int(minimise),
                         _ptr(mask), int(dual_ascent_neurons))
    h = np.zeros((N, G), dtype=np.int32)
    nu = np.zeros((N, I), dtype=np.int32)
    jf = _I64()
    j = ctypes.c_double()
    sw = _I32()
    f = ("float32",)
    _check(lib().dtp_coordinate_ascent(N, G, I, L, _dev(A_up, "A_up", f, N * G * I),
                                       _dev(A_down, "A_down", f, (N - 1) * I * G, True), ctypes.byref(opt),
                                       _ptr(h), _ptr(nu), ctypes.byref(j), ctypes.byref(jf),
                                       ctypes.byref(sw), _stream(stream)))
    return {"h": h, "nu": nu, "J_fixed": jf.value, "J": j.value, "sweeps": sw.value}


def dtp_random_layout(N, G, I, L, seed):
    """(h [N, G], nu [N, I]) int32 host arrays of the seeded balanced layouts."""
    h = np.zeros((N, G), dtype=np.int32)
    nu = np.zeros((N, I), dtype=np.int32)
    _check(lib().dtp_random_layout(N, G, I, L, ctypes.c_uint64(seed & (2 ** 64 - 1)), _ptr(h), _ptr(nu)))
    return h, nu


def dtp_layout_objective(N, G, I, L, Q_up, Q_down, h, nu):
    """J_int of a layout from host codes (int64 arrays), as a Python int."""
    Q_up = np.ascontiguousarray(Q_up, dtype=np.int64)
    Q_down = None if Q_down is None else np.ascontiguousarray(Q_down, dtype=np.int64)
    h = np.ascontiguousarray(h, dtype=np.int32)
    nu = np.ascontiguousarray(nu, dtype=np.int32)
    J = _I64()
    _check(lib().dtp_layout_objective(N, G, I, L, _ptr(Q_up), _ptr(Q_down), _ptr(h), _ptr(nu),
                                      ctypes.byref(J)))
    return int(J.value)


def dtp_layer_optimum(G, I, L, Q_up):
    """(h [G], nu [I], J_int) of one layer's exact optimum from host codes."""
    Q_up = np.ascontiguousarray(Q_up, dtype=np.int64)
    h = np.zeros(G, dtype=np.int32)
    nu = np.zeros(I, dtype=np.int32)
    J = _I64()
    _check(lib().dtp_layer_optimum(G, I, L, _ptr(Q_up), _ptr(h), _ptr(nu), ctypes.byref(J)))
    return h, nu, int(J.value)


def dtp_layout_orders(G, I, L, h, nu):
    """(group_order [G], neuron_order [I]) int32: new position -> original index."""
    h = np.ascontiguousarray(h, dtype=np.int32)
    nu = np.ascontiguousarray(nu, dtype=np.int32)
    go = np.zeros(G, dtype=np.int32)
    no = np.zeros(I, dtype=np.int32)
    _check(lib().dtp_layout_orders(G, I, L, _ptr(h), _ptr(nu), _ptr(go), _ptr(no)))
    return go, no


WEIGHT_ORDER = ("w_q", "w_k", "w_v", "w_o", "w_gate", "w_up", "w_down")


def dtp_apply_layout(d_model, n_neurons, n_q_heads, n_kv_groups, head_dim, dtype, L, h, nu, src,
                     dst, stream=None):
    """Permute a layer's weights: ``src`` and ``dst`` map WEIGHT_ORDER names to tensors."""
    desc = dtp_layer_desc(d_model, n_neurons, n_q_heads, n_kv_groups, head_dim, 0.0, int(dtype))
    h = _host(h, "h", np.int32, n_kv_groups)
    nu = _host(nu, "nu", np.int32, n_neurons)
    d, I, HD, GD = d_model, n_neurons, n_q_heads * head_dim, n_kv_groups * head_dim
    sizes = dict(w_q=HD * d, w_k=GD * d, w_v=GD * d, w_o=d * HD, w_gate=I * d, w_up=I * d, w_down=d * I)
    ad = _act_dtypes(dtype)
    srcp = (ctypes.c_void_p * 7)(*[_dev(src[k], "src " + k, ad, sizes[k]) for k in WEIGHT_ORDER])
    dstp = (ctypes.c_void_p * 7)(*[_dev(dst[k], "dst " + k, ad, sizes[k]) for k in WEIGHT_ORDER])
    _check(lib().dtp_apply_layout(ctypes.byref(desc), L, _ptr(h), _ptr(nu),
                                  ctypes.cast(srcp, ctypes.c_void_p), ctypes.cast(dstp, ctypes.c_void_p),
                                  _stream(stream)))
