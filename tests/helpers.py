"""Shared plumbing of the GPU tests: upload seeded inputs, run the library, compare."""
from __future__ import annotations

import numpy as np

from paper_2609_13846_amd import dtp, synth

REL_TOL = 1e-2        # relative error allowed on entries above THRESH * max(A)
THRESH = 1e-3


def torch_dev(arr: np.ndarray, device="cuda"):
    """Storage array (uint16 bf16 bits or float32) -> device tensor with the same bytes."""
    import torch
    if arr.dtype == np.uint16:
        return torch.from_numpy(arr.view(np.int16).copy()).view(torch.bfloat16).to(device)
    return torch.from_numpy(np.ascontiguousarray(arr)).to(device)


def layer_for(wl: synth.Workload):
    dt = dtp.DTP_BF16 if wl.dtype == "bf16" else dtp.DTP_F32
    return dtp.dtp_layer_create(wl.d_model, wl.n_neurons, wl.n_q_heads, wl.n_kv_groups,
                                wl.head_dim, wl.rms_eps, dt)


def gpu_affinity(wl: synth.Workload, w: synth.LayerWeights, x: np.ndarray, a: np.ndarray,
                 chunks=None, A0=None, score="fo") -> np.ndarray:
    """A [G, I] float32 from the library, accumulated over token chunks (sizes); score
    "fo" (first order) or "add"."""
    import torch
    T = x.shape[0]
    layer = layer_for(wl)
    try:
        dw = [torch_dev(v) for v in (w.w_o, w.gamma, w.w_gate, w.w_up, w.w_down)]
        dtp.dtp_layer_set_weights(layer, *dw)
        dx, da = torch_dev(x), torch_dev(a)
        A = torch.zeros(wl.n_kv_groups, wl.n_neurons, dtype=torch.float32, device="cuda")
        if A0 is not None:
            A.copy_(torch.from_numpy(A0))
        bounds = [0]
        for c in (chunks or [T]):
            bounds.append(bounds[-1] + c)
        assert bounds[-1] == T
        for t0, t1 in zip(bounds, bounds[1:]):
            fn = dtp.dtp_affinity_accumulate if score == "fo" else dtp.dtp_affinity_accumulate_add
            fn(layer, dx[t0:t1], da[t0:t1], t1 - t0, A)
        torch.cuda.synchronize()
        return A.cpu().numpy()
    finally:
        dtp.dtp_layer_destroy(layer)


def oracle_inputs(w: synth.LayerWeights, x, a):
    f = synth.to_f64
    return dict(x=f(x), attn=f(a), w_o=f(w.w_o), gamma=f(w.gamma), w_gate=f(w.w_gate),
                w_up=f(w.w_up), w_down=f(w.w_down))


def assert_affinity_close(A_gpu: np.ndarray, A_ref: np.ndarray, rel=REL_TOL, thresh=THRESH):
    """Relative error <= rel on entries above thresh * max; the rest within rel * thresh * max."""
    A_gpu = np.asarray(A_gpu, dtype=np.float64)
    assert A_gpu.shape == A_ref.shape
    assert np.all(np.isfinite(A_gpu))
    top = A_ref.max()
    big = A_ref > thresh * top
    err = np.abs(A_gpu - A_ref)
    rel_err = err[big] / A_ref[big]
    assert rel_err.max() <= rel, f"max rel err {rel_err.max():.3e} (mean {rel_err.mean():.3e})"
    assert err[~big].max(initial=0.0) <= rel * thresh * top
    return float(rel_err.max())


def device_chain(wl: synth.Workload, n_layers=None, tokens=None):
    """Raw up and down affinity of a whole layer chain at the workload's full token count,
    on data generated on the device chunk by chunk (as the full-model benchmark streams
    it): A_up [N, G, I] and A_down [N-1, I, G] device tensors (A_down None when N = 1).
    Layer i's down edge reads the residual entering layer i+1 (its x_pre) and layer
    i+1's attention weights."""
    import torch
    dev = torch.device("cuda", 0)
    N = n_layers or wl.n_layers
    T = tokens or wl.tokens
    G, I = wl.n_kv_groups, wl.n_neurons
    dt = dtp.DTP_BF16 if wl.dtype == "bf16" else dtp.DTP_F32
    A = torch.zeros(N, G, I, dtype=torch.float32, device=dev)
    A_down = torch.zeros(max(N - 1, 1), I, G, dtype=torch.float32, device=dev)
    s_down = torch.zeros(I, dtype=torch.float32, device=dev)
    B = torch.zeros(G, I, dtype=torch.float32, device=dev)
    weights = [synth.device_weights(wl, i, dev) for i in range(N)]
    for i in range(N):
        w = weights[i]
        layer = layer_for(wl)
        try:
            dtp.dtp_layer_set_weights(layer, w["w_o"], w["gamma"], w["w_gate"], w["w_up"], w["w_down"])
            s_down.zero_()
            for c in range(T // wl.chunk):
                x, a = synth.device_tokens(wl, i, w, wl.chunk, c, dev)
                if i + 1 < N:
                    _, _, x_next = synth.device_tokens(wl, i + 1, weights[i + 1], wl.chunk, c, dev,
                                                       with_pre=True)
                    dtp.dtp_affinity_accumulate_down(layer, x, a, x_next, wl.rms_eps, wl.chunk, A[i], s_down)
                else:
                    dtp.dtp_affinity_accumulate(layer, x, a, wl.chunk, A[i])
            if i + 1 < N:
                an = synth.device_attn_weights(wl, i + 1, dev)
                dtp.dtp_down_weights(wl.d_model, I, wl.n_q_heads, G, wl.head_dim, dt, an["w_q"], an["w_k"],
                                     an["w_v"], an["gamma"], w["w_down"], B)
                dtp.dtp_down_affinity(I, G, s_down, B, A_down[i])
            torch.cuda.synchronize()
        finally:
            dtp.dtp_layer_destroy(layer)
    return A, (A_down if N > 1 else None)
