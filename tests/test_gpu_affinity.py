"""GPU parity of the affinity accumulation against the fp64 oracle (through the C ABI).

Bar: relative error <= 1e-2 on every entry above 1e-3 * max(A) (bf16 inputs, fp32
accumulation); smaller entries within 1e-2 * 1e-3 * max(A) absolute.  Sizes are chosen so
the oracle finishes in seconds while spanning several token and neuron tiles and a
ragged token tail; the full Qwen3-0.6B-shaped layer (65,536 tokens, the benchmarked
launch) is checked on sampled neurons the oracle computes one by one.
"""
import sys

import numpy as np
import pytest

from oracle import affinity as orc
from paper_2609_13846_amd import dtp, synth
from tests import helpers as hp

pytestmark = pytest.mark.gpu


def announce(msg):
    print(f"[gpu] {msg}", file=sys.stderr, flush=True)


def case(name, T, layer=0, **shape):
    wl = synth.shaped(synth.WORKLOADS[name], **shape) if shape else synth.WORKLOADS[name]
    w = synth.host_weights(wl, layer)
    x, a = synth.host_tokens(wl, layer, w, T)
    return wl, w, x, a


def oracle(wl, w, x, a, neurons=None):
    return orc.affinity_folded(**hp.oracle_inputs(w, x, a), n_kv_groups=wl.n_kv_groups,
                               eps=wl.rms_eps, neurons=neurons)


@pytest.mark.parametrize("name,T,shape", [
    ("tiny", 512, {}),
    ("tiny", 37, {}),
    ("qwen3-0.6b-layer", 300, {}),
    ("danube3-500m", 257, {}),
    ("qwen3-0.6b-layer", 200, dict(n_neurons=1000)),               # ragged neuron tile
    ("qwen3-0.6b-layer", 150, dict(n_neurons=1003)),               # I % 8 != 0: scalar norm pass
    ("qwen3-0.6b-layer", 130, dict(n_q_heads=2, n_kv_groups=1)),    # one group
    ("qwen3-0.6b-layer", 129, dict(n_q_heads=8, n_kv_groups=8, head_dim=48)),  # H = G, dh % 32 = 16
    ("qwen3-0.6b-layer", 100, dict(n_q_heads=32, n_kv_groups=32, head_dim=64)),  # G at its limit
    # the largest G with six copy buffers in the LDS, and the smallest that falls back to three
    ("qwen3-0.6b-layer", 90, dict(n_q_heads=26, n_kv_groups=26, head_dim=64)),
    ("qwen3-0.6b-layer", 90, dict(n_q_heads=27, n_kv_groups=27, head_dim=64)),
    ("danube3-500m", 64, dict(d_model=272, n_neurons=192)),         # d % 32 = 16
    # two 64-deep stages and two 32-deep stages: the weight ring wraps within a tile
    ("qwen3-0.6b-layer", 70, dict(d_model=64, n_q_heads=1, n_kv_groups=1, head_dim=64, n_neurons=128)),
    ("danube3-500m", 40, dict(d_model=32, n_q_heads=1, n_kv_groups=1, head_dim=32, n_neurons=64)),
    # an odd number of stages (three), so the last one ends an unfinished pair of stages
    ("qwen3-0.6b-layer", 600, dict(d_model=128, n_q_heads=1, n_kv_groups=1, head_dim=64, n_neurons=128)),
    ("danube3-500m", 300, dict(d_model=64, n_q_heads=1, n_kv_groups=1, head_dim=32, n_neurons=64)),
    # three-stage heads (nine copy buffers): six stages, fewer than the ring, and nine
    ("danube3-500m", 300, dict(d_model=96, n_q_heads=1, n_kv_groups=1, head_dim=96, n_neurons=64)),
    ("danube3-500m", 600, dict(d_model=96, n_q_heads=2, n_kv_groups=1, head_dim=96, n_neurons=128)),
])
def test_affinity_matches_oracle(name, T, shape):
    wl, w, x, a = case(name, T, **shape)
    announce(f"affinity {name} T={T} {shape}")
    A = hp.gpu_affinity(wl, w, x, a)
    hp.assert_affinity_close(A, oracle(wl, w, x, a))


def test_unaligned_down_weights_give_the_same_affinity():
    """W_down at an address 2 bytes past a 16-byte boundary takes the norms' scalar pass
    instead of its 16-byte loads; each column is summed in the same order either way, so
    the affinity is bit-identical."""
    import torch
    wl, w, x, a = case("qwen3-0.6b-layer", 300)
    announce("affinity with W_down 2 bytes off a 16-byte boundary")
    dw = [hp.torch_dev(v) for v in (w.w_o, w.gamma, w.w_gate, w.w_up, w.w_down)]
    wd = dw[4].reshape(-1)
    shifted = torch.empty(wd.numel() + 8, dtype=wd.dtype, device="cuda")
    shifted[1:1 + wd.numel()].copy_(wd)
    wd_off = shifted[1:1 + wd.numel()]
    assert wd_off.data_ptr() % 16 == 2
    dx, da = hp.torch_dev(x), hp.torch_dev(a)
    out = []
    for w_down in (dw[4], wd_off):
        layer = hp.layer_for(wl)
        try:
            dtp.dtp_layer_set_weights(layer, dw[0], dw[1], dw[2], dw[3], w_down)
            A = torch.zeros(wl.n_kv_groups, wl.n_neurons, dtype=torch.float32, device="cuda")
            dtp.dtp_affinity_accumulate(layer, dx, da, x.shape[0], A)
            torch.cuda.synchronize()
            out.append(A.cpu().numpy())
        finally:
            dtp.dtp_layer_destroy(layer)
    np.testing.assert_array_equal(out[0], out[1])
    hp.assert_affinity_close(out[1], oracle(wl, w, x, a))


def test_affinity_8b_class_sampled_neurons():
    wl, w, x, a = case("8b-class-4layer", 200, layer=3)
    announce("affinity 8b-class T=200 sampled neurons")
    A = hp.gpu_affinity(wl, w, x, a)
    cols = np.r_[0:64, 7000:7064, wl.n_neurons - 64:wl.n_neurons]
    hp.assert_affinity_close(A[:, cols], oracle(wl, w, x, a, neurons=cols))


@pytest.mark.parametrize("G", [26, 32])
def test_affinity_many_tiles_per_block_sampled_neurons(G):
    """8,192 tokens at G = 26 (six copy buffers) and G = 32 (three): 32 tiles of 256 tokens
    over 16 token splits, so each block runs two tiles back to back."""
    wl, w, x, a = case("qwen3-0.6b-layer", 8192, n_q_heads=G, n_kv_groups=G, head_dim=64)
    announce(f"affinity G={G} T=8192 sampled neurons")
    A = hp.gpu_affinity(wl, w, x, a)
    cols = np.r_[0:32, 1500:1532, wl.n_neurons - 32:wl.n_neurons]
    hp.assert_affinity_close(A[:, cols], oracle(wl, w, x, a, neurons=cols))


def test_affinity_danube_many_tiles_per_block_sampled_neurons():
    """8,192 Danube-shaped tokens (nine copy buffers): 32 tiles over 12 token splits."""
    wl, w, x, a = case("danube3-500m", 8192)
    announce("affinity danube3-500m T=8192 sampled neurons")
    A = hp.gpu_affinity(wl, w, x, a)
    cols = np.r_[0:32, 2000:2032, wl.n_neurons - 32:wl.n_neurons]
    hp.assert_affinity_close(A[:, cols], oracle(wl, w, x, a, neurons=cols))


def test_empty_and_single_token():
    """T = 0 leaves A alone.  T = 1 is checked entry by entry against the rounding model of
    the bf16 operands (tests/error_model.py): with one token nothing averages the rounding
    of W' and F_h, and an entry's error is about kappa * 2^-8 / sqrt(3), kappa its
    condition number from the inputs.  Every entry must lie within its own bound; entries
    whose bound fits inside 1e-2 are held to 1e-2; the others are counted as exempt."""
    from tests import error_model as em
    wl, w, x, a = case("qwen3-0.6b-layer", 1)
    announce("affinity T=0 and T=1")
    A0 = np.full((wl.n_kv_groups, wl.n_neurons), 0.25, np.float32)
    A = hp.gpu_affinity(wl, w, x[:0], a[:0], chunks=[0], A0=A0)
    np.testing.assert_array_equal(A, A0)
    A1 = hp.gpu_affinity(wl, w, x, a)
    f = synth.to_f64
    ref, sig, sec = em.up_affinity_error(f(x), f(a), f(w.w_o), f(w.gamma), f(w.w_gate), f(w.w_up),
                                         f(w.w_down), wl.n_kv_groups, wl.rms_eps)
    np.testing.assert_allclose(ref, oracle(wl, w, x, a), rtol=1e-10)
    rep = em.check_entrywise(A1, ref, sig, sec, label="T=1")
    announce(f"T=1: {rep}")


def test_deterministic_and_chunk_additive():
    wl, w, x, a = case("qwen3-0.6b-layer", 1000)
    announce("affinity determinism and chunks T=1000")
    A1 = hp.gpu_affinity(wl, w, x, a)
    A2 = hp.gpu_affinity(wl, w, x, a)
    np.testing.assert_array_equal(A1, A2)
    A3 = hp.gpu_affinity(wl, w, x, a, chunks=[384, 333, 283])
    np.testing.assert_allclose(A3, A1, rtol=1e-5)


def test_token_order_and_row_slot_do_not_matter():
    """A is a sum over tokens: permuting them, or shifting every token to another row of
    its tile by prepending all-zero tokens (u = 0 gives both coefficients zero, so such a
    token adds exactly nothing), changes only the fp32 summation order.  Catches per-row
    differences in the arithmetic, e.g. a coefficient rounded once in some rows and twice
    in others."""
    wl, w, x, a = case("qwen3-0.6b-layer", 1000)
    announce("affinity: token permutation and row-slot shifts, T=1000")
    A = hp.gpu_affinity(wl, w, x, a)
    perm = np.random.default_rng(7).permutation(x.shape[0])
    np.testing.assert_allclose(hp.gpu_affinity(wl, w, x[perm], a[perm]), A, rtol=1e-5)
    for k in (1, 13, 31, 100):
        xs = np.concatenate([np.zeros_like(x[:k]), x])
        as_ = np.concatenate([np.zeros_like(a[:k]), a])
        np.testing.assert_allclose(hp.gpu_affinity(wl, w, xs, as_), A, rtol=1e-5)


@pytest.mark.parametrize("c", [2.0, 0.5])
def test_power_of_two_head_scale_is_exact(c):
    """Scaling the query heads of one KV group by 2^k scales its row by 4^k bit for bit
    (bf16 inputs stay exact and fp32 sums scale exactly); other rows are untouched."""
    wl, w, x, a = case("qwen3-0.6b-layer", 700)
    announce(f"affinity head scale {c}")
    A = hp.gpu_affinity(wl, w, x, a)
    g = 3
    hpg = wl.n_q_heads // wl.n_kv_groups
    a2 = synth.to_f64(a).copy()
    a2[:, g * hpg:(g + 1) * hpg] *= c
    A2 = hp.gpu_affinity(wl, w, x, synth.store(a2, "bf16"))
    np.testing.assert_array_equal(A2[g], A[g] * np.float32(c * c))
    np.testing.assert_array_equal(np.delete(A2, g, 0), np.delete(A, g, 0))


def test_neuron_permutation_equivariance():
    wl, w, x, a = case("qwen3-0.6b-layer", 400)
    announce("affinity neuron permutation")
    perm = np.random.default_rng(5).permutation(wl.n_neurons)
    w2 = synth.LayerWeights(w.w_o, w.gamma, w.w_gate[perm].copy(), w.w_up[perm].copy(),
                            w.w_down[:, perm].copy(), w.outliers)
    A = hp.gpu_affinity(wl, w, x, a)
    A2 = hp.gpu_affinity(wl, w2, x, a)
    # each (group, neuron) entry is computed independently of its tile position
    np.testing.assert_array_equal(A2, A[:, perm])


# ----------------------------------------------------------------------------- ADD score
def add_oracle(wl, w, x, a, neurons=None):
    kw = hp.oracle_inputs(w, x, a)
    kw.pop("w_down")
    return orc.affinity_add_folded(**kw, n_kv_groups=wl.n_kv_groups, eps=wl.rms_eps, neurons=neurons)


@pytest.mark.parametrize("name,T,shape", [
    ("tiny", 512, {}),
    ("qwen3-0.6b-layer", 300, {}),
    ("danube3-500m", 257, {}),
    ("danube3-500m", 64, dict(d_model=272, n_neurons=192)),         # 16-deep stages
    ("qwen3-0.6b-layer", 100, dict(n_q_heads=32, n_kv_groups=32, head_dim=64)),
])
def test_add_score_matches_oracle(name, T, shape):
    wl, w, x, a = case(name, T, **shape)
    announce(f"add score {name} T={T} {shape}")
    A = hp.gpu_affinity(wl, w, x, a, score="add")
    hp.assert_affinity_close(A, add_oracle(wl, w, x, a))


def test_add_score_full_qwen_layer_sampled_neurons():
    wl, w, x, a = case("qwen3-0.6b-layer", 65536)
    announce("add score qwen 65536 sampled neurons")
    A = hp.gpu_affinity(wl, w, x, a, score="add")
    cols = np.r_[0:32, 1500:1532, wl.n_neurons - 32:wl.n_neurons]
    hp.assert_affinity_close(A[:, cols], add_oracle(wl, w, x, a, neurons=cols))


def test_add_score_power_of_two_head_scale_is_exact():
    wl, w, x, a = case("qwen3-0.6b-layer", 300)
    H, G = wl.n_q_heads, wl.n_kv_groups
    g = 3
    heads = [h for h in range(H) if h // (H // G) == g]
    a2 = synth.to_f64(a).copy()
    a2[:, heads] *= 2.0
    a2 = synth.store(a2, "bf16")
    A1 = hp.gpu_affinity(wl, w, x, a, score="add")
    A2 = hp.gpu_affinity(wl, w, x, a2, score="add")
    np.testing.assert_array_equal(A2[g], 4.0 * A1[g])
    np.testing.assert_array_equal(np.delete(A2, g, axis=0), np.delete(A1, g, axis=0))


@pytest.mark.parametrize("name", ["danube3-500m", "8b-class-4layer"])
def test_affinity_full_workload_sampled_neurons(name):
    """The whole calibration set of one layer (131,072 tokens, streamed in the workload's
    16,384-token chunks as the full-model run does), generated on the device; the oracle
    recomputes 32 sampled neurons chunk by chunk from the same bytes (token sums add)."""
    import torch
    wl = synth.WORKLOADS[name]
    dev = torch.device("cuda", 0)
    announce(f"affinity {name} T={wl.tokens} in chunks of {wl.chunk} (full, device data)")
    w = synth.device_weights(wl, 0, dev)
    layer = hp.layer_for(wl)
    A = torch.zeros(wl.n_kv_groups, wl.n_neurons, dtype=torch.float32, device=dev)
    rng = np.random.default_rng(1)
    cols = np.sort(np.concatenate([rng.choice(wl.n_neurons, 28, replace=False),
                                   [0, 63, 64, wl.n_neurons - 1]]))
    f = lambda t: t.float().cpu().numpy().astype(np.float64)
    wh = {k: f(w[k]) for k in ("w_o", "gamma", "w_gate", "w_up", "w_down")}
    ref = np.zeros((wl.n_kv_groups, len(cols)))
    try:
        dtp.dtp_layer_set_weights(layer, w["w_o"], w["gamma"], w["w_gate"], w["w_up"], w["w_down"])
        for c in range(wl.tokens // wl.chunk):
            x, a = synth.device_tokens(wl, 0, w, wl.chunk, c, dev)
            dtp.dtp_affinity_accumulate(layer, x, a, wl.chunk, A)
            ref += orc.affinity_folded(f(x), f(a).reshape(wl.chunk, wl.n_q_heads, wl.head_dim),
                                       wh["w_o"], wh["gamma"], wh["w_gate"], wh["w_up"],
                                       wh["w_down"], wl.n_kv_groups, wl.rms_eps, neurons=cols)
        torch.cuda.synchronize()
        hp.assert_affinity_close(A.cpu().numpy()[:, cols], ref)
    finally:
        dtp.dtp_layer_destroy(layer)


def test_two_layers_accumulated_from_two_threads_match_serial():
    """Two layers (their own workspaces), each fed from its own host thread and stream at
    the same time, give exactly what each gives alone."""
    import threading

    import torch
    announce("two layers accumulated concurrently from two threads")
    wl = synth.WORKLOADS["qwen3-0.6b-layer"]
    data = []
    for layer_idx in range(2):
        w = synth.host_weights(wl, layer_idx)
        x, a = synth.host_tokens(wl, layer_idx, w, 3000)
        data.append((w, x, a))
    serial = [hp.gpu_affinity(wl, w, x, a) for (w, x, a) in data]
    layers, inputs, outs = [], [], []
    try:
        for (w, x, a) in data:
            layer = hp.layer_for(wl)
            layers.append(layer)
            dtp.dtp_layer_set_weights(layer, *(hp.torch_dev(v) for v in (w.w_o, w.gamma, w.w_gate, w.w_up, w.w_down)))
            inputs.append((hp.torch_dev(x), hp.torch_dev(a)))
            outs.append(torch.zeros(wl.n_kv_groups, wl.n_neurons, dtype=torch.float32, device="cuda"))
        torch.cuda.synchronize()

        def worker(i):
            stream = torch.cuda.Stream()
            for _ in range(3):
                dtp.dtp_affinity_accumulate(layers[i], inputs[i][0], inputs[i][1], 3000, outs[i], stream=stream)
            stream.synchronize()

        threads = [threading.Thread(target=worker, args=(i,)) for i in range(2)]
        for th in threads:
            th.start()
        for th in threads:
            th.join()
        for i in range(2):  # three accumulations of the same tokens: 3x the single pass
            np.testing.assert_allclose(outs[i].cpu().numpy(), 3 * serial[i], rtol=1e-6)
    finally:
        for layer in layers:
            dtp.dtp_layer_destroy(layer)
