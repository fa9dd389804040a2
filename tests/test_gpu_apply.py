"""GPU: applying a layout to a layer's weights (Section 3, "The layout as a free variable").

The library's permuted weights must equal the oracle's bit for bit (pure data movement),
and the permuted layer must compute the same function: the paper checks a maximum logit
difference of 1e-4 in fp32, which is repeated here with a fp32 decoder layer on the GPU
(GQA attention with per-head norms and rotary embedding, SwiGLU FFN) and a random
unembedding.
"""
import numpy as np
import pytest

from oracle import apply as ap
from oracle import layout as lay
from paper_2609_13846_amd import dtp, synth
from tests.helpers import torch_dev

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


def stored_weights(wl):
    w = synth.host_weights(wl, 0)
    an = synth.host_attn_weights(wl, 0)
    return {"w_q": an.w_q, "w_k": an.w_k, "w_v": an.w_v, "w_o": w.w_o, "w_gate": w.w_gate,
            "w_up": w.w_up, "w_down": w.w_down}, w, an


def gpu_apply(wl, L, h, nu, stored):
    src = {k: torch_dev(v) for k, v in stored.items()}
    dst = {k: torch.empty_like(v) for k, v in src.items()}
    dt = dtp.DTP_BF16 if wl.dtype == "bf16" else dtp.DTP_F32
    dtp.dtp_apply_layout(wl.d_model, wl.n_neurons, wl.n_q_heads, wl.n_kv_groups, wl.head_dim, dt,
                         L, h, nu, src, dst)
    torch.cuda.synchronize()
    return src, dst


def _bits(t):
    return t.view(torch.int16).cpu().numpy() if t.dtype == torch.bfloat16 else t.cpu().numpy()


@pytest.mark.parametrize("name,L,seed", [("qwen3-0.6b-layer", 4, 1000), ("qwen3-0.6b-layer", 2, 1003),
                                         ("danube3-500m", 4, 1001), ("tiny", 2, 1002)])
def test_apply_layout_bit_exact(name, L, seed):
    wl = synth.WORKLOADS[name]
    stored, _, _ = stored_weights(wl)
    hs, nus = lay.random_layout(1, wl.n_kv_groups, wl.n_neurons, L, seed)
    _, dst = gpu_apply(wl, L, hs[0], nus[0], stored)
    ref = ap.apply_layout(stored, hs[0], nus[0], wl.n_q_heads, wl.n_kv_groups, wl.head_dim, L)
    for k in dtp.WEIGHT_ORDER:
        got = _bits(dst[k])
        want = ref[k].view(np.int16) if ref[k].dtype == np.uint16 else ref[k]
        np.testing.assert_array_equal(got, want, err_msg=k)


def _rms(x, g, eps):
    return g * x * torch.rsqrt(torch.mean(x * x, dim=-1, keepdim=True) + eps)


def _rope(x):
    T, _, dh = x.shape
    half = dh // 2
    inv = 10000.0 ** (-torch.arange(half, device=x.device, dtype=x.dtype) / half)
    ang = torch.arange(T, device=x.device, dtype=x.dtype)[:, None] * inv[None, :]
    c, s = torch.cos(ang)[:, None, :], torch.sin(ang)[:, None, :]
    a, b = x[..., :half], x[..., half:]
    return torch.cat([a * c - b * s, a * s + b * c], dim=-1)


def layer_fp32(x, w, H, G, dh, eps):
    T = x.shape[0]
    n = _rms(x, w["gamma_attn"], eps)
    q = _rope(_rms((n @ w["w_q"].T).reshape(T, H, dh), w["q_norm"], eps))
    k = _rope(_rms((n @ w["w_k"].T).reshape(T, G, dh), w["k_norm"], eps))
    v = (n @ w["w_v"].T).reshape(T, G, dh)
    k = k.repeat_interleave(H // G, dim=1)
    v = v.repeat_interleave(H // G, dim=1)
    qh = q.permute(1, 0, 2).contiguous()              # [H, T, dh]
    kt = k.permute(1, 2, 0).contiguous()              # [H, dh, T]
    vh = v.permute(1, 0, 2).contiguous()              # [H, T, dh]
    s = torch.bmm(qh, kt) / dh ** 0.5
    s = s + torch.triu(torch.full((T, T), float("-inf"), device=x.device), 1)
    o = torch.bmm(torch.softmax(s, dim=-1), vh).permute(1, 0, 2).reshape(T, H * dh)
    x1 = x + o @ w["w_o"].T
    n2 = _rms(x1, w["gamma"], eps)
    return x1 + (torch.nn.functional.silu(n2 @ w["w_gate"].T) * (n2 @ w["w_up"].T)) @ w["w_down"].T


@pytest.mark.parametrize("L,seed", [(2, 1004), (4, 1005)])
def test_permuted_layer_same_logits_fp32(L, seed):
    wl = synth.shaped(synth.WORKLOADS["tiny"], d_model=256, n_neurons=512, n_q_heads=8,
                      n_kv_groups=4, head_dim=32)
    stored, w, an = stored_weights(wl)
    hs, nus = lay.random_layout(1, wl.n_kv_groups, wl.n_neurons, L, seed)
    src, dst = gpu_apply(wl, L, hs[0], nus[0], stored)
    rng = np.random.default_rng(seed)
    extra = {"gamma_attn": torch_dev(an.gamma), "gamma": torch_dev(w.gamma),
             "q_norm": torch.tensor(1 + 0.1 * rng.standard_normal(wl.head_dim), dtype=torch.float32, device="cuda"),
             "k_norm": torch.tensor(1 + 0.1 * rng.standard_normal(wl.head_dim), dtype=torch.float32, device="cuda")}
    x = torch.tensor(rng.standard_normal((64, wl.d_model)), dtype=torch.float32, device="cuda")
    unembed = torch.tensor(rng.standard_normal((512, wl.d_model)) * 0.05, dtype=torch.float32, device="cuda")
    args = (wl.n_q_heads, wl.n_kv_groups, wl.head_dim, wl.rms_eps)
    y0 = layer_fp32(x, {**src, **extra}, *args) @ unembed.T
    y1 = layer_fp32(x, {**dst, **extra}, *args) @ unembed.T
    diff = (y0 - y1).abs().max().item()
    assert diff <= 1e-4, diff
    assert not torch.equal(src["w_q"], dst["w_q"])
