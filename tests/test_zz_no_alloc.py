"""The allocation-free entry point dtp_down_weights_noalloc against dtp_down_weights,
through the C ABI: the same B bit for bit, on calls in a row whose inputs shrink (the
second and third calls reuse the per-device scratch array the first one filled)."""
import sys

import pytest
import torch

from paper_2609_13846_amd import dtp, synth

pytestmark = pytest.mark.gpu


def announce(msg):
    print(f"[gpu] {msg}", file=sys.stderr, flush=True)


def _both(wl):
    dev = torch.device("cuda", 0)
    w = synth.device_weights(wl, 0, dev)
    an = synth.device_attn_weights(wl, 1, dev)
    G, I = wl.n_kv_groups, wl.n_neurons
    args = (wl.d_model, I, wl.n_q_heads, G, wl.head_dim, dtp.DTP_BF16, an["w_q"], an["w_k"], an["w_v"],
            an["gamma"], w["w_down"])
    B_ref = torch.zeros(G, I, dtype=torch.float32, device=dev)
    B_na = torch.full((G, I), float("nan"), dtype=torch.float32, device=dev)
    dtp.dtp_down_weights(*args, B_ref)
    dtp.dtp_down_weights_noalloc(*args, B_na)
    torch.cuda.synchronize()
    return B_ref, B_na


def test_noalloc_down_weights_equals_the_allocating_entry_point():
    # the largest shape first (688,128 of the 2^20 partial sums), then smaller inputs
    for name in ["8b-class-4layer", "danube3-500m", "qwen3-0.6b-model"]:
        wl = synth.WORKLOADS[name]
        announce(f"noalloc down weights {name}")
        B_ref, B_na = _both(wl)
        assert torch.isfinite(B_ref).all() and (B_ref > 0).all()
        assert torch.equal(B_na, B_ref), name


def test_noalloc_refuses_more_than_its_scratch():
    dev = torch.device("cuda", 0)
    d, I, H, G, dh = 64, 65536, 32, 8, 128     # 8 * 65536 * 6 partial sums > 2^20
    t = lambda *sh: torch.zeros(*sh, dtype=torch.bfloat16, device=dev)
    B = torch.zeros(G, I, dtype=torch.float32, device=dev)
    with pytest.raises(dtp.DtpError) as e:
        dtp.dtp_down_weights_noalloc(d, I, H, G, dh, dtp.DTP_BF16, t(H * dh, d), t(G * dh, d), t(G * dh, d),
                                     t(d), t(d, I), B)
    assert e.value.status == dtp.DTP_ERR_UNSUPPORTED and "allocation-free scratch" in str(e.value)
