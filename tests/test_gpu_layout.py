"""GPU head step and coordinate ascent against the exact oracle, bit for bit.

Given the same affinity, partition scores, neuron assignments, layouts, J_int and the
number of sweeps must be identical; from independently computed affinities (GPU bf16 vs
oracle fp64) the final co-located affinity must agree within 1e-3 relative.
"""
import sys

import numpy as np
import pytest
import torch

from oracle import affinity as orc
from oracle import dual_ascent as da
from oracle import layout as lay
from paper_2609_13846_amd import dtp, synth
from tests import helpers as hp

pytestmark = pytest.mark.gpu


def announce(msg):
    print(f"[gpu] {msg}", file=sys.stderr, flush=True)


def rand_A(rng, shape):
    return (rng.gamma(0.4, size=shape) * 1e-3).astype(np.float32)


@pytest.mark.parametrize("G,I,L,down,minimise", [
    (8, 3072, 4, False, False), (8, 3072, 4, True, False), (8, 3072, 2, True, False),
    (8, 4096, 2, False, True), (4, 128, 2, True, False), (8, 14336, 4, True, False),
    # unusual group and device counts: 40,320, 12,870, 34,650, 2 and 1 partitions
    (8, 512, 8, True, False), (16, 256, 2, False, False), (12, 96, 3, True, True),
    (2, 8, 2, True, False), (4, 32, 1, True, False),
])
def test_partition_scores_bit_exact(G, I, L, down, minimise):
    announce(f"partition scores G={G} I={I} L={L} down={down} min={minimise}")
    rng = np.random.default_rng(G + I + L)
    Qu = lay.encode(rand_A(rng, (G, I)))
    nu = rng.permutation(np.arange(I) // (I // L)).astype(np.int32)
    Qd = lay.encode(rand_A(rng, (I, G))) if down else None
    nup = rng.permutation(np.arange(I) // (I // L)).astype(np.int32) if down else None
    P = dtp.dtp_partition_count(G, L)
    scores = torch.zeros(P, dtype=torch.int64, device="cuda")
    dev = lambda v: None if v is None else torch.from_numpy(v).cuda()
    best = dtp.dtp_partition_scores(G, I, L, dev(Qu), dev(nu), dev(Qd), dev(nup), minimise, scores)
    C = lay.head_gain(Qu, nu, L, Qd, nup)
    parts = lay.partitions(G, L)
    ref = lay.partition_scores(C, parts)
    np.testing.assert_array_equal(scores.cpu().numpy(), ref)
    assert best == lay.best_partition(ref, minimise)


def test_partition_scores_refuse_more_than_2_pow_24_partitions():
    """G = 16 over L = 4 devices has 63,063,000 labelled partitions, beyond the 2^24 the
    scoring supports: refused before any work, whatever the buffers."""
    G, I, L = 16, 64, 4
    assert dtp.dtp_partition_count(G, L) == 63063000
    Qu = torch.zeros(G, I, dtype=torch.int64, device="cuda")
    nu = torch.zeros(I, dtype=torch.int32, device="cuda")
    scores = torch.zeros(1, dtype=torch.int64, device="cuda")
    with pytest.raises(dtp.DtpError) as e:
        lib = dtp.lib()
        best = dtp._I64()
        dtp._check(lib.dtp_partition_scores(G, I, L, Qu.data_ptr(), nu.data_ptr(), None, None, 0,
                                            scores.data_ptr(), dtp.ctypes.byref(best), None))
    assert e.value.status == dtp.DTP_ERR_UNSUPPORTED


def test_partition_scores_ties_take_lowest_rank():
    announce("partition scores ties")
    G, I, L = 8, 64, 4
    Qu = np.zeros((G, I), np.int64)
    nu = (np.arange(I) // (I // L)).astype(np.int32)
    scores = torch.zeros(2520, dtype=torch.int64, device="cuda")
    best = dtp.dtp_partition_scores(G, I, L, torch.from_numpy(Qu).cuda(), torch.from_numpy(nu).cuda(),
                                    None, None, False, scores)
    assert best == 0


@pytest.mark.parametrize("N,G,I,L,down", [(1, 8, 3072, 2, False), (4, 8, 3072, 4, True),
                                          (3, 8, 4096, 2, True), (2, 4, 128, 2, True),
                                          (2, 8, 64, 8, True), (2, 16, 96, 2, True)])
def test_coordinate_ascent_bit_exact(N, G, I, L, down):
    announce(f"coordinate ascent N={N} G={G} I={I} L={L} down={down}")
    rng = np.random.default_rng(N * 100 + L)
    Au = rand_A(rng, (N, G, I))
    Ad = rand_A(rng, (N - 1, I, G)) if down else None
    res = dtp.dtp_coordinate_ascent(N, G, I, L, torch.from_numpy(Au).cuda(),
                                    None if Ad is None else torch.from_numpy(Ad).cuda())
    Qu = [lay.encode(Au[i]) for i in range(N)]
    Qd = [lay.encode(Ad[i]) for i in range(N - 1)] if down else None
    hs, nus, J, sweeps = lay.coordinate_ascent(Qu, Qd, L)
    np.testing.assert_array_equal(res["h"], np.array(hs))
    np.testing.assert_array_equal(res["nu"], np.array(nus))
    assert res["J_fixed"] == J
    assert res["sweeps"] == sweeps
    assert res["J"] == J / 2 ** 48


def test_coordinate_ascent_modes_bit_exact():
    announce("coordinate ascent modes")
    rng = np.random.default_rng(9)
    N, G, I, L = 4, 8, 256, 4
    Au = rand_A(rng, (N, G, I))
    Ad = rand_A(rng, (N - 1, I, G))
    Qu = [lay.encode(Au[i]) for i in range(N)]
    Qd = [lay.encode(Ad[i]) for i in range(N - 1)]
    du, dd = torch.from_numpy(Au).cuda(), torch.from_numpy(Ad).cuda()
    for kw in [dict(freeze_heads=True), dict(freeze_neurons=True), dict(minimise=True),
               dict(layer_mask=[1, 0, 1, 0]), dict(max_sweeps=1)]:
        res = dtp.dtp_coordinate_ascent(N, G, I, L, du, dd, **kw)
        hs, nus, J, sweeps = lay.coordinate_ascent(Qu, Qd, L, **kw)
        np.testing.assert_array_equal(res["h"], np.array(hs), err_msg=str(kw))
        np.testing.assert_array_equal(res["nu"], np.array(nus), err_msg=str(kw))
        assert res["J_fixed"] == J and res["sweeps"] == sweeps, kw


@pytest.mark.parametrize("N,G,I,L,down", [(1, 8, 3072, 4, False), (3, 8, 1024, 4, True),
                                          (2, 8, 3072, 2, True)])
def test_coordinate_ascent_with_dual_ascent_neurons_bit_exact(N, G, I, L, down):
    """The ascent with the paper's approximate neuron step, against the oracle ascent with
    the oracle of that step; with L = 2 it also equals the exact ascent."""
    announce(f"coordinate ascent, dual-ascent neurons N={N} G={G} I={I} L={L} down={down}")
    rng = np.random.default_rng(N * 31 + L)
    Au = rand_A(rng, (N, G, I))
    Ad = rand_A(rng, (N - 1, I, G)) if down else None
    res = dtp.dtp_coordinate_ascent(N, G, I, L, torch.from_numpy(Au).cuda(),
                                    None if Ad is None else torch.from_numpy(Ad).cuda(),
                                    dual_ascent_neurons=True)
    Qu = [lay.encode(Au[i]) for i in range(N)]
    Qd = [lay.encode(Ad[i]) for i in range(N - 1)] if down else None
    step = lambda M, minimise: da.assign(-M if minimise else M)[0]
    hs, nus, J, sweeps = lay.coordinate_ascent(Qu, Qd, L, neuron_step=step)
    np.testing.assert_array_equal(res["h"], np.array(hs))
    np.testing.assert_array_equal(res["nu"], np.array(nus))
    assert res["J_fixed"] == J and res["sweeps"] == sweeps
    exact = lay.coordinate_ascent(Qu, Qd, L)
    if L == 2:
        assert J == exact[2]


def test_layout_from_gpu_affinity_matches_oracle_objective():
    """Affinity from the GPU and from the oracle (same inputs) lead to layouts whose
    co-located affinity, measured on the oracle's matrix, agrees within 1e-3."""
    wl = synth.WORKLOADS["qwen3-0.6b-layer"]
    T = 2048
    w = synth.host_weights(wl, 0)
    x, a = synth.host_tokens(wl, 0, w, T)
    announce("layout from GPU affinity, qwen3-0.6b-layer T=2048")
    A_gpu = hp.gpu_affinity(wl, w, x, a)
    A_ref = orc.affinity_folded(**hp.oracle_inputs(w, x, a), n_kv_groups=wl.n_kv_groups, eps=wl.rms_eps)
    hp.assert_affinity_close(A_gpu, A_ref)
    L = 2
    res = dtp.dtp_coordinate_ascent(1, wl.n_kv_groups, wl.n_neurons, L, torch.from_numpy(A_gpu).cuda())
    Q_ref = lay.encode(A_ref.astype(np.float32))
    hs, nus, J_ref, _ = lay.coordinate_ascent([Q_ref], None, L)
    J_gpu_layout = lay.objective([Q_ref], None, [res["h"][0]], [res["nu"][0]])
    assert abs(J_gpu_layout - J_ref) <= 1e-3 * J_ref
    # and the library reproduces the oracle's layout bit for bit on the GPU's own matrix
    hs2, nus2, J2, _ = lay.coordinate_ascent([lay.encode(A_gpu)], None, L)
    np.testing.assert_array_equal(res["nu"][0], nus2[0])
    assert res["J_fixed"] == J2


def test_concurrent_ascents_from_several_threads_match_serial():
    """Four host threads, each with its own stream, run coordinate ascents at once (chains
    with down edges, L = 2 and 4, and a call that fails on a degenerate matrix); every
    result equals the same call run alone, and each failure reports its own error.  This
    exercises the pinned staging pool, the stream-ordered scratch and the per-thread error
    message under concurrency."""
    import threading
    announce("concurrent coordinate ascents, 4 threads")
    rng = np.random.default_rng(77)
    cases = []
    for t in range(8):
        N, L = (3, 4) if t % 2 else (2, 2)
        G, I = 8, 512
        Au = torch.from_numpy(rand_A(rng, (N, G, I))).cuda()
        Ad = torch.from_numpy(rand_A(rng, (N - 1, I, G))).cuda()
        cases.append((N, G, I, L, Au, Ad))
    bad = torch.zeros(1, 8, 512, dtype=torch.float32, device="cuda")  # all zero: degenerate
    torch.cuda.synchronize()
    serial = [dtp.dtp_coordinate_ascent(*c) for c in cases]
    results, errors = {}, {}

    def worker(w):
        stream = torch.cuda.Stream()
        for rep in range(3):
            for i in range(w, len(cases), 4):
                results[(w, rep, i)] = dtp.dtp_coordinate_ascent(*cases[i], stream=stream)
            try:
                dtp.dtp_coordinate_ascent(1, 8, 512, 2, bad, stream=stream)
                errors[(w, rep)] = None
            except dtp.DtpError as e:
                errors[(w, rep)] = e.status

    threads = [threading.Thread(target=worker, args=(w,)) for w in range(4)]
    for th in threads:
        th.start()
    for th in threads:
        th.join()
    assert len(results) == 3 * len(cases)
    for (w, rep, i), res in results.items():
        ref = serial[i]
        np.testing.assert_array_equal(res["h"], ref["h"])
        np.testing.assert_array_equal(res["nu"], ref["nu"])
        assert res["J_fixed"] == ref["J_fixed"] and res["sweeps"] == ref["sweeps"]
    assert all(s == dtp.DTP_ERR_DEGENERATE for s in errors.values()) and len(errors) == 12


def test_ascent_beside_the_next_affinity_pass_matches_serial():
    """Steps as a calibration over many layers runs them (and as bench.py times them): step
    k's ascent on a second stream, after an event marking its affinity pass done, while
    step k+1's fold and affinity pass fill the other of two buffers on the first stream.
    Each step's layout, J and sweep count equal the same step run alone."""
    announce("ascent beside the next affinity pass, 4 steps")
    wl = synth.WORKLOADS["qwen3-0.6b-layer"]
    G, I, L, T = wl.n_kv_groups, wl.n_neurons, 2, 8192
    dev = torch.device("cuda", 0)
    w = synth.device_weights(wl, 0, dev)
    toks = [synth.device_tokens(wl, 0, w, T, c, dev) for c in range(4)]
    layer = hp.layer_for(wl)
    try:
        def gpu_part(c, A):
            dtp.dtp_layer_set_weights(layer, w["w_o"], w["gamma"], w["w_gate"], w["w_up"], w["w_down"])
            A.zero_()
            dtp.dtp_affinity_accumulate(layer, toks[c][0], toks[c][1], T, A)

        A = torch.zeros(G, I, device=dev)
        serial = []
        for c in range(4):
            gpu_part(c, A)
            serial.append(dtp.dtp_coordinate_ascent(1, G, I, L, A))
        bufs = [torch.zeros(G, I, device=dev) for _ in range(2)]
        main, side = torch.cuda.current_stream(), torch.cuda.Stream()
        done = [torch.cuda.Event() for _ in range(2)]
        piped = []
        gpu_part(0, bufs[0])
        done[0].record(main)
        for k in range(4):
            if k + 1 < 4:
                gpu_part(k + 1, bufs[(k + 1) % 2])
                done[(k + 1) % 2].record(main)
            side.wait_event(done[k % 2])
            piped.append(dtp.dtp_coordinate_ascent(1, G, I, L, bufs[k % 2], stream=side))
            main.wait_stream(side)
        torch.cuda.synchronize()
    finally:
        dtp.dtp_layer_destroy(layer)
    assert len({r["J_fixed"] for r in serial}) > 1  # the steps differ
    for r, ref in zip(piped, serial):
        np.testing.assert_array_equal(r["h"], ref["h"])
        np.testing.assert_array_equal(r["nu"], ref["nu"])
        assert r["J_fixed"] == ref["J_fixed"] and r["sweeps"] == ref["sweeps"]
