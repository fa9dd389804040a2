#!/usr/bin/env python3
"""Benchmark of the affinity-aware sharding hot path on one MI355X.

A step is one pass of the whole path over one layer's calibration batch: fold the
weights, accumulate the first-order up affinity over all tokens, encode it, and run the
coordinate ascent (exact neuron assignment on the host, partition scores on the GPU).
Steps run as a calibration over many layers runs them: step k's ascent on a second
stream while step k+1's fold and affinity pass occupy the GPU (``serial_ms_per_step``
gives the same steps one after another).  The default workload is the Qwen3-0.6B-shaped
layer: d=1024, I=3072, 16 query / 8 KV heads of 128, 65,536 tokens, L=2 logical devices,
bf16.  Inputs are synthetic and seeded (generated on the device before timing).

The JSON line reports calibration tokens/s per layer (value), the MFMA roofline of the
dominant kernel timed with HIP events on its launch stream, and the fp64 oracle timed on
a bounded token sample on the host cores.  ``full_model`` gives the full-model layout time
of the 28-layer Qwen3-0.6B-shaped model (262,144 tokens per layer, L=4), the 16-layer
Danube3-500M-shaped model (131,072 tokens, L=2 and 4) and the 4-layer 8B-class stack
(131,072 tokens, L=4), each with its affinity TFLOP/s and the oracle's tokens/s beside it;
``layout.layer_optimum`` gives the ascent's gap to the exact optimum of the layer.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6   # MI355X dense bf16 MFMA
METRIC = "affinity calibration tokens/s per layer + % bf16 MFMA peak; full-model layout time"
KERNEL_SRC = os.path.join(ROOT, "paper_2609_13846_amd", "csrc", "affinity.hip")
PROFILES = os.path.join(ROOT, "profiles")


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def flops_per_token(wl) -> float:
    """Algorithmic FLOPs per token: operating point 4*I*d plus per-head products 4*I*H*dh."""
    return 4.0 * wl.n_neurons * (wl.n_q_heads * wl.head_dim + wl.d_model)


def kernel_hash() -> str:
    return hashlib.sha256(open(KERNEL_SRC, "rb").read()).hexdigest()[:16]


def traffic_record(wl):
    """The committed PMC summary of the affinity kernel (HBM bytes, MFMA busy fraction and
    clock per launch), if it was taken on this kernel source and workload; else {}."""
    try:
        rec = json.load(open(os.path.join(PROFILES, f"affinity_traffic_{wl.name}.json")))
    except (OSError, ValueError):
        return {}
    if rec.get("kernel_sha") != kernel_hash() or rec.get("workload") != wl.name:
        return {}
    return rec


def make_layer(dtp, synth, wl, layer_idx, device):
    w = synth.device_weights(wl, layer_idx, device)
    layer = dtp.dtp_layer_create(wl.d_model, wl.n_neurons, wl.n_q_heads, wl.n_kv_groups,
                                 wl.head_dim, wl.rms_eps,
                                 dtp.DTP_BF16 if wl.dtype == "bf16" else dtp.DTP_F32)
    return layer, w


def library_gemm(torch, device, wl, tokens):
    """A plain bf16 torch.matmul (the vendor GEMM library) with the FLOPs of one affinity
    launch: [tokens x (d + H*dh)] @ [(d + H*dh) x 2I], no epilogue.  Context for the fused
    kernel's fraction of peak: what a library GEMM of the same size reaches on this GPU."""
    K = wl.d_model + wl.n_q_heads * wl.head_dim
    gen = torch.Generator(device=device).manual_seed(0)
    a = torch.randn(tokens, K, device=device, dtype=torch.bfloat16, generator=gen)
    b = torch.randn(K, 2 * wl.n_neurons, device=device, dtype=torch.bfloat16, generator=gen) * 0.02
    for _ in range(3):
        c = a @ b
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    reps = 10
    e0.record()
    for _ in range(reps):
        c = a @ b
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    tflops = 2.0 * tokens * K * 2 * wl.n_neurons / (ms * 1e-3) / 1e12
    del a, b, c
    return {"what": f"torch.matmul bf16 [{tokens} x {K}] @ [{K} x {2 * wl.n_neurons}], no epilogue",
            "ms": ms, "tflops": tflops, "frac": tflops / PEAK_BF16_TFLOPS}


def cpu_baseline(wl, x, attn, w, L, n_tokens):
    """The oracle as it stands on the first n_tokens of the workload (host cores)."""
    import numpy as np
    from threadpoolctl import threadpool_info, threadpool_limits

    from oracle import affinity as orc
    from oracle import layout as lay

    xs = x[:n_tokens].float().cpu().numpy().astype(np.float64)
    as_ = attn[:n_tokens].float().cpu().numpy().astype(np.float64)
    wts = {k: w[k].float().cpu().numpy().astype(np.float64) for k in ("w_o", "gamma", "w_gate", "w_up", "w_down")}
    cores = len(os.sched_getaffinity(0))
    with threadpool_limits(limits=cores):
        blas_threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
        t0 = time.perf_counter()
        A = orc.affinity_folded(xs, as_, wts["w_o"], wts["gamma"], wts["w_gate"], wts["w_up"],
                                wts["w_down"], wl.n_kv_groups, wl.rms_eps)
        t1 = time.perf_counter()
        lay.coordinate_ascent([lay.encode(A.astype(np.float32))], None, L)
        t2 = time.perf_counter()
        # the literal form (every p_h materialised in model space) on a smaller sample
        n_lit = max(1, min(n_tokens, n_tokens // 24))
        orc.affinity_literal(xs[:n_lit], as_[:n_lit], wts["w_o"], wts["gamma"], wts["w_gate"],
                             wts["w_up"], wts["w_down"], wl.n_kv_groups, wl.rms_eps)
        t3 = time.perf_counter()
    return {"value": n_tokens / (t2 - t0), "unit": "tokens/s", "cores": int(min(cores, blas_threads)),
            "kind": "oracle",
            "sample": f"first {n_tokens} tokens of the {wl.name} workload, all {wl.n_neurons} neurons: "
                      f"fp64 folded affinity ({t1 - t0:.1f} s) + exact layout optimiser ({t2 - t1:.1f} s)",
            "affinity_tokens_per_s": {
                "folded": n_tokens / (t1 - t0),
                "literal": n_lit / (t3 - t2),
                "literal_sample": f"first {n_lit} tokens ({t3 - t2:.1f} s)"}}


def oracle_rate(wl, w, x, attn, n_tokens):
    """The oracle as it stands (fp64 folded affinity, all neurons) on the first n_tokens of
    layer 0 of a workload, on the host cores: tokens per second per layer."""
    import numpy as np
    from threadpoolctl import threadpool_info, threadpool_limits

    from oracle import affinity as orc

    xs = x[:n_tokens].float().cpu().numpy().astype(np.float64)
    as_ = attn[:n_tokens].float().cpu().numpy().astype(np.float64)
    wts = {k: w[k].float().cpu().numpy().astype(np.float64) for k in ("w_o", "gamma", "w_gate", "w_up", "w_down")}
    cores = len(os.sched_getaffinity(0))
    with threadpool_limits(limits=cores):
        blas_threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
        t0 = time.perf_counter()
        orc.affinity_folded(xs, as_, wts["w_o"], wts["gamma"], wts["w_gate"], wts["w_up"], wts["w_down"],
                            wl.n_kv_groups, wl.rms_eps)
        dt = time.perf_counter() - t0
    return {"tokens_per_s": n_tokens / dt, "cores": int(min(cores, blas_threads)), "kind": "oracle",
            "sample": f"first {n_tokens} tokens of layer 0, all {wl.n_neurons} neurons, fp64 folded "
                      f"affinity including its fold ({dt:.1f} s)"}


ORACLE_SAMPLE = {"qwen3-0.6b-model": 8192, "danube3-500m": 8192, "8b-class-4layer": 1024}


def full_model(dtp, synth, device, torch, name, with_oracle=True):
    """Full-model layout time: every layer's fold + affinity (up edge, and the down edge into
    the next layer), then encode + ascent to convergence for each shard count.  One
    untimed pass over the first layer and chunk warms the kernels first."""
    wl = synth.WORKLOADS[name]
    N, G, I = wl.n_layers, wl.n_kv_groups, wl.n_neurons
    nch = wl.tokens // wl.chunk
    dt = dtp.DTP_BF16 if wl.dtype == "bf16" else dtp.DTP_F32
    log(f"full model {name}: generating {N} layers x {wl.tokens} tokens on the device")
    layers, weights, attn_w, data = [], [], [], []
    for i in range(N):
        layer, w = make_layer(dtp, synth, wl, i, device)
        layers.append(layer)
        weights.append(w)
        attn_w.append(synth.device_attn_weights(wl, i, device))
        data.append([synth.device_tokens(wl, i, w, wl.chunk, c, device, with_pre=True)
                     for c in range(nch)])
    A = torch.zeros(N, G, I, dtype=torch.float32, device=device)
    s_down = torch.zeros(max(N - 1, 1), I, dtype=torch.float32, device=device)
    B = torch.zeros(G, I, dtype=torch.float32, device=device)
    A_down = torch.zeros(max(N - 1, 1), I, G, dtype=torch.float32, device=device)

    def layer_pass(i, chunks):
        w = weights[i]
        dtp.dtp_layer_set_weights(layers[i], w["w_o"], w["gamma"], w["w_gate"], w["w_up"], w["w_down"])
        for c in range(chunks):
            x, a, _ = data[i][c]
            if i + 1 < N:
                x_next = data[i + 1][c][2]   # residual entering layer i+1's attention pre-norm
                dtp.dtp_affinity_accumulate_down(layers[i], x, a, x_next, wl.rms_eps, x.shape[0], A[i],
                                                 s_down[i])
            else:
                dtp.dtp_affinity_accumulate(layers[i], x, a, x.shape[0], A[i])
        if i + 1 < N:
            an = attn_w[i + 1]
            dtp.dtp_down_weights(wl.d_model, I, wl.n_q_heads, G, wl.head_dim, dt, an["w_q"], an["w_k"],
                                 an["w_v"], an["gamma"], w["w_down"], B)
            dtp.dtp_down_affinity(I, G, s_down[i], B, A_down[i])

    layer_pass(0, 1)                      # warm-up (kernels, allocator), then start clean
    for L in wl.shards:
        dtp.dtp_coordinate_ascent(N, G, I, L, A + 1.0, (A_down + 1.0) if N > 1 else None)
    A.zero_()
    s_down.zero_()
    A_down.zero_()
    torch.cuda.synchronize()
    log(f"full model {name}: timing")
    t0 = time.perf_counter()
    for i in range(N):
        layer_pass(i, nch)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    f_alg = flops_per_token(wl) * wl.tokens * N
    out = {"workload": wl.name, "layers": N, "tokens_per_layer": wl.tokens, "affinity_s": t1 - t0,
           "affinity_tflops": f_alg / (t1 - t0) / 1e12,
           "affinity_frac_of_peak": f_alg / (t1 - t0) / 1e12 / PEAK_BF16_TFLOPS,
           "tokens_per_s_per_layer": wl.tokens * N / (t1 - t0),
           "edges": 2 * N - 1, "by_shards": []}
    for L in wl.shards:
        ta = time.perf_counter()
        res = dtp.dtp_coordinate_ascent(N, G, I, L, A, A_down if N > 1 else None)
        tb = time.perf_counter()
        out["by_shards"].append({"shards": L, "optimiser_s": tb - ta, "layout_time_s": (t1 - t0) + (tb - ta),
                                 "sweeps": res["sweeps"], "J": res["J"],
                                 "J_random_expectation": (2 * N - 1) / L})
    for layer in layers:
        dtp.dtp_layer_destroy(layer)
    if with_oracle:
        n = ORACLE_SAMPLE.get(name, 1024)
        log(f"full model {name}: oracle on {n} tokens of layer 0")
        x0, a0, _ = data[0][0]
        out["oracle"] = oracle_rate(wl, weights[0], x0, a0, n)
    del data
    torch.cuda.empty_cache()
    out["context"] = "paper: affinity pass + optimisation under two minutes per model on one RTX 5090"
    return out


def layer_optimum(dtp, A, G, I, shard_counts):
    """The ascent's J against the exact optimum of the layer (every head partition up to
    relabelling, each with its exact neuron step), for each shard count."""
    import numpy as np
    Q = dtp.dtp_encode_affinity(A.cpu().numpy())
    out = {}
    for L in shard_counts:
        if G % L or I % L:
            continue
        ca = dtp.dtp_coordinate_ascent(1, G, I, L, A)
        t0 = time.perf_counter()
        _, _, J_opt = dtp.dtp_layer_optimum(G, I, L, Q)
        t1 = time.perf_counter()
        out[f"L{L}"] = {"J_opt": J_opt / 2.0 ** 48, "J_ca": ca["J"], "gap": (J_opt - ca["J_fixed"]) / J_opt,
                        "optimum_s": t1 - t0}
    assert all(np.isfinite(v["J_opt"]) for v in out.values())
    return out


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="qwen3-0.6b-layer")
    ap.add_argument("--cpu-sample-tokens", type=int, default=49152)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-library-gemm", action="store_true",
                    help="skip the library GEMM of the same FLOPs (context, untimed)")
    ap.add_argument("--full-model", nargs="*", default=None, metavar="WORKLOAD",
                    help="workloads of the full-model layout time (default: "
                         "qwen3-0.6b-model danube3-500m 8b-class-4layer)")
    ap.add_argument("--no-full-model", action="store_true", help="skip the full-model layout time")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of this many MiB (HBM counter scale)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: the shard count is a logical layout parameter and the "
              "path runs on a single device; --gpus must be 1", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2609_13846_amd import dtp, synth

    device = torch.device("cuda", 0)
    torch.cuda.set_device(device)
    if args.copy_calibration:
        n = args.copy_calibration << 20
        src = torch.empty(n, dtype=torch.uint8, device=device).fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": n, "launches": 3}), flush=True)
        return
    wl = synth.WORKLOADS[args.workload]
    L = wl.shards[0]
    T, G, I = wl.tokens, wl.n_kv_groups, wl.n_neurons
    log(f"workload {wl.name}: T={T} d={wl.d_model} I={I} H={wl.n_q_heads} G={G} dh={wl.head_dim} L={L}")
    layer, w = make_layer(dtp, synth, wl, 0, device)
    x, attn = synth.device_tokens(wl, 0, w, T, 0, device)
    # Two affinity buffers: a step's ascent reads one while the next step's affinity fills
    # the other.
    A_buf = [torch.zeros(G, I, dtype=torch.float32, device=device) for _ in range(2)]
    A = A_buf[0]
    main_stream = torch.cuda.current_stream()
    ascent_stream = torch.cuda.Stream()  # default priority
    torch.cuda.synchronize()

    def gpu_part(Ak):
        dtp.dtp_layer_set_weights(layer, w["w_o"], w["gamma"], w["w_gate"], w["w_up"], w["w_down"])
        Ak.zero_()
        dtp.dtp_affinity_accumulate(layer, x, attn, T, Ak)

    def step():
        gpu_part(A)
        return dtp.dtp_coordinate_ascent(1, G, I, L, A)   # synchronises the stream

    def pipelined_steps(K):
        """K steps, each the fold, the affinity pass and the ascent of one layer, as a
        calibration over many layers runs them: step k's ascent (host neuron steps, small
        kernels) on a second stream while step k+1's fold and affinity occupy the GPU."""
        done = [torch.cuda.Event() for _ in range(2)]
        gpu_part(A_buf[0])
        done[0].record(main_stream)
        r = None
        for k in range(K):
            if k + 1 < K:
                gpu_part(A_buf[(k + 1) % 2])
                done[(k + 1) % 2].record(main_stream)
            ascent_stream.wait_event(done[k % 2])
            r = dtp.dtp_coordinate_ascent(1, G, I, L, A_buf[k % 2], stream=ascent_stream)
            main_stream.wait_stream(ascent_stream)  # the buffer's next fill follows its ascent
        return r

    for _ in range(args.warmup):
        res = step()
    # The second stream's first ascent sets up its stream-ordered memory; done here, with
    # the GPU otherwise idle, it does not stall an affinity launch running beside it.
    dtp.dtp_coordinate_ascent(1, G, I, L, A, stream=ascent_stream)
    pipelined_steps(2)
    # phase breakdown (untimed pass with synchronisation between phases)
    torch.cuda.synchronize()
    b0 = time.perf_counter()
    dtp.dtp_layer_set_weights(layer, w["w_o"], w["gamma"], w["w_gate"], w["w_up"], w["w_down"])
    torch.cuda.synchronize()
    b1 = time.perf_counter()
    A.zero_()
    dtp.dtp_affinity_accumulate(layer, x, attn, T, A)
    torch.cuda.synchronize()
    b2 = time.perf_counter()
    dtp.dtp_coordinate_ascent(1, G, I, L, A)
    b3 = time.perf_counter()
    # the same steps one after another, each ascent waiting for its own affinity pass
    torch.cuda.synchronize()
    s0 = time.perf_counter()
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    serial_ms = (time.perf_counter() - s0) * 1e3 / args.steps

    log(f"timing {args.steps} steps")
    dtp.dtp_layer_profile(layer, 1)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    res = pipelined_steps(args.steps)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    kern_ms, launches = dtp.dtp_layer_profile_read(layer)
    dtp.dtp_layer_profile(layer, 0)
    # The paper's approximate neuron step against the exact one, on this layer's affinity
    # (untimed): J of the ascent with each, at the workload's shard count and at L = 4.
    neuron_steps = {}
    for Ls in sorted({L, 4}):
        if G % Ls or I % Ls:
            continue
        ex = dtp.dtp_coordinate_ascent(1, G, I, Ls, A)
        du = dtp.dtp_coordinate_ascent(1, G, I, Ls, A, dual_ascent_neurons=True)
        neuron_steps[f"L{Ls}"] = {"J_exact": ex["J"], "J_dual_ascent": du["J"],
                                  "relative_gap": (ex["J"] - du["J"]) / ex["J"]}
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    value = T / (ms_per_step * 1e-3)
    # The library splits a call into slices, one kernel launch each: the algorithmic work
    # of a launch is the FLOPs of the tokens it covers.
    launches_per_step = launches / max(args.steps, 1)
    f_launch = flops_per_token(wl) * T / max(launches_per_step, 1)
    avg_ms = kern_ms / max(launches, 1)
    achieved = f_launch / (avg_ms * 1e-3) / 1e12
    pmc = traffic_record(wl)
    out = {
        "metric": METRIC,
        "value": value,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded, generated on the device; shapes and distributions of the workload)",
        "config": {"workload": wl.name, "tokens": T, "d_model": wl.d_model, "n_neurons": I,
                   "n_q_heads": wl.n_q_heads, "n_kv_groups": G, "head_dim": wl.head_dim,
                   "shards": L, "parallelism": "single GPU; shards are logical"},
        "roofline": {"bound": "mfma", "kernel": "affinity_bf16_kernel",
                     "achieved": achieved, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": achieved / PEAK_BF16_TFLOPS, "traffic": pmc.get("bytes_per_launch"),
                     "traffic_gbs": (pmc["bytes_per_launch"] / (avg_ms * 1e-3) / 1e9
                                     if pmc.get("bytes_per_launch") else None),
                     "mfma_busy_pmc": pmc.get("mfma_busy"), "clock_ghz_pmc": pmc.get("clock_ghz"),
                     "wave_cycles_pmc": pmc.get("wave_cycles"),
                     "avg_launch_ms": avg_ms, "launches": launches,
                     "tokens_per_launch": T / max(launches_per_step, 1),
                     "flops_per_launch": f_launch},
        "step_tflops": flops_per_token(wl) * T / (ms_per_step * 1e-3) / 1e12,
        "pipelining": "step k's ascent runs on a second stream beside step k+1's fold and "
                      "affinity; every step does all its work",
        "serial_ms_per_step": serial_ms,
        "breakdown_ms": {"fold": (b1 - b0) * 1e3, "affinity": (b2 - b1) * 1e3,
                         "layout": (b3 - b2) * 1e3},
        "layout": {"J": res["J"], "sweeps": res["sweeps"], "neuron_step": neuron_steps,
                   "layer_optimum": layer_optimum(dtp, A, G, I, sorted({L, 4}))},
        "context": "paper: 65,536-token affinity pass of a 28-layer model in 51 s on one RTX 5090",
    }
    if not args.no_library_gemm:
        out["roofline"]["library_gemm_same_flops"] = library_gemm(
            torch, device, wl, int(T / max(launches_per_step, 1)))
    if not args.no_cpu_baseline:
        log(f"cpu baseline: oracle on {args.cpu_sample_tokens} tokens")
        out["cpu_baseline"] = cpu_baseline(wl, x, attn, w, L, args.cpu_sample_tokens)
    dtp.dtp_layer_destroy(layer)
    if not args.no_full_model:
        del x, attn
        torch.cuda.empty_cache()
        names = args.full_model or ["qwen3-0.6b-model", "danube3-500m", "8b-class-4layer"]
        out["full_model"] = [full_model(dtp, synth, device, torch, n, with_oracle=not args.no_cpu_baseline)
                             for n in names]
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
