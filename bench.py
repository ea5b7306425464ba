#!/usr/bin/env python3
"""Benchmark of the compressed-MoE decode layer on one MI355X.

A step is one full layer call (route + top-k + gating, shared projections,
grouped gate/up, down and combine) on one batch of synthetic input; steps
rotate over several independently seeded layers so that the weights are read
from HBM, not from the 256 MB last-level cache. Prints one JSON line.

value  = compressed-weight bytes touched per step (active experts' codes and
         low-rank coefficients, plus the shared bases and code books) summed
         over the timed steps, divided by the timed wall time (GB/s).

Protocol: the rotated layers are drawn on the device (``synth_device``: the
synthetic recipe's laws, torch generators); one running input index runs
through the warm-up and every timed pass, so no pass starts on inputs the
previous one just read, and the rotation is sized so that more than 256 MB
(the last-level cache) is read between two visits of any input. Passes, each
followed by a check of the workspace status word: warm-up; a wall-clock pass
(``ms_per_step``, ``value``); a pass with a HIP event pair around every step
(per-step latency: median and a 10,000-resample bootstrap 95% interval,
Sec. 5.1's timing method); a pass with event pairs recorded by each kernel's
own dispatch (per-kernel durations, ``roofline``).
"""

from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "MoE-layer decode µs at batch 1/16; achieved HBM GB/s (% of peak)"
HBM_PEAK_GBPS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="qwen3_30b_a3b_moe_layer_b1")
    ap.add_argument("--also", default="qwen3_30b_a3b_moe_layer_b16,wide_h4096_i1536_e64_top6_b4_skewed,"
                    "qwen3_48_layer_decode_step_b16,deepseek_v2_lite_moe_layer_b1,"
                    "olmoe_1b_7b_moe_layer_b1,gemma4_26b_a4b_moe_layer_b1,"
                    "nemotron3_nano_moe_layer_b1,nemotron3_nano_moe_layer_b16",
                    help="comma-separated extra workloads timed the same way (reported under 'also')")
    ap.add_argument("--dense", default="qwen3_30b_a3b_moe_layer_b1,qwen3_30b_a3b_moe_layer_b16,"
                    "nemotron3_nano_moe_layer_b1,nemotron3_nano_moe_layer_b16",
                    help="workloads also timed with dense bf16 expert weights (the uncompressed "
                         "layer and the dense-down layer) on the same routing and inputs")
    ap.add_argument("--sweep", action="store_true",
                    help="instead of the benchmark line: time the Qwen3-shaped layer at batch 1 and "
                         "16 over block lengths d in {2, 4, 8} and ranks r in {0, 128, 256, 384, 512} "
                         "(the selections-versus-bytes trade-off) and print one JSON line")
    ap.add_argument("--gateup-ab", default="",
                    help="instead of the benchmark line: time these workloads (name or name@batch, "
                         "comma-separated) with code-word and with projection-code-book gate/up tiles "
                         "and print one JSON line")
    ap.add_argument("--layers", type=int, default=8, help="independently seeded layers rotated")
    ap.add_argument("--inputs", type=int, default=64,
                    help="distinct seeded inputs rotated (a multiple of --layers), so that the "
                         "experts touched over a rotation exceed the 256 MB last-level cache")
    ap.add_argument("--summarize-pmc", nargs=4, metavar=("FETCH_CSV", "WRITE_CSV", "CAL_FETCH_CSV",
                                                         "CAL_WRITE_CSV"),
                    help="write profiles/k_expert_<workload>_pmc.json from rocprofv3 --pmc "
                         "FETCH_SIZE / WRITE_SIZE counter CSVs of a bench run and of a "
                         "--calibrate-copy-mb run, then exit")
    ap.add_argument("--pmc-kernel", default="k_expert",
                    help="--summarize-pmc: substring of the kernel name summarized (e.g. "
                         "'k_expert<8, 1, 2>' for the dense layer's expert kernel)")
    ap.add_argument("--pmc-name", default=None,
                    help="--summarize-pmc: record name (default: --workload)")
    ap.add_argument("--summarize-counters", nargs="+", metavar="CSV",
                    help="print the mean per dispatch of every (kernel, counter) pair in rocprofv3 "
                         "--pmc counter CSVs as one JSON line, then exit")
    ap.add_argument("--calibrate-copy-mb", type=int, default=0,
                    help="only run a plain device copy of this many MiB (counter calibration)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="budget of the oracle sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    return ap.parse_args()


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2609_21137_amd", "csrc")
    for name in sorted(os.listdir(csrc)):
        if name.endswith((".hip", ".h")):
            with open(os.path.join(csrc, name), "rb") as f:
                h.update(name.encode() + f.read())
    return h.hexdigest()[:16]


def n_proj(w) -> int:
    """Input-side projections per expert: gate and up, or up alone."""
    return 1 if w.act == "relu2_up" else 2


def compressed_bytes(w, n_active: int, z_sep: bool = False) -> dict:
    """Algorithmic bytes of one step: what the method must read at least once.

    Per active expert: gate and up codes (H*I/d bytes each) and coefficients
    V (r*I bf16 each); down codes (I*H/d) and A (I*r bf16). Shared: the basis
    U (one per projection when separate), the output basis B and three code
    books. Up-only experts have no gate codes, coefficients or code book.
    The router weights are counted separately.
    """
    npj = n_proj(w)
    per_gateup = npj * (w.H * w.I // w.d) + npj * (w.r * w.I * 2)
    per_down = (w.I * w.H // w.d) + (w.I * w.r * 2)
    basis_u = (2 if z_sep else 1) * w.H * w.r * 2
    basis_b = w.r * w.H * 2
    codebooks = (npj + 1) * w.K * w.d * 2
    router = w.H * w.E * 2 + w.E * 4
    return {"compressed": n_active * (per_gateup + per_down) + basis_u + basis_b + codebooks,
            "expert_kernel": n_active * (per_gateup + per_down) + basis_b + codebooks,
            "route_kernel": router + basis_u,
            "per_expert_gateup": per_gateup, "per_expert_down": per_down}


def dense_bytes(w, n_active: int, form: str) -> dict:
    """Algorithmic bytes of one step of a dense-weight form: the active
    experts' bf16 matrices (and, for the dense-down form, the compressed
    gate/up factors, the basis U and two code books); router counted apart."""
    router = w.H * w.E * 2 + w.E * 4
    dn = w.I * w.H * 2
    if form == "dense":
        expert = n_active * (n_proj(w) * w.H * w.I * 2 + dn)
        return {"weights": expert, "expert_kernel": expert, "route_kernel": router}
    gu = 2 * (w.H * w.I // w.d) + 2 * (w.r * w.I * 2)
    expert = n_active * (gu + dn) + 2 * w.K * w.d * 2
    basis_u = w.H * w.r * 2
    return {"weights": expert + basis_u, "expert_kernel": expert, "route_kernel": router + basis_u}


def load_traffic(kernel: str, workload: str, src_hash: str):
    """HBM bytes per launch from committed rocprofv3 counter runs, if they were
    taken on the current kernel sources (else None)."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload}_pmc.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("kernel_source_hash") != src_hash:
        return None
    return rec.get("hbm_bytes_per_launch")


def dense_weights(torch, w, n_layers, dense_cache, form):
    """Dense bf16 expert matrices per rotated layer, drawn on the device
    (``synth_device``; drawing 1.2 GB per layer on the host would dominate
    the run)."""
    from paper_2609_21137_amd import synth_device
    key = (w.H, w.I, w.E, w.seed, form, w.act)
    if key not in dense_cache:
        dense_cache.clear()
        torch.cuda.empty_cache()
        if form == "dense":
            names = (("W_gate",) if n_proj(w) == 2 else ()) + ("W_up", "W_down")
        else:
            names = ("W_down",)
        dense_cache[key] = [synth_device.dense_tensors(w, li, names) for li in range(n_layers)]
    return dense_cache[key]


MALL_BYTES = 256 << 20


def device_layers(C, torch, w, n_layers, layers_cache):
    """``n_layers`` independently seeded layers of workload ``w`` on the device."""
    from paper_2609_21137_amd import synth_device
    key = (w.H, w.I, w.E, w.d, w.K, w.r, w.seed, w.hot_experts, w.hot_bias, w.act)
    have = layers_cache.get(key, [])
    if len(have) < n_layers:
        if not have:
            layers_cache.clear()
            torch.cuda.empty_cache()
        have = have + [C.DeviceLayer(synth_device.layer_tensors(w, li))
                       for li in range(len(have), n_layers)]
        layers_cache[key] = have
    return have[:n_layers]


def bootstrap_ci(v, n_boot=10_000, seed=0):
    """Median of v and the 2.5 / 97.5 percentiles of the median over
    ``n_boot`` resamples with replacement."""
    v = np.asarray(v, dtype=np.float64)
    rng = np.random.default_rng(seed)
    meds = np.median(v[rng.integers(0, len(v), size=(n_boot, len(v)))], axis=1)
    return float(np.median(v)), float(np.percentile(meds, 2.5)), float(np.percentile(meds, 97.5))


def hold_stream(torch, ms):
    """Keeps the current stream busy for about ``ms`` so the host can enqueue
    a whole pass ahead of the device (per-step event pairs then time the GPU,
    not host launch gaps). Returns False where torch has no sleep kernel."""
    try:
        torch.cuda._sleep(int(ms * 2.4e6))
        return True
    except Exception:
        return False


def time_workload(C, torch, w, steps, warmup, n_layers, n_inputs, layers_cache, form="compressed",
                  dense_cache=None):
    from paper_2609_21137_amd import synth
    shape = C.shape_of(w)
    dls = device_layers(C, torch, w, n_layers, layers_cache)
    # input j always runs on layer j % n_layers
    xs = [C.bf16_tensor(synth.workload_input(w, j % n_layers, step=j // n_layers))
          for j in range(n_inputs)]
    ws = C.new_workspace(shape, w.B)
    y = torch.empty((w.B, w.H), dtype=torch.float32, device="cuda")
    idx = torch.empty((w.B, w.top_k), dtype=torch.int32, device="cuda")
    wt = torch.empty((w.B, w.top_k), dtype=torch.float32, device="cuda")
    structs = [dl.struct() for dl in dls]

    # routing (hence the active-expert count) is fixed per (layer, input)
    # and the same in every form (the router weights are the layer's)
    up_only = w.act == "relu2_up"
    layer_call = C.moe_layer_relu2 if up_only else C.moe_layer
    n_act = []
    for j in range(n_inputs):
        layer_call(shape, xs[j], dls[j % n_layers], ws=ws, out=y, idx=idx, w=wt)
        torch.cuda.synchronize()
        n_act.append(len(np.unique(idx.cpu().numpy())))

    import ctypes
    lib = C.lib()
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    args_tail = (ctypes.c_void_p(y.data_ptr()), ctypes.c_void_p(idx.data_ptr()),
                 ctypes.c_void_p(wt.data_ptr()), ctypes.c_void_p(ws.data_ptr()), ws.numel(), stream)
    B = w.B
    if form == "compressed":
        fn = lib.cardan_moe_layer_relu2 if up_only else lib.cardan_moe_layer
        ptrs = [(ctypes.c_void_p(xs[j].data_ptr()), structs[j % n_layers]) for j in range(n_inputs)]

        def call(xp, st):
            return fn(ctypes.byref(shape), B, xp, ctypes.byref(st), *args_tail)
    elif form == "dense_down":
        fn = lib.cardan_moe_layer_dense_down
        mats = dense_weights(torch, w, n_layers, dense_cache, form)
        ptrs = [(ctypes.c_void_p(xs[j].data_ptr()),
                 (structs[j % n_layers], ctypes.c_void_p(mats[j % n_layers]["W_down"].data_ptr())))
                for j in range(n_inputs)]

        def call(xp, st):
            return fn(ctypes.byref(shape), B, xp, ctypes.byref(st[0]), st[1], *args_tail)
    else:
        fn = lib.cardan_dense_moe_layer_relu2 if up_only else lib.cardan_dense_moe_layer
        mats = dense_weights(torch, w, n_layers, dense_cache, form)
        dstructs = [C.DenseLayer({"router_w": dls[li].tensors["router_w"],
                                  "router_bias": dls[li].tensors["router_bias"], **mats[li]}).struct(
                                      shape, up_only=up_only)
                    for li in range(n_layers)]
        ptrs = [(ctypes.c_void_p(xs[j].data_ptr()), dstructs[j % n_layers]) for j in range(n_inputs)]

        def call(xp, st):
            return fn(ctypes.byref(shape), B, xp, ctypes.byref(st), *args_tail)

    def step_bytes(j):
        if form == "compressed":
            return compressed_bytes(w, n_act[j])
        b = dense_bytes(w, n_act[j], form)
        b["compressed"] = b["weights"]  # the form's own weight bytes
        return b

    per_input = [step_bytes(j)["compressed"] for j in range(n_inputs)]
    rotation = sum(per_input)
    pos = [0]  # one running input index through every pass

    def step():
        j = pos[0] % n_inputs
        pos[0] += 1
        xp, st = ptrs[j]
        rc = call(xp, st)
        if rc != 0:
            raise RuntimeError(lib.cardan_last_error().decode())
        return j

    def check_status(what):
        torch.cuda.synchronize()
        st = C.workspace_status(ws)
        if st != 0:
            raise RuntimeError(f"{w.name} ({form}): {st} in-kernel waits gave up during the {what}")

    for _ in range(warmup):
        step()
    check_status("warm-up")

    def pass_bytes(js):
        tot = {"compressed": 0, "expert_kernel": 0, "route_kernel": 0}
        for j in js:
            b = step_bytes(j)
            for k in tot:
                tot[k] += b[k]
        return tot

    # wall pass: exactly `steps` layer calls, bracketed by device syncs
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    js_wall = [step() for _ in range(steps)]
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    check_status("wall-clock pass")

    # per-step pass: an event pair around every layer call on the launch stream
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    held = hold_stream(torch, 0.05 * steps)
    js_ev = []
    for i in range(steps):
        ev[i][0].record()
        js_ev.append(step())
        ev[i][1].record()
    check_status("per-step event pass")
    per_step_us = [1e3 * a.elapsed_time(b) for a, b in ev]

    # kernel pass: event pairs recorded by each kernel's own dispatch
    C.profile_begin(steps)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    js_k = [step() for _ in range(steps)]
    torch.cuda.synchronize()
    wall_events = time.perf_counter() - t1
    prof = C.profile_end()
    check_status("kernel event pass")

    return {"wall_s": wall, "wall_events_s": wall_events, "prof": prof, "bytes": pass_bytes(js_wall),
            "bytes_kernel_pass": pass_bytes(js_k), "per_step_us": per_step_us, "stream_held": held,
            "mean_active": float(np.mean([n_act[j] for j in js_wall])), "layers": n_layers,
            "inputs": n_inputs, "rotation_bytes": rotation,
            "min_bytes_between_revisits": rotation - max(per_input)}


def time_decode_step(C, torch, w, steps, warmup, layers_cache):
    """The stacked-layer decode step: w.layers MoE layers with independently
    seeded weights (drawn on the device), each layer's output RMS-normalised
    (bf16) into the next layer's input. Two forms of the same step, each
    captured once as a HIP graph and replayed (eager launches are the
    fallback): the library's decode step (cardan_moe_decode_step: the
    normalisation inside the next layer's routing kernel; two kernels per
    layer) and the unfused chain
    (cardan_moe_layer, then cardan_rmsnorm_bf16: three kernels per layer).
    Per-step latency: an event pair around every replay."""
    import ctypes

    from paper_2609_21137_amd import synth
    shape = C.shape_of(w)
    B, L = w.B, w.layers
    dls = device_layers(C, torch, w, L, layers_cache)
    structs = [dl.struct() for dl in dls]
    arr = (C.LayerStruct * L)(*structs)
    x0 = C.bf16_tensor(synth.workload_input(w, 0))
    xa = torch.empty_like(x0)
    xb = torch.empty_like(x0)
    y = torch.empty((B, w.H), dtype=torch.float32, device="cuda")
    idx = torch.empty((L, B, w.top_k), dtype=torch.int32, device="cuda")
    wt = torch.empty((L, B, w.top_k), dtype=torch.float32, device="cuda")
    ws = C.new_workspace(shape, B)
    lib = C.lib()

    def fused(stream):
        rc = lib.cardan_moe_decode_step(ctypes.byref(shape), B, L, ctypes.c_void_p(x0.data_ptr()), arr,
                                        ctypes.c_float(1e-6), ctypes.c_void_p(y.data_ptr()), None,
                                        ctypes.c_void_p(idx.data_ptr()), ctypes.c_void_p(wt.data_ptr()),
                                        ctypes.c_void_p(ws.data_ptr()), ws.numel(), ctypes.c_void_p(stream))
        if rc != 0:
            raise RuntimeError(lib.cardan_last_error().decode())

    def unfused(stream):
        st = ctypes.c_void_p(stream)
        xin = x0
        for li in range(L):
            xout = xa if li % 2 == 0 else xb
            rc = lib.cardan_moe_layer(ctypes.byref(shape), B, ctypes.c_void_p(xin.data_ptr()),
                                      ctypes.byref(structs[li]), ctypes.c_void_p(y.data_ptr()),
                                      ctypes.c_void_p(idx[li].data_ptr()),
                                      ctypes.c_void_p(wt[li].data_ptr()),
                                      ctypes.c_void_p(ws.data_ptr()), ws.numel(), st)
            if rc != 0:
                raise RuntimeError(lib.cardan_last_error().decode())
            rc = lib.cardan_rmsnorm_bf16(B, w.H, ctypes.c_void_p(y.data_ptr()), ctypes.c_float(1e-6),
                                         ctypes.c_void_p(xout.data_ptr()), st)
            if rc != 0:
                raise RuntimeError(lib.cardan_last_error().decode())
            xin = xout

    def measure(one_step):
        stream = torch.cuda.current_stream().cuda_stream
        for _ in range(max(1, warmup)):
            one_step(stream)
        torch.cuda.synchronize()
        mode = "hip_graph"
        try:
            g = torch.cuda.CUDAGraph()
            s = torch.cuda.Stream()
            s.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(s):
                with torch.cuda.graph(g, stream=s):
                    one_step(torch.cuda.current_stream().cuda_stream)
            torch.cuda.current_stream().wait_stream(s)
            g.replay()
            torch.cuda.synchronize()
            run = g.replay
        except Exception as e:  # capture unsupported here: time the eager launches
            print(f"[bench] graph capture failed ({e}); timing eager launches", file=sys.stderr)
            mode = "eager"
            run = lambda: one_step(stream)  # noqa: E731
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            run()
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
        for a, b in ev:
            a.record()
            run()
            b.record()
        torch.cuda.synchronize()
        st = C.workspace_status(ws)
        if st != 0:
            raise RuntimeError(f"{w.name}: {st} in-kernel waits gave up")
        med, lo, hi = bootstrap_ci([a.elapsed_time(b) for a, b in ev])
        return mode, wall, med, lo, hi

    mode, wall, med, lo, hi = measure(fused)
    n_act = [len(np.unique(idx[li].cpu().numpy())) for li in range(L)]
    _, wall_u, med_u, lo_u, hi_u = measure(unfused)
    bytes_step = sum(compressed_bytes(w, a)["compressed"] for a in n_act)
    return {"workload": w.name, "B": B, "layers": L, "distinct_layers": len(dls), "mode": mode,
            "form": "cardan_moe_decode_step (normalisation fused into the next routing kernel)",
            "ms_per_step": round(1e3 * wall / steps, 4),
            "ms_per_step_median": round(med, 4), "ms_per_step_ci95": [round(lo, 4), round(hi, 4)],
            "us_per_layer": round(1e6 * wall / steps / L, 3),
            "us_per_layer_median": round(1e3 * med / L, 3),
            "GBps": round(bytes_step * steps / wall / 1e9, 2),
            "bytes_per_step": bytes_step,
            "mean_active_experts": float(np.mean(n_act)),
            "unfused_chain": {"ms_per_step": round(1e3 * wall_u / steps, 4),
                              "ms_per_step_median": round(med_u, 4),
                              "ms_per_step_ci95": [round(lo_u, 4), round(hi_u, 4)],
                              "us_per_layer": round(1e6 * wall_u / steps / L, 3)}}


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, budget_s):
    """The float64 oracle timed on this host's cores on a bounded sample: all
    the cores this process may use (the reported value), then one core."""
    import threadpoolctl

    import oracle.cardan_oracle as O
    from paper_2609_21137_amd import synth
    cores = len(os.sched_getaffinity(0))
    L = synth.workload_layer(w, 0)
    x = synth.workload_input(w, 0)

    def leg(threads, budget):
        n, t_tot, nbytes = 0, 0.0, 0
        with threadpoolctl.threadpool_limits(threads):
            while t_tot < budget or n == 0:
                t0 = time.perf_counter()
                _, idx, _, _ = O.moe_layer_factored(x, L, w.top_k, w.d)
                t_tot += time.perf_counter() - t0
                nbytes += compressed_bytes(w, len(np.unique(idx)))["compressed"]
                n += 1
        return n, t_tot, nbytes

    n, t_tot, nbytes = leg(cores, budget_s * 0.6)
    n1, t1, b1 = leg(1, budget_s * 0.4)
    return {"value": round(nbytes / t_tot / 1e9, 4), "unit": "GB/s", "cores": cores,
            "kind": "oracle", "cpu_model": cpu_model(),
            "sample": f"{n} steps of {w.name} (layer 0), float64 numpy factored form, "
                      f"{t_tot:.1f} s total, {1e3 * t_tot / n:.1f} ms/step",
            "one_core": {"value": round(b1 / t1 / 1e9, 4), "unit": "GB/s", "cores": 1,
                         "sample": f"{n1} steps, {t1:.1f} s total, {1e3 * t1 / n1:.1f} ms/step"}}


def summarize(w, r, src_hash, name=None):
    prof = r["prof"]
    steps = prof["expert"][1]
    ex_ms = prof["expert"][0] / max(1, steps)
    ex_bytes = r["bytes_kernel_pass"]["expert_kernel"] / max(1, steps)
    achieved = ex_bytes / (ex_ms * 1e-3) / 1e9
    name = name or w.name
    traffic = load_traffic("k_expert", name, src_hash)
    n = len(r["per_step_us"])
    med, lo, hi = bootstrap_ci(r["per_step_us"])
    return {
        "workload": name,
        "B": w.B,
        "us_per_layer": round(1e6 * r["wall_s"] / n, 3),
        "us_per_layer_median": round(med, 3),
        "us_per_layer_ci95": [round(lo, 3), round(hi, 3)],
        "us_per_layer_event_mean": round(float(np.mean(r["per_step_us"])), 3),
        "us_per_layer_with_kernel_events": round(1e6 * r["wall_events_s"] / n, 3),
        "GBps": round(r["bytes"]["compressed"] / r["wall_s"] / 1e9, 2),
        "GBps_median": round(r["bytes"]["compressed"] / n / (med * 1e-6) / 1e9, 2),
        "mean_active_experts": r["mean_active"],
        "kernel_us": {k: round(1e3 * v[0] / max(1, v[1]), 3) for k, v in prof.items() if v[1]},
        "roofline": {"kernel": "k_expert", "bound": "hbm", "achieved": round(achieved, 2),
                     "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": traffic,
                     "bytes_per_launch": round(ex_bytes)},
        "rotation": {"layers": r["layers"], "inputs": r["inputs"], "bytes": r["rotation_bytes"],
                     "min_bytes_between_revisits": r["min_bytes_between_revisits"],
                     "exceeds_last_level_cache": r["min_bytes_between_revisits"] > MALL_BYTES,
                     "per_step_pass_host_ahead": r["stream_held"]},
    }


def gateup_ab(C, torch, args):
    """Code-word against projection-code-book gate/up tiles (CARDAN_GATEUP)
    on the same layers and inputs, per workload; one JSON line."""
    import dataclasses

    from paper_2609_21137_amd.configs import WORKLOADS
    names = [n for n in args.gateup_ab.split(",") if n]
    rows = []
    cache = {}
    for name in names:
        base, _, b = name.partition("@")
        w = WORKLOADS[base]
        if b:
            w = dataclasses.replace(w, B=int(b), name=f"{base}_b{b}")
        row = {"workload": w.name, "B": w.B, "d": w.d}
        for form in ("codeword", "tbook", "codeword", "tbook"):  # twice, interleaved
            os.environ["CARDAN_GATEUP"] = form
            print(f"[gateup-ab] {w.name} {form}", file=sys.stderr, flush=True)
            rr = time_workload(C, torch, w, args.steps, args.warmup, w.rotate_layers or 2, args.inputs, cache)
            sm = summarize(w, rr, kernel_source_hash())
            row.setdefault(form, []).append({"us_per_layer_median": sm["us_per_layer_median"],
                                             "us_per_layer_ci95": sm["us_per_layer_ci95"],
                                             "kernel_us": sm["kernel_us"]})
        rows.append(row)
    os.environ.pop("CARDAN_GATEUP", None)
    print(json.dumps({"gateup_ab": "code-word vs projection-code-book gate/up tiles", "steps": args.steps,
                      "rows": rows, "kernel_source_hash": kernel_source_hash()}))


def sweep(C, torch, args):
    """Compressed layer latency over (d, r) at the Qwen3 shape, batches 1 and
    16, each point over two rotated layers (the touched experts of a rotation
    exceed the last-level cache)."""
    import dataclasses

    from paper_2609_21137_amd.configs import QWEN3_B1
    rows = []
    cache = {}
    for d in (8, 4, 2):
        for r in (0, 128, 256, 384, 512):
            for B in (1, 16):
                w = dataclasses.replace(QWEN3_B1, d=d, r=r, B=B, name=f"qwen3_shape_d{d}_r{r}_b{B}")
                print(f"[sweep] {w.name}", file=sys.stderr, flush=True)
                rr = time_workload(C, torch, w, args.steps, args.warmup, 2, args.inputs, cache)
                sm = summarize(w, rr, kernel_source_hash())
                per_e = compressed_bytes(w, 1)
                rows.append({"d": d, "r": r, "B": B, "us_per_layer": sm["us_per_layer"],
                             "GBps": sm["GBps"], "kernel_us": sm["kernel_us"],
                             "mean_active_experts": sm["mean_active_experts"],
                             "bytes_per_expert": per_e["per_expert_gateup"] + per_e["per_expert_down"],
                             "bits_per_weight": round(8.0 * (per_e["per_expert_gateup"] + per_e["per_expert_down"])
                                                      / (3 * w.H * w.I), 3)})
    print(json.dumps({"sweep": "qwen3 shape, compressed layer, (d, r) x batch", "steps": args.steps,
                      "rows": rows, "kernel_source_hash": kernel_source_hash()}))


def calibrate_copy(torch, mib):
    """A plain device-to-device copy of `mib` MiB, run 5 times: under
    rocprofv3 --pmc its FETCH_SIZE / WRITE_SIZE per dispatch against the
    known byte count gives the counter scale."""
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": n * 4, "launches": 5}))


def _pmc_means(path):
    """Mean counter value (KiB) per kernel name of a rocprofv3 counter CSV."""
    import csv
    acc = {}
    with open(path) as f:
        for row in csv.DictReader(f):
            acc.setdefault(row["Kernel_Name"], []).append(float(row["Counter_Value"]))
    return {k: (len(v), sum(v) / len(v)) for k, v in acc.items()}


def summarize_counters(paths):
    """Mean value per dispatch of each counter of each cardan kernel in
    rocprofv3 --pmc counter CSVs (several counters per run)."""
    import csv
    acc = {}
    for path in paths:
        with open(path) as f:
            for row in csv.DictReader(f):
                if "cardan" not in row["Kernel_Name"]:
                    continue
                key = (row["Kernel_Name"], row["Counter_Name"])
                acc.setdefault(key, []).append(float(row["Counter_Value"]))
    out = {}
    for (k, c), v in sorted(acc.items()):
        out.setdefault(k, {"dispatches": len(v)})[c] = round(sum(v) / len(v), 3)
    print(json.dumps({"kernel_source_hash": kernel_source_hash(), "per_dispatch_mean": out}))


def summarize_pmc(args):
    """HBM bytes per k_expert launch: FETCH_SIZE and WRITE_SIZE per dispatch,
    each scaled by what the same counter reads for a plain copy of known size."""
    fetch, write, cal_f, cal_w = (_pmc_means(p) for p in args.summarize_pmc)
    copy = "__amd_rocclr_copyBuffer"
    copy_bytes = args.calibrate_copy_mb * (1 << 20)
    f_scale = copy_bytes / (cal_f[copy][1] * 1024)
    w_scale = copy_bytes / (cal_w[copy][1] * 1024)
    name = next(k for k in fetch if args.pmc_kernel in k)
    wl = args.pmc_name or args.workload
    rec = {
        "kernel": name, "workload": wl, "kernel_source_hash": kernel_source_hash(),
        "dispatches": fetch[name][0],
        "FETCH_SIZE_KiB_per_dispatch": round(fetch[name][1], 3),
        "WRITE_SIZE_KiB_per_dispatch": round(write[name][1], 3),
        "copy_calibration": {"copy_bytes": copy_bytes, "FETCH_SIZE_KiB": round(cal_f[copy][1], 3),
                             "WRITE_SIZE_KiB": round(cal_w[copy][1], 3),
                             "fetch_scale": round(f_scale, 4), "write_scale": round(w_scale, 4)},
        "hbm_read_bytes_per_launch": round(fetch[name][1] * 1024 * f_scale),
        "hbm_write_bytes_per_launch": round(write[name][1] * 1024 * w_scale),
    }
    rec["hbm_bytes_per_launch"] = rec["hbm_read_bytes_per_launch"] + rec["hbm_write_bytes_per_launch"]
    kshort = "k_route" if "k_route" in name else "k_expert"
    out = os.path.join(ROOT, "profiles", f"{kshort}_{wl}_pmc.json")
    with open(out, "w") as f:
        json.dump(rec, f, indent=1)
        f.write("\n")
    print(json.dumps(rec))


def main():
    args = parse()
    if args.summarize_counters:
        summarize_counters(args.summarize_counters)
        return
    if args.summarize_pmc:
        if not args.calibrate_copy_mb:
            print("--summarize-pmc needs --calibrate-copy-mb (the calibration copy size)",
                  file=sys.stderr)
            sys.exit(2)
        summarize_pmc(args)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU: this build has no multi-GPU path "
              f"(asked for --gpus {args.gpus}).", file=sys.stderr)
        sys.exit(2)
    import torch

    from paper_2609_21137_amd import cardan as C
    from paper_2609_21137_amd.configs import WORKLOADS
    if not torch.cuda.is_available():
        print("no GPU visible", file=sys.stderr)
        sys.exit(1)
    if args.calibrate_copy_mb:
        calibrate_copy(torch, args.calibrate_copy_mb)
        return
    if args.gateup_ab:
        gateup_ab(C, torch, args)
        return
    if args.sweep:
        sweep(C, torch, args)
        return
    if args.inputs % args.layers:
        print("--inputs must be a multiple of --layers", file=sys.stderr)
        sys.exit(2)
    src_hash = kernel_source_hash()
    w = WORKLOADS[args.workload]
    cache = {}
    print(f"[bench] {w.name}: drawing {args.layers} layers on the device", file=sys.stderr, flush=True)
    r = time_workload(C, torch, w, args.steps, args.warmup, args.layers, args.inputs, cache)
    main_sum = summarize(w, r, src_hash)
    print(f"[bench] {w.name}: {main_sum['us_per_layer']} us/layer", file=sys.stderr, flush=True)
    also = []
    for name in [s for s in args.also.split(",") if s]:
        ww = WORKLOADS[name]
        if ww.layers > 1:
            print(f"[bench] {ww.name}: {ww.layers}-layer decode step", file=sys.stderr, flush=True)
            also.append(time_decode_step(C, torch, ww, max(5, args.steps // 4), 2, cache))
            print(f"[bench] {ww.name}: {also[-1]['ms_per_step']} ms/step", file=sys.stderr, flush=True)
            continue
        print(f"[bench] {ww.name}", file=sys.stderr, flush=True)
        rr = time_workload(C, torch, ww, args.steps, args.warmup, ww.rotate_layers or args.layers,
                           args.inputs, cache)
        also.append(summarize(ww, rr, src_hash))
        print(f"[bench] {ww.name}: {also[-1]['us_per_layer']} us/layer", file=sys.stderr,
              flush=True)
    # the same workloads with dense bf16 expert weights: the uncompressed layer
    # and the dense-down layer, on the compressed layers' routing and inputs
    dense_cache = {}
    by_name = {main_sum["workload"]: main_sum, **{a["workload"]: a for a in also}}
    for name in [s for s in args.dense.split(",") if s]:
        ww = WORKLOADS[name]
        # the dense-down form has gate and up projections (no up-only variant)
        forms = (("dense", "_dense_bf16"),) + (() if ww.act == "relu2_up" else (("dense_down", "_dense_down"),))
        for form, suffix in forms:
            print(f"[bench] {ww.name} ({form})", file=sys.stderr, flush=True)
            rr = time_workload(C, torch, ww, args.steps, args.warmup, args.layers, args.inputs, cache,
                               form=form, dense_cache=dense_cache)
            sm = summarize(ww, rr, src_hash, name=ww.name + suffix)
            sm["form"] = form
            sm["weight_GBps"] = sm.pop("GBps")
            comp = by_name.get(ww.name)
            if comp is not None:
                sm["compressed_us_per_layer"] = comp["us_per_layer"]
                sm["compressed_speedup"] = round(sm["us_per_layer"] / comp["us_per_layer"], 3)
            also.append(sm)
            print(f"[bench] {ww.name} ({form}): {sm['us_per_layer']} us/layer", file=sys.stderr,
                  flush=True)
        dense_cache.clear()
    cache.clear()
    cpu = None
    if not args.no_cpu_baseline:
        print("[bench] cpu baseline (oracle)", file=sys.stderr, flush=True)
        cpu = cpu_baseline(w, args.cpu_seconds)
    steps = args.steps
    line = {
        "metric": METRIC,
        "value": main_sum["GBps"],
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": args.warmup,
        "ms_per_step": round(1e3 * r["wall_s"] / steps, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "H": w.H, "I": w.I, "E": w.E, "top_k": w.top_k, "d": w.d,
                   "K": w.K, "r": w.r, "B": w.B, "layers_rotated": args.layers,
                   "inputs_rotated": args.inputs,
                   "parallelism": "none"},
        "us_per_layer": main_sum["us_per_layer"],
        "us_per_layer_median": main_sum["us_per_layer_median"],
        "us_per_layer_ci95": main_sum["us_per_layer_ci95"],
        "hbm_frac_of_peak": round(main_sum["GBps"] / HBM_PEAK_GBPS, 4),
        "rotation": main_sum["rotation"],
        "kernel_us": main_sum["kernel_us"],
        "mean_active_experts": main_sum["mean_active_experts"],
        "us_per_layer_with_kernel_events": main_sum["us_per_layer_with_kernel_events"],
        "roofline": main_sum["roofline"],
        "cpu_baseline": cpu,
        "also": also,
        "kernel_source_hash": src_hash,
    }
    print(json.dumps(line))


if __name__ == "__main__":
    main()
