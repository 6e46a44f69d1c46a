"""Benchmark of one expert server's forward step on one MI355X.

A step is one eaas_expert_forward over one batch of the named synthetic
workload (routing, grouped gate/up GEMM + SiLU*mul, grouped down GEMM into
by-slot rows, weighted combine), inputs resident in HBM.  Prints one JSON line.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_FP8_TFLOPS = 5000.0    # MI355X dense fp8 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E


def cpu_threads() -> int:
    n = len(os.sched_getaffinity(0))
    omp = os.environ.get("OMP_NUM_THREADS")
    return min(n, int(omp)) if omp and omp.isdigit() else n


def algorithmic(d: dict, counts: np.ndarray) -> dict:
    """Algorithmic flops and bytes of the step and of each GEMM kernel."""
    T, H, I, E, k = d["T"], d["H"], d["I"], d["E"], d["k"]
    R = int(counts.sum())
    n_act = int((counts > 0).sum())
    wb = 1 if d["wdtype"] == "fp8" else 2
    sgu = (2 * I // 128) * (H // 128) * 4 if wb == 1 else 0
    sdn = (H // 128) * (I // 128) * 4 if wb == 1 else 0
    if d.get("act8"):
        # fp8 activations: x and h enter the GEMMs as e4m3 codes (1 byte) plus
        # one fp32 scale per row and 128 channels
        gu_bytes = n_act * (2 * I * H + sgu) + T * H + T * H // 32 + R * I + R * I // 32 + R * 4
        dn_bytes = n_act * (H * I + sdn) + R * I + R * I // 32 + T * H * 2 + R * 4
    else:
        gu_bytes = n_act * (2 * I * H * wb + sgu) + T * H * 2 + R * I * 2 + R * 4
        dn_bytes = n_act * (H * I * wb + sdn) + R * I * 2 + T * H * 2 + R * 4
    return dict(flops=6.0 * R * H * I, gu_flops=4.0 * R * H * I, dn_flops=2.0 * R * H * I,
                gu_bytes=gu_bytes, dn_bytes=dn_bytes, bytes=gu_bytes + dn_bytes + T * k * 4)


def gate_up_kernel_name(d: dict) -> str:
    """The gate/up kernel the library dispatches for this workload's shape."""
    T, I, E, k = d["T"], d["I"], d["E"], d["k"]
    if d.get("act8"):
        return "grouped_gemm_w8a8_kernel<gate/up>"
    if d["wdtype"] == "fp8":
        return "grouped_gemm_dma_kernel<gate/up, fp8 weights>"
    if (2 * I) % 256:
        return "grouped_gemm_kernel<gate/up, register-staged>"
    return "grouped_gemm_pp_kernel<gate/up>"


def kernel_source_sha256() -> str:
    h = hashlib.sha256()
    for f in ("gemm.hip", "common.h", "internal.h"):
        with open(os.path.join(ROOT, "paper_2509_17863_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(workload: str):
    """HBM bytes per gate/up launch from the committed rocprofv3 FETCH_SIZE and
    WRITE_SIZE runs of this workload, scaled by a copy kernel of known size;
    None when there is no record or the kernel sources changed since."""
    path = os.path.join(ROOT, "profiles", f"kernels_{workload}.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m = re.search(r"```json\n(\{.*?\})\n```", text, re.S)
    if not m:
        return None
    rec = json.loads(m.group(1))
    if rec.get("kernel_source_sha256") != kernel_source_sha256():
        return None
    return int(rec["traffic_bytes"])


def host_info() -> dict:
    """CPU model of the host and the BLAS NumPy calls (the oracle's matmuls)."""
    model = None
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    blas = None
    try:
        b = np.show_config(mode="dicts")["Build Dependencies"]["blas"]
        blas = f"{b.get('name')} {b.get('version')}"
        conf = b.get("openblas configuration")
        if conf:
            blas += f" ({conf})"
    except Exception:  # noqa: BLE001 - metadata only
        pass
    return {"cpu_model": model, "blas": blas, "numpy": np.__version__}


def _median_runs(run, T: int, target_s: float, repeats: int = 3):
    """Calibrate a token count so one run takes about target_s, then time
    `repeats` runs on fresh samples of that size; the median rate."""
    n = min(T, 64)
    t = run(n)
    if t < target_s and n < T:
        n = int(min(T, max(n, n * target_s / max(t, 1e-3))))
    times = [run(n) for _ in range(repeats)]
    return n, times


def cpu_baseline(d: dict, target_s: float = 5.0) -> dict:
    """The oracle, untuned, on bounded token samples of the same batch
    (weights pre-converted to fp64 outside the timed region); median of 3."""
    from oracle import eaas_oracle as O

    if d.get("act8"):
        return cpu_baseline_w8a8(d, target_s)

    E = d["E"]
    w64 = ([], [])
    for e in range(E):
        wg, wu, wd = O.expert_weights_f64(d, e)
        w64[0].append(np.concatenate([wg, wu]))
        w64[1].append(wd)
    rng = np.random.default_rng(7)

    def run(n):
        tok = np.sort(rng.choice(d["T"], size=n, replace=False))
        sub = O.sub_batch(d, tok)
        t0 = time.perf_counter()
        O.expert_forward(sub, weights=w64)
        return time.perf_counter() - t0

    n, times = _median_runs(run, d["T"], target_s)
    t = float(np.median(times))
    flops = 6.0 * n * d["k"] * d["H"] * d["I"]
    return {"value": round(n / t, 1), "unit": "tokens/s", "cores": cpu_threads(), "kind": "oracle",
            "gflops": round(flops / t / 1e9, 1), "runs_s": [round(x, 2) for x in times],
            **host_info(),
            "sample": f"{n} of {d['T']} tokens of the same batch, median of {len(times)} runs "
                      f"on fresh samples (oracle expert_forward on the sub-batch, fp64 BLAS; "
                      "weights converted to fp64 beforehand)"}


def cpu_baseline_w8a8(d: dict, target_s: float = 5.0) -> dict:
    """The fp8-activation oracle, untuned, on bounded token samples (it
    dequantizes each active expert's weights inside the timed region);
    median of 3."""
    from oracle import eaas_oracle as O
    from oracle import w8a8_oracle as W

    rng = np.random.default_rng(7)

    def run(n):
        tok = np.sort(rng.choice(d["T"], size=n, replace=False))
        sub = O.sub_batch(d, tok)
        t0 = time.perf_counter()
        W.expert_forward_w8a8(sub)
        return time.perf_counter() - t0

    n, times = _median_runs(run, d["T"], target_s)
    t = float(np.median(times))
    return {"value": round(n / t, 1), "unit": "tokens/s", "cores": cpu_threads(), "kind": "oracle",
            "runs_s": [round(x, 2) for x in times], **host_info(),
            "sample": f"{n} of {d['T']} tokens of the same batch, median of {len(times)} runs "
                      "(fp8-activation oracle on the sub-batch, fp64 BLAS, including the "
                      "per-expert weight dequantization)"}


def time_graph(step, steps: int, warmup: int) -> tuple[float, dict]:
    """ms per step of `step` captured once in a graph and replayed (wall clock
    over all replays), and the median / p10 / p90 of the replays' event times
    (a second pass, each replay bracketed by events on the replay stream)."""
    import torch

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for _ in range(warmup):
        g.replay()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        g.replay()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(steps)]
    cur = torch.cuda.current_stream()
    for a, b in ev:
        a.record(cur)
        g.replay()
        b.record(cur)
    torch.cuda.synchronize()
    t = np.array([a.elapsed_time(b) for a, b in ev])
    return ms, {"median": round(float(np.median(t)), 4), "p10": round(float(np.percentile(t, 10)), 4),
                "p90": round(float(np.percentile(t, 90)), 4)}


def gpu_clocks() -> dict | None:
    """Current engine (sclk) and memory (mclk) clock levels of the first GPU
    from sysfs (the level marked '*'); None where the files are absent."""
    import glob

    out = {}
    for dev in sorted(glob.glob("/sys/class/drm/card*/device")):
        for name in ("pp_dpm_sclk", "pp_dpm_mclk", "pp_dpm_fclk"):
            try:
                with open(os.path.join(dev, name)) as fh:
                    for line in fh:
                        if "*" in line:
                            m = re.search(r"(\d+)\s*[Mm]hz", line)
                            if m:
                                out[name[-4:]] = int(m.group(1))
            except OSError:
                pass
        if out:
            return out
    return None


def time_segments(d: dict, dev: dict, clients: int, steps: int, warmup: int, ms_single: float,
                  tiled: bool = False):
    """The same batch as `clients` requests in separate buffers, through
    eaas_expert_forward_segments (counts on the device, capacity T)."""
    import torch

    from paper_2509_17863_amd import eaas

    T, H, I, E, k = d["T"], d["H"], d["I"], d["E"], d["k"]
    bounds = np.linspace(0, T, clients + 1).astype(int)
    bufs = []
    for a, b in zip(bounds[:-1], bounds[1:]):
        bufs.append((dev["x"][a:b].clone(), dev["topk_ids"][a:b].clone(),
                     dev["topk_weights"][a:b].clone(),
                     torch.empty((max(b - a, 1), H), dtype=torch.bfloat16, device="cuda")))
    table = eaas.segment_table(bufs)
    counts = torch.tensor(np.diff(bounds), dtype=torch.int32, device="cuda")
    act8 = bool(d.get("act8"))
    wdt = (eaas.EAAS_FP8_E4M3_A8 if act8 else eaas.EAAS_FP8_E4M3) if d["wdtype"] == "fp8" \
        else eaas.EAAS_BF16
    if tiled:
        wdt = eaas.EAAS_FP8_E4M3_TILED
    ws = eaas.alloc_segments_workspace(T, H, I, E, k, wdt)

    def step():
        eaas.eaas_expert_forward_segments(table, counts, clients, T, k, dev["w_gate_up"],
                                          dev["w_down"], ws, eaas.EAAS_BF16,
                                          dev["w_gate_up_scale"], dev["w_down_scale"],
                                          act8=act8, tiled=tiled)
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    return {"entry": "eaas_expert_forward_segments", "clients": clients,
            "tokens_per_client": f"{int(np.diff(bounds).min())}-{int(np.diff(bounds).max())}",
            "ms_per_step": round(ms, 4), "value": round(T / (ms * 1e-3), 1), "unit": "tokens/s",
            "vs_single_batch": round(ms / ms_single, 4)}


def time_server(d: dict, dev: dict, n_slots: int, steps: int, warmup: int, ms_single: float,
                tiled: bool = False):
    """The batch spread over `n_slots` client slots of one layer, served by
    eaas_server_step.  The step writes its results over the hidden states, so
    before every step the clients' requests are posted again: the hidden
    states are copied back into the payloads and all flags set ready (a copy
    of T*H bf16 and a fill kernel, inside the timed loop)."""
    import torch

    from paper_2509_17863_amd import eaas

    T, H, I, E, k = d["T"], d["H"], d["I"], d["E"], d["k"]
    bounds = np.linspace(0, T, n_slots + 1).astype(int)
    flags = torch.ones(n_slots, dtype=torch.int32, device="cuda")
    hdr = torch.tensor([[0, b - a] for a, b in zip(bounds[:-1], bounds[1:])], dtype=torch.int32,
                       device="cuda")
    slots = [(flags[i:i + 1], hdr[i], dev["x"][a:b].clone(), dev["topk_ids"][a:b].clone(),
              dev["topk_weights"][a:b].clone())
             for i, (a, b) in enumerate(zip(bounds[:-1], bounds[1:]))]
    stab = eaas.slot_table(slots)
    ltab = eaas.layer_table([(dev["w_gate_up"], dev["w_gate_up_scale"], dev["w_down"],
                              dev["w_down_scale"])])
    act8 = bool(d.get("act8"))
    wdt = (eaas.EAAS_FP8_E4M3_A8 if act8 else eaas.EAAS_FP8_E4M3) if d["wdtype"] == "fp8" \
        else eaas.EAAS_BF16
    if tiled:
        wdt = eaas.EAAS_FP8_E4M3_TILED
    ws = eaas.alloc_server_workspace(T, H, I, E, k, 1, wdt)

    def step():
        for i, (a, b) in enumerate(zip(bounds[:-1], bounds[1:])):
            slots[i][2].copy_(dev["x"][a:b])
        flags.fill_(eaas.EAAS_SLOT_READY)
        eaas.eaas_server_step(stab, n_slots, ltab, 1, T, H, I, E, k, ws, wdt)
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    done = int((flags == eaas.EAAS_SLOT_DONE).sum().item())
    return {"entry": "eaas_server_step", "slots": n_slots, "slots_done_last_step": done,
            "timed": "re-post of every request (payload copy, flags) + server step",
            "ms_per_step": round(ms, 4), "value": round(T / (ms * 1e-3), 1), "unit": "tokens/s",
            "vs_single_batch": round(ms / ms_single, 4)}


def measure(name: str, steps: int, warmup: int, tiled_fp8: bool = True):
    """Time eaas_expert_forward on one workload: a graph-replayed pass for the
    step time and an eager pass with events between the kernels."""
    import torch

    from paper_2509_17863_amd import eaas, synth
    from paper_2509_17863_amd.device_io import to_device

    wl = synth.WORKLOADS[name]
    d = synth.make_workload(name)
    dev = to_device(d)
    T, H, I, E, k = d["T"], d["H"], d["I"], d["E"], d["k"]
    act8 = bool(d.get("act8"))
    wdt = (eaas.EAAS_FP8_E4M3_A8 if act8 else eaas.EAAS_FP8_E4M3) if d["wdtype"] == "fp8" \
        else eaas.EAAS_BF16
    # fp8 weights (bf16 activations) are rearranged once, as a server would
    # when it loads them, into the tiled layout the fp8 GEMMs stream
    tiled = tiled_fp8 and wdt == eaas.EAAS_FP8_E4M3 and H % 256 == 0
    if tiled:
        for key, which in (("w_gate_up", eaas.EAAS_GATE_UP), ("w_down", eaas.EAAS_DOWN)):
            t = torch.empty_like(dev[key])
            eaas.eaas_tile_weights_fp8(dev[key], which, H, I, t)
            dev[key] = t
        torch.cuda.synchronize()
        wdt = eaas.EAAS_FP8_E4M3_TILED
    ws = eaas.alloc_workspace(T, H, I, E, k, wdt)
    out = torch.empty((T, H), dtype=torch.bfloat16, device="cuda")
    counts = np.bincount(d["topk_ids"].ravel()[d["topk_ids"].ravel() >= 0], minlength=E)
    alg = algorithmic(d, counts)

    stream = torch.cuda.current_stream()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(steps)]

    def step(ev=None):
        if ev is None:
            eaas.eaas_expert_forward(dev["x"], dev["topk_ids"], dev["topk_weights"],
                                     dev["w_gate_up"], dev["w_down"], out, ws,
                                     dev["w_gate_up_scale"], dev["w_down_scale"], act8=act8,
                                     tiled=tiled)
        else:
            eaas.eaas_expert_forward_profiled(dev["x"], dev["topk_ids"], dev["topk_weights"],
                                              dev["w_gate_up"], dev["w_down"], out, ws,
                                              dev["w_gate_up_scale"], dev["w_down_scale"],
                                              events=ev, act8=act8, tiled=tiled)

    for ev in evs:  # create the events before the timed region
        for e in ev:
            e.record(stream)
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        step(evs[i])
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms = (t1 - t0) * 1e3 / steps

    def mean_ms(a, b):
        return float(np.mean([evs[i][a].elapsed_time(evs[i][b]) for i in range(steps)]))

    # the step as the paper deploys it (§4.3): captured once in a graph, then
    # replayed; the same kernels with no launches from the host per step
    ms_graph, graph_stats = time_graph(step, steps, warmup)

    t_route, t_gu, t_dn, t_comb = mean_ms(0, 1), mean_ms(1, 2), mean_ms(2, 3), mean_ms(3, 4)
    t_step_ev = mean_ms(0, 4)
    # the gate/up launch's bound: HBM when its algorithmic intensity is below
    # the ridge of the MFMA peak it runs on (fp8 x fp8 with fp8 activations,
    # bf16 otherwise), the matrix cores above it
    peak_flops = PEAK_FP8_TFLOPS if act8 else PEAK_BF16_TFLOPS
    intensity = alg["gu_flops"] / alg["gu_bytes"]
    hbm_bound = intensity < peak_flops * 1e12 / (PEAK_HBM_GBS * 1e9)
    if hbm_bound:
        achieved = alg["gu_bytes"] / (t_gu * 1e-3) / 1e9
        roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4)}
    else:
        # a contraction is priced against the MFMA peak of its own dtype
        achieved = alg["gu_flops"] / (t_gu * 1e-3) / 1e12
        roof = {"bound": "mfma", "achieved": round(achieved, 1), "peak": peak_flops,
                "unit": "TFLOP/s", "frac": round(achieved / peak_flops, 4)}
    roof["traffic"] = measured_traffic(name)
    roof["traffic_unit"] = "bytes per launch"
    roof["algorithmic_bytes"] = int(alg["gu_bytes"])
    roof["algorithmic_flops"] = alg["gu_flops"]
    roof["launch_ms"] = round(t_gu, 4)
    roof["kernel"] = gate_up_kernel_name(d) + (", tiled weights" if tiled else "")
    res = {
        "value": round(T / (ms_graph * 1e-3), 1),
        "ms_per_step": round(ms_graph, 4),
        "graph_replay_ms": graph_stats,
        "eager": {"ms_per_step": round(ms, 4), "value": round(T / (ms * 1e-3), 1),
                  "graph_speedup": round(ms / ms_graph, 4)},
        "dtype": "fp8e4m3" if act8 else "bf16",
        "config": {"workload": name, "T": T, "H": H, "I": I, "E": E, "k": k,
                   "weights": d["wdtype"], "activations": "fp8e4m3" if act8 else "bf16",
                   "weight_layout": "tiled" if tiled else "row_major",
                   "seed": wl.seed, "zipf": wl.zipf,
                   "active_experts": int((counts > 0).sum()), "parallelism": "none (1 GPU)"},
        "step_tflops": round(alg["flops"] / (ms_graph * 1e-3) / 1e12, 1),
        "step_frac_bf16_peak": round(alg["flops"] / (ms_graph * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
        # the two grouped GEMMs alone: 6RHI over their summed event times
        "gemm_tflops": round(alg["flops"] / ((t_gu + t_dn) * 1e-3) / 1e12, 1),
        "gemm_frac_bf16_peak": round(alg["flops"] / ((t_gu + t_dn) * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 4),
        "kernels_ms": {"route": round(t_route, 4), "gate_up": round(t_gu, 4),
                       "down": round(t_dn, 4), "combine": round(t_comb, 4),
                       "step_events": round(t_step_ev, 4)},
        "down_tflops": round(alg["dn_flops"] / (t_dn * 1e-3) / 1e12, 1),
        "roofline": roof,
    }
    if hbm_bound:
        # the weight-streaming regime: algorithmic bytes of both GEMMs over
        # the whole replayed step, and the gate/up launch alone
        step_gbs = (alg["gu_bytes"] + alg["dn_bytes"]) / (ms_graph * 1e-3) / 1e9
        res["step_hbm_gbs"] = round(step_gbs, 1)
        res["step_hbm_frac"] = round(step_gbs / PEAK_HBM_GBS, 4)
    res["_tiled"] = tiled
    return res, d, dev, ms


def scheduler_ablation(d: dict, dev: dict, steps: int, warmup: int, tiled: bool = False) -> dict:
    """The step with each build of the GEMM tile scheduler (§4.1
    group-shrink ablation): the compacted active-expert list (the library),
    the same parallel prefix scan over all E experts, and every workgroup
    walking the E experts with one global read per expert.  Same inputs,
    libraries interleaved twice; the outputs must agree bit for bit."""
    import torch

    from paper_2509_17863_amd import _build, eaas

    T, H, I, E, k = d["T"], d["H"], d["I"], d["E"], d["k"]
    act8 = bool(d.get("act8"))
    wdt = (eaas.EAAS_FP8_E4M3_A8 if act8 else eaas.EAAS_FP8_E4M3) if d["wdtype"] == "fp8" \
        else eaas.EAAS_BF16
    if tiled:
        wdt = eaas.EAAS_FP8_E4M3_TILED
    variants = {"group_shrink": None, "scan_all": _build.variant_library("scan_all"),
                "walk_all": _build.variant_library("walk_all")}
    ws = eaas.alloc_workspace(T, H, I, E, k, wdt)
    out = torch.empty((T, H), dtype=torch.bfloat16, device="cuda")
    times = {n: [] for n in variants}
    kern = {n: [] for n in variants}
    same = {}
    ref = None
    try:
        for _ in range(2):
            for name, path in variants.items():
                eaas.use_library(path)

                def step(ev=None):
                    args = (dev["x"], dev["topk_ids"], dev["topk_weights"], dev["w_gate_up"],
                            dev["w_down"], out, ws, dev["w_gate_up_scale"], dev["w_down_scale"])
                    if ev is None:
                        eaas.eaas_expert_forward(*args, act8=act8, tiled=tiled)
                    else:
                        eaas.eaas_expert_forward_profiled(*args, events=ev, act8=act8,
                                                          tiled=tiled)

                ms, _ = time_graph(step, steps, warmup)
                times[name].append(ms)
                evs = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(steps)]
                for ev in evs:
                    step(ev)
                torch.cuda.synchronize()
                kern[name].append([float(np.mean([ev[a].elapsed_time(ev[a + 1]) for ev in evs]))
                                   for a in range(4)])
                bits = out.view(torch.int16).clone()
                if ref is None:
                    ref = bits
                same[name] = same.get(name, True) and bool(torch.equal(bits, ref))
    finally:
        eaas.use_library(None)
    base = float(np.median(times["group_shrink"]))
    res = {}
    for name in variants:
        t = float(np.median(times[name]))
        kmean = np.mean(np.array(kern[name]), axis=0)
        res[name] = {"ms_per_step": round(t, 4), "vs_group_shrink": round(t / base, 4),
                     "gate_up_ms": round(float(kmean[1]), 4), "down_ms": round(float(kmean[2]), 4),
                     "runs_ms": [round(x, 4) for x in times[name]], "bitwise_equal": same[name]}
    return res


def decode_summary(r: dict) -> dict:
    """The decode-sized workload's figures for the headline line."""
    out = {"workload": r["config"]["workload"], "config": r["config"],
           "ms_per_step": r["ms_per_step"], "value": r["value"], "unit": "tokens/s",
           "graph_replay_ms": r["graph_replay_ms"], "kernels_ms": r["kernels_ms"],
           "gate_up_roofline": r["roofline"]}
    for key in ("step_hbm_gbs", "step_hbm_frac"):
        if key in r:
            out[key] = r[key]
    return out


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="dsv3_prefill",
                    help="headline workload (default: the DeepSeek-V3-shaped prefill shard, "
                         "the largest configuration)")
    ap.add_argument("--decode-workload", default="dsv3_decode",
                    help="decode-sized workload timed in the same run for the HBM figures")
    ap.add_argument("--no-decode", action="store_true")
    ap.add_argument("--row-major-fp8", action="store_true",
                    help="time fp8 weights in their row-major [E,N,K] layout instead of the "
                         "tiled layout of eaas_tile_weights_fp8")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--scheduler-ablation", action="store_true",
                    help="also time the step with the two other builds of the GEMM tile "
                         "scheduler (all E experts scanned; all E walked with a global read "
                         "each) on the headline workload")
    ap.add_argument("--server-slots", type=int, default=0,
                    help="also time the server step over this many client slots holding the "
                         "batch (flags set ready before every step)")
    ap.add_argument("--clients", type=int, default=0,
                    help="also time the dynamic-batch entry point with the batch split into "
                         "this many client requests (token counts read on the device)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one expert server on one GPU; --gpus {args.gpus} is not "
              "supported (the step has no cross-GPU exchange; experts shard by server)",
              file=sys.stderr)
        return 2

    import torch

    assert torch.cuda.is_available(), "no GPU"
    clocks_before = gpu_clocks()
    r, d, dev, ms_eager = measure(args.workload, args.steps, args.warmup,
                                  tiled_fp8=not args.row_major_fp8)
    clocks_after = gpu_clocks()
    res = {
        "metric": "expert-FFN tokens/s",
        "value": r["value"],
        "unit": "tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": r["ms_per_step"],
        "timing": "hipGraph replay of eaas_expert_forward (per-kernel times from an eager pass "
                  "with events in the same run)",
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "data": "synthetic",
    }
    tiled = r.pop("_tiled", False)
    res.update({key: v for key, v in r.items() if key not in res})
    if args.clients > 0:
        res["segments"] = time_segments(d, dev, args.clients, args.steps, args.warmup, ms_eager,
                                        tiled)
    if args.server_slots > 0:
        res["server_step"] = time_server(d, dev, args.server_slots, args.steps, args.warmup,
                                         ms_eager, tiled)
    if args.scheduler_ablation:
        res["scheduler_ablation"] = scheduler_ablation(d, dev, args.steps, args.warmup, tiled)
    res["clocks_mhz"] = {"before": clocks_before, "after": clocks_after}
    if not args.no_decode and args.decode_workload != args.workload:
        del dev
        torch.cuda.empty_cache()
        # a decode step is 0.3-0.4 ms: 200 warm-up and 200 timed steps, so the
        # figure is taken with the engine clock settled (it starts from idle
        # and a few milliseconds of short steps do not bring it up)
        rd, _, _, _ = measure(args.decode_workload, max(args.steps, 200), max(args.warmup, 200),
                              tiled_fp8=not args.row_major_fp8)
        rd.pop("_tiled", None)
        res["decode"] = decode_summary(rd)
        res["decode"]["steps"] = max(args.steps, 200)
        res["decode"]["warmup"] = max(args.warmup, 200)
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(d)
    print(json.dumps(res), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
