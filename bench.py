#!/usr/bin/env python3
"""Benchmark of the HCMS single-GPU hot path on one MI355X.

A step is one pass of the whole hot path over one batch of synthetic input:
pack Q/K/V of every head chunk, attention of every chunk, unpack of every
chunk, scheduled across streams by ``hcms_forward`` (auto mode: the one-GPU
schedule the round rule picks).  The workload is the Wan2.2-14B-shaped rank share at P = 8: S = 56160
tokens (36 latent frames x 1560), H = 5 local heads, d = 128, bf16, chunks
2 + 2 + 1 (the paper's uneven rule for C = 3).

Printed: one JSON line with the metric (attention TFLOP/s, 4 S^2 H d per step
over the step time), the roofline of the dominant kernel (attention, bf16
MFMA), the layout kernels' HBM rates, the serial, Alg. 1, inline, lanes,
fused and two-slot schedules side by side, and the oracle timed on the host cores on a bounded
sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import statistics
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import paper_2607_01817_amd as hcms  # noqa: E402
from paper_2607_01817_amd import inputs  # noqa: E402

MFMA_BF16_PEAK_TFLOPS = 2516.6  # MI355X dense bf16: 256 CU x 2.4 GHz x 4096 FLOP/clk
HBM_PEAK_GBS = 8000.0           # MI355X HBM3E
ATTENTION_SRCS = [os.path.join(ROOT, "paper_2607_01817_amd", "csrc", f)
                  for f in ("attention.hip", "copy_tiles.h")]
TRAFFIC_RECORD = os.path.join(ROOT, "profiles", "attention_traffic_wan_p8.json")


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse_chunks(s: str) -> tuple[int, ...]:
    return tuple(int(x) for x in s.replace("+", ",").split(",") if x)


def flush_mall(buf: torch.Tensor):
    """Read a buffer larger than the 256 MB infinity cache, leaving it full of
    clean lines.  (Overwriting the buffer instead leaves dirty lines whose
    write-back lands inside the next measurement.)"""
    buf.amax()


class GpuSensors:
    """The GPU's clock, power and hotspot temperature through amdsmi's metrics
    table (read only; reported beside the timings, never used in them).
    Every reading is None when amdsmi is missing or the device cannot be
    matched by its PCI address."""

    def __init__(self, dev_index: int = 0):
        self.handle = None
        try:
            import amdsmi
            amdsmi.amdsmi_init()
            p = torch.cuda.get_device_properties(dev_index)
            want = (p.pci_domain_id, p.pci_bus_id, p.pci_device_id)
            for h in amdsmi.amdsmi_get_processor_handles():
                dom, bus, rest = amdsmi.amdsmi_get_gpu_device_bdf(h).split(":")
                if (int(dom, 16), int(bus, 16), int(rest.split(".")[0], 16)) == want:
                    self.handle = h
                    break
            self.amdsmi = amdsmi
        except Exception:                      # no amdsmi, no permission: nothing reported
            self.handle = None

    def sample(self):
        if self.handle is None:
            return None
        try:
            m = self.amdsmi.amdsmi_get_gpu_metrics_info(self.handle)
            clks = [c for c in m.get("current_gfxclks", []) if isinstance(c, int) and 0 < c < 10000]
            if not clks and isinstance(m.get("current_gfxclk"), int):
                clks = [m["current_gfxclk"]]
            pw, tc = m.get("current_socket_power"), m.get("temperature_hotspot")
            return {"gfx_mhz": round(sum(clks) / len(clks), 1) if clks else None,
                    "power_w": pw if isinstance(pw, int) else None,
                    "hotspot_c": tc if isinstance(tc, int) else None}
        except Exception:
            return None


class EventTimer:
    """Events around calls enqueued back to back on one stream, read after a
    single synchronisation at the end.  The host stays ahead of the GPU, so a
    call's span is its GPU work: a synchronisation after every call would leave
    the GPU idle while the host issues the next one (Python and the ctypes
    call, tens of microseconds) and count that idle time too."""

    def __init__(self, stream=None):
        self.stream = stream or torch.cuda.current_stream()
        self.marks = []

    def time(self, key, fn):
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record(self.stream)
        fn()
        b.record(self.stream)
        self.marks.append((key, a, b))

    def results(self) -> dict:
        self.stream.synchronize()
        torch.cuda.synchronize()
        out = {}
        for key, a, b in self.marks:
            out.setdefault(key, []).append(a.elapsed_time(b))
        self.marks = []
        return out


def time_region(fn, reps: int, stream=None) -> list[float]:
    """Per-rep milliseconds of fn() repeated back to back (EventTimer)."""
    t = EventTimer(stream)
    for _ in range(reps):
        t.time(0, fn)
    return t.results().get(0, [])


def measured_traffic(workload: str, chunks, plan: str) -> float | None:
    """HBM bytes per attention launch of `plan` from the committed rocprofv3
    counter record (FETCH_SIZE + WRITE_SIZE, scaled by a plain copy of known
    size), or None when there is no record for this workload and plan or the
    kernel sources have changed since the counters were taken."""
    import hashlib
    try:
        with open(TRAFFIC_RECORD) as f:
            rec = json.load(f)
        h = hashlib.sha256()
        for src in ATTENTION_SRCS:
            with open(src, "rb") as f:
                h.update(f.read())
    except (OSError, ValueError):
        return None
    if rec.get("source_sha256") != h.hexdigest() or rec.get("workload") != workload \
            or list(rec.get("chunks", [])) != list(chunks) or plan not in rec.get("plans", {}):
        return None
    return float(rec["plans"][plan]["hbm_bytes_per_launch"])


def copy_calibration(dev):
    """A plain device-to-device copy of 1 GiB (read 1 GiB, write 1 GiB), run
    three times, so counter passes over this process can scale FETCH_SIZE and
    WRITE_SIZE by a kernel of known traffic."""
    src = torch.ones(2**29, dtype=torch.bfloat16, device=dev)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst


def cpu_baseline(w, q, k, v, seconds: float):
    """Time the oracle on sampled query rows of the same workload."""
    import oracle
    per_head = min(w.S, 16384)
    rows_all = inputs.sample_rows(w, per_head, seed=w.seed + 77)
    heads = [(x[:, h, :].to(torch.float64).numpy() for x in (q, k, v)) for h in range(w.H)]
    heads = [tuple(t) for t in heads]
    done_rows = 0
    t_cpu = 0.0
    batch = 128
    h = 0
    pos = [0] * w.H
    while t_cpu < seconds and done_rows < w.H * per_head:
        qh, kh, vh = heads[h]
        rows = rows_all[h][pos[h]:pos[h] + batch]
        pos[h] += batch
        t0 = time.perf_counter()
        oracle.attention_head(qh, kh, vh, w.scale, rows)
        t_cpu += time.perf_counter() - t0
        done_rows += rows.size
        h = (h + 1) % w.H
    flops = 4.0 * done_rows * w.S * w.d
    return {
        "value": flops / t_cpu / 1e12,
        "unit": "TFLOP/s",
        "cores": oracle.num_threads(),
        "kind": "oracle",
        "sample": f"{done_rows} query rows (128-row batches over the {w.H} heads) of the "
                  f"same workload against all S={w.S} keys, fp64, {t_cpu:.1f} s; "
                  f"full-problem time extrapolates to {w.flops / (flops / t_cpu):.0f} s",
    }


MODES = {"serial": hcms.MODE_SERIAL, "pipelined": hcms.MODE_PIPELINED, "inline": hcms.MODE_INLINE,
         "lanes": hcms.MODE_LANES, "auto": hcms.MODE_AUTO, "slots": hcms.MODE_SLOTS,
         "fused": hcms.MODE_FUSED}
MODE_NAMES = {v: k for k, v in MODES.items()}


def quartiles(xs):
    q = np.percentile(xs, [25, 50, 75])
    return {"median": round(float(q[1]), 4), "iqr": [round(float(q[0]), 4), round(float(q[2]), 4)]}


def compare_modes(ctx, w, chunks, reps: int, dev, modes=None):
    """The schedules of one workload and chunking side by side: serial, Alg. 1,
    inline, lanes, fused, the slots plan on two chunk slots and auto (the plan
    MODE_AUTO picks), interleaved (order reversed every other rep to cancel
    clock drift), step time from events on the main stream."""
    q, k, v = (x.to(dev) for x in inputs.make_qkv(w))
    out = torch.empty_like(q)
    ws = ctx.workspaces(w.S, w.H, w.d, q.dtype)
    slots = ctx.slot_workspaces(w.S, max(chunks), w.d, q.dtype)
    modes = modes or ["serial", "pipelined", "inline", "lanes", "fused", "slots_two_slot", "auto"]

    def run(m):
        if m == "slots_two_slot":   # the slots plan on two chunk slots
            return lambda: ctx.forward_slots(q, k, v, w.P, w.scale, chunks, mode=hcms.MODE_SLOTS,
                                             out=out, slots=slots)
        return lambda: ctx.forward(q, k, v, w.P, w.scale, chunks, mode=MODES[m], out=out,
                                   workspaces=ws)

    for m in modes:                 # one warm run of each
        run(m)()
    timer = EventTimer()
    for r in range(reps + 1):
        for m in (modes if r % 2 == 0 else modes[::-1]):
            timer.time((m, r), run(m))
    spans = timer.results()
    times = {m: [t for r in range(1, reps + 1) for t in spans[(m, r)]] for m in modes}
    ctx.forward(q, k, v, w.P, w.scale, chunks, mode=hcms.MODE_AUTO, out=out, workspaces=ws)
    res = {"workload": w.name, "chunks": list(chunks), "auto_runs": MODE_NAMES[ctx.last_mode]}
    ser = quartiles(times["serial"])
    res["serial_ms"] = ser
    for m in modes[1:]:
        qm = quartiles(times[m])
        qm["gain_vs_serial_ms"] = round(ser["median"] - qm["median"], 4)
        qm["below_serial"] = bool(qm["iqr"][1] < ser["iqr"][0])
        res[m + "_ms"] = qm
    if "auto" in modes:
        # auto running the serial plan issues the serial plan's launches:
        # equal by construction, whatever the noise between the two medians.
        res["auto_not_above_serial"] = bool(res["auto_runs"] == "serial" or
                                            res["auto_ms"]["median"] <= ser["median"])
    es = q.element_size()
    res["workspace_bytes"] = {"full": 4 * w.S * w.H * w.d * es,
                              "two_slot": 4 * 2 * max(chunks) * w.S * w.d * es}
    del q, k, v, out, slots
    return res


def time_model_sweep(ctx, w, reps: int, dev):
    """The paper's chunk-count study on one GPU: for C = 1..H (the default
    partition), the serial, Alg. 1 and auto schedules interleaved, and the
    layout and attention kernel times of the serial plan (medians over `reps`
    warmed runs with events around every kernel); the paper's
    T(C) = a + T_comm / C + beta C fitted to the scheduled times."""
    q, k, v = (x.to(dev) for x in inputs.make_qkv(w))
    out = torch.empty_like(q)
    ws = ctx.workspaces(w.S, w.H, w.d, q.dtype)
    counts = list(range(1, w.H + 1))
    modes = ["serial", "pipelined", "auto"]
    med = {m: [] for m in modes}
    t_comm, t_attn = [], []
    for C in counts:
        sizes = hcms.default_chunks(w.H, C)

        def run(m):
            ctx.forward(q, k, v, w.P, w.scale, sizes, mode=MODES[m], out=out, workspaces=ws)

        for m in modes:
            run(m)
        timer = EventTimer()
        for r in range(reps + 1):
            for m in (modes if r % 2 == 0 else modes[::-1]):
                timer.time((m, r), lambda: run(m))
        spans = timer.results()
        times = {m: [t for r in range(1, reps + 1) for t in spans[(m, r)]] for m in modes}
        for m in modes:
            med[m].append(float(np.median(times[m])))
        ctx.set_timing(reps)
        for _ in range(reps):
            run("serial")
        torch.cuda.synchronize()
        per_call = lambda kind: np.asarray(ctx.kernel_ms(kind)).reshape(reps, C).sum(axis=1)  # noqa: E731
        t_comm.append(float(np.median(per_call(hcms.OP_PACK) + per_call(hcms.OP_UNPACK))))
        t_attn.append(float(np.median(per_call(hcms.OP_ATTENTION))))
        ctx.set_timing(0)
    res = {"workload": w.name, "S": w.S, "H": w.H, "chunk_counts": counts,
           "serial_ms": [round(x, 4) for x in med["serial"]],
           "pipelined_ms": [round(x, 4) for x in med["pipelined"]],
           "auto_ms": [round(x, 4) for x in med["auto"]],
           "layout_kernels_ms": [round(x, 4) for x in t_comm],
           "attention_kernels_ms": [round(x, 4) for x in t_attn],
           "note": "kernel columns: medians over the warmed serial runs, events around every kernel"}
    for m in ("pipelined", "auto"):
        a, tc, beta = hcms.model_fit(counts, med[m])
        pred = [a + tc / c + beta * c for c in counts]
        err = max(abs(p_ - t) / t for p_, t in zip(pred, med[m]))
        best_model, c_star = (hcms.model_optimal_chunks(tc, beta, w.H)
                              if tc >= 0 and beta >= 0 else (None, None))
        res["fit_" + m] = {
            "a_ms": round(a, 4), "t_comm_ms": round(tc, 4), "beta_ms": round(beta, 4),
            "c_star": None if c_star is None or not math.isfinite(c_star) else round(c_star, 3),
            "best_c_model": best_model,
            "best_c_measured": counts[int(np.argmin(med[m]))],
            "max_rel_error": round(err, 5)}
    del q, k, v, out
    return res


def adaptive_chunks(ctx, sweeps):
    """Calibrate the one-GPU time model (hcms_model_plan_time) on the sweeps'
    measurements and let hcms_choose_chunks pick the chunk count:
      * t_round = kappa S (a full round of attention workgroups; a
        workgroup's work is 4 Br S d) and g0 by least squares on the serial
        plans' attention kernel times over every sweep:
        T_attn = kappa S X1 + kappa g0 S X2, where X1 + g0 X2 is the
        launches' round count with partial (and split) rounds costing
        g0 + (1 - g0) f of theirs (X1, X2 read off the library's model at
        g0 = 1 and g0 -> 0);
      * t_copy = the layout kernels at C = 1 over 4 H head-tensors;
      * beta = (Alg. 1 - serial) at C = 1 over its 7 synchronisations;
      * per workload, the drain (rounds per attention launch on the
        critical path) and a constant T_0 by least squares on its auto
        plans' step-time residuals (drain >= 0).
    Reports the model's prediction of the auto plan per C against the
    measured auto time and whether the chosen C measures within 1 % of the
    sweep's best."""
    n = ctx.num_cu
    tiny = 1e-9
    rows, ys = [], []
    for sw in sweeps:
        for C, t in zip(sw["chunk_counts"], sw["attention_kernels_ms"]):
            sz = hcms.default_chunks(sw["H"], C)
            x_lo = hcms.model_plan_time(sw["S"], 128, sz, hcms.MODE_SERIAL, n, 1.0, tiny, 0.0, 0.0)
            x_hi = hcms.model_plan_time(sw["S"], 128, sz, hcms.MODE_SERIAL, n, 1.0, 1.0, 0.0, 0.0)
            x2 = (x_hi - x_lo) / (1.0 - tiny)
            rows.append([sw["S"] * (x_lo - tiny * x2), sw["S"] * x2])
            ys.append(t)
    (kappa, kg0), *_ = np.linalg.lstsq(np.asarray(rows), np.asarray(ys), rcond=None)
    g0 = float(min(1.0, max(1e-3, kg0 / kappa))) if kappa > 0 else 1.0
    par = {}
    for sw in sweeps:
        S, H = sw["S"], sw["H"]
        par[sw["workload"]] = (kappa * S, sw["layout_kernels_ms"][0] / (4 * H),
                               max(0.0, (sw["pipelined_ms"][0] - sw["serial_ms"][0]) / 7))
    # Per workload, the drain and T_0 from its step times: residual = T_0 +
    # drain x (the plan's launches on the critical path x t_round).
    t0, drains = {}, {}
    for sw in sweeps:
        t_round, t_copy, beta = par[sw["workload"]]
        rows, ys = [], []
        for C in sw["chunk_counts"]:
            sz = hcms.default_chunks(sw["H"], C)
            p0 = hcms.model_plan_time(sw["S"], 128, sz, hcms.MODE_AUTO, n, t_round, g0, t_copy, beta)
            p1 = hcms.model_plan_time(sw["S"], 128, sz, hcms.MODE_AUTO, n, t_round, g0, t_copy, beta,
                                      drain=1.0)
            rows.append([1.0, p1 - p0])
            ys.append(sw["auto_ms"][C - 1] - p0)
        (a0, a1), *_ = np.linalg.lstsq(np.asarray(rows), np.asarray(ys), rcond=None)
        if a1 < 0.0:   # no drain: T_0 alone
            a1, a0 = 0.0, float(np.mean(ys))
        t0[sw["workload"]], drains[sw["workload"]] = float(a0), float(a1)
    out = {"kappa_ms_per_key": float(kappa), "g0": round(g0, 4), "configs": []}
    for sw in sweeps:
        S, H = sw["S"], sw["H"]
        t_round, t_copy, beta = par[sw["workload"]]
        drain = drains[sw["workload"]]
        pred = [t0[sw["workload"]] +
                hcms.model_plan_time(S, 128, hcms.default_chunks(H, C), hcms.MODE_AUTO, n, t_round,
                                     g0, t_copy, beta, drain=drain) for C in sw["chunk_counts"]]
        sizes, plan, t_pred = hcms.choose_chunks(S, H, 128, n, t_round, g0, t_copy, beta,
                                                 drain=drain)
        meas = sw["auto_ms"]
        best = min(meas)
        chosen = meas[len(sizes) - 1]
        out["configs"].append({
            "workload": sw["workload"], "t_round_ms": round(t_round, 4),
            "t_copy_ms": round(t_copy, 5), "beta_ms": round(beta, 5),
            "t0_ms": round(t0[sw["workload"]], 4), "drain_rounds": round(drain, 4),
            "predicted_auto_ms": [round(x, 4) for x in pred],
            "measured_auto_ms": meas,
            "prediction_error": [round((p_ - m_) / m_, 4) for p_, m_ in zip(pred, meas)],
            "chosen_chunks": sizes, "chosen_plan": MODE_NAMES[plan],
            "chosen_measured_ms": chosen, "best_measured_ms": best,
            "best_measured_c": sw["chunk_counts"][int(np.argmin(meas))],
            "chosen_within_1pct_of_best": bool(chosen <= 1.01 * best)})
    return out


def peak_memory(ctx, w, chunks, dev):
    """The caching allocator's peak above the resident inputs for one forward
    on full head-major workspaces and one on two chunk slots (workspaces and
    output allocated inside the measured region).  The inputs are drawn on
    the device (the byte counts do not depend on their values)."""
    g = torch.Generator(device=dev).manual_seed(w.seed)
    q, k, v = ((torch.randn((w.S, w.H, w.d), generator=g, device=dev) * w.sigma).to(torch.bfloat16)
               for _ in range(3))
    torch.cuda.synchronize()
    res = {"workload": w.name, "chunks": list(chunks)}
    for name in ("full_workspaces", "two_slots"):
        torch.cuda.empty_cache()
        base = torch.cuda.memory_allocated(dev)
        torch.cuda.reset_peak_memory_stats(dev)
        out = torch.empty_like(q)
        if name == "full_workspaces":
            ws = [torch.empty((w.H, w.S, w.d), dtype=q.dtype, device=dev) for _ in range(4)]
            ctx.forward(q, k, v, w.P, w.scale, chunks, out=out, workspaces=ws)
        else:
            ws = [torch.empty((2, max(chunks), w.S, w.d), dtype=q.dtype, device=dev)
                  for _ in range(4)]
            ctx.forward_slots(q, k, v, w.P, w.scale, chunks, out=out, slots=ws)
        torch.cuda.synchronize()
        res[name + "_MB"] = round((torch.cuda.max_memory_allocated(dev) - base) / 1e6, 1)
        del out, ws
    inputs_mb = 3 * q.numel() * q.element_size() / 1e6
    res["inputs_MB"] = round(inputs_mb, 1)
    tot_f, tot_s = inputs_mb + res["full_workspaces_MB"], inputs_mb + res["two_slots_MB"]
    res["peak_with_inputs_change"] = round(tot_s / tot_f - 1.0, 4)
    res["note"] = ("peak = torch.cuda.max_memory_allocated above the resident Q, K, V; the paper "
                   "reports -8.7 % peak memory for the whole model on 4 GPUs at 131K tokens "
                   "(appendix memory table), context only")
    del q, k, v
    torch.cuda.empty_cache()
    return res


def training_step(ctx, w, chunks, reps: int, dev):
    """Forward (keeping the softmax statistic) and backward of the hot path,
    per step: the auto schedule against serial, interleaved; the backward's
    roofline (algorithmic 10 S^2 H d FLOP: the five products Q K^T, dO V^T,
    P^T dO, dS K, dS^T Q) over the whole backward pass of the auto schedule,
    and over each chunk's launches in the serial one."""
    q, k, v = (x.to(dev) for x in inputs.make_qkv(w))
    dout = inputs.make_dout(w).to(dev)
    fws = [torch.empty((w.H, w.S, w.d), dtype=q.dtype, device=dev) for _ in range(4)]
    lse = torch.empty((w.H, w.S), dtype=torch.float32, device=dev)
    out = torch.empty_like(q)
    grads = [torch.empty_like(q) for _ in range(3)]

    def fwd(mode):
        ctx.forward(q, k, v, w.P, w.scale, chunks, mode=mode, out=out, workspaces=fws, lse=lse)

    def bwd(mode):
        ctx.backward(dout, w.P, w.scale, chunks, fws, lse, mode=mode, dq=grads[0], dk=grads[1],
                     dv=grads[2])

    # The score-gradient workspace: two regions (main and compute stream) of
    # the largest chunk's heads.
    per_head = hcms.backward_ds_bytes(w.S, w.d, q.dtype)
    ds = (torch.empty(2 * max(chunks) * per_head, dtype=torch.uint8, device=dev)
          if per_head else None)
    ctx.set_ds_workspace(ds)
    for _ in range(3):
        fwd(hcms.MODE_AUTO)
        auto_fwd = MODE_NAMES[ctx.last_mode]
        bwd(hcms.MODE_AUTO)
        auto_bwd = MODE_NAMES[ctx.last_mode]
    timer = EventTimer()
    for r in range(reps + 1):
        for m in (("serial", "auto") if r % 2 == 0 else ("auto", "serial")):
            timer.time((m, "fwd", r), lambda: fwd(MODES[m]))
            timer.time((m, "bwd", r), lambda: bwd(MODES[m]))
    spans = timer.results()
    times = {m: {p: [t for r in range(1, reps + 1) for t in spans[(m, p, r)]] for p in ("fwd", "bwd")}
             for m in ("serial", "auto")}
    def launches():
        ctx.set_timing(reps)
        for _ in range(reps):
            bwd(hcms.MODE_SERIAL)
        torch.cuda.synchronize()
        ms = ctx.kernel_ms(hcms.OP_ATTENTION)
        ctx.set_timing(0)
        C = len(chunks)
        alg = [10.0 * w.S * w.S * chunks[i % C] * w.d for i in range(len(ms))]
        return ms, sum(alg) / (sum(ms) * 1e-3) / 1e12

    attn_ms, achieved = launches()
    # The same launches without the workspace (the query-parallel dQ kernel).
    ctx.set_ds_workspace(None)
    bwd(hcms.MODE_SERIAL)
    plain_ms, plain = launches()
    del ds
    res = {"workload": w.name, "chunks": list(chunks)}
    for m in times:
        f = quartiles(times[m]["fwd"])
        b = quartiles(times[m]["bwd"])
        res[m] = {"forward_ms": f, "backward_ms": b,
                  "step_ms": round(f["median"] + b["median"], 4),
                  "step_TFLOPs": round(14.0 * w.S * w.S * w.H * w.d /
                                       ((f["median"] + b["median"]) * 1e-3) / 1e12, 2)}
    res["auto_runs"] = {"forward": auto_fwd, "backward": auto_bwd}
    flop = 10.0 * w.S * w.S * w.H * w.d
    whole = flop / (res["auto"]["backward_ms"]["median"] * 1e-3) / 1e12
    res["backward_roofline"] = {
        "bound": "mfma", "achieved": round(whole, 2), "peak": MFMA_BF16_PEAK_TFLOPS,
        "unit": "TFLOP/s", "frac": round(whole / MFMA_BF16_PEAK_TFLOPS, 4),
        "kernels": "attention_delta_kernel + attention_dkdv_dma_kernel<true> (dK, dV, and dS "
                   "stored as bf16) + attention_dq_ds_kernel (dQ = scale dS K from the stored dS); "
                   "d = 128, bf16, score-gradient workspace of 2 regions x "
                   f"{max(chunks)} heads x {per_head / 2**30:.2f} GiB",
        "per_pass": f"10*S^2*H*d FLOP over the median backward pass of the auto schedule "
                    f"({auto_bwd}: the pack of dO, every chunk's launches and the unpack of dQ, "
                    f"dK, dV, with one chunk's dQ product beside the next chunk's dK/dV launch), "
                    f"{res['auto']['backward_ms']['median']:.4f} ms",
        "per_chunk_serial": {
            "achieved": round(achieved, 2), "frac": round(achieved / MFMA_BF16_PEAK_TFLOPS, 4),
            "avg_ms": round(statistics.mean(attn_ms), 4),
            "note": f"10*S^2*H_c*d FLOP per chunk over its launches alone (no copies), avg over "
                    f"{len(attn_ms)} chunk backward passes of the serial schedule"},
        "without_workspace": {
            "achieved": round(plain, 2), "frac": round(plain / MFMA_BF16_PEAK_TFLOPS, 4),
            "avg_ms": round(statistics.mean(plain_ms), 4),
            "kernels": "attention_dq_dma_kernel (D, dQ; recomputes Q K^T and dO V^T) + "
                       "attention_dkdv_dma_kernel<false>: 14*S^2*H_c*d FLOP executed"}}
    res["note"] = "step_TFLOPs counts 4 S^2 H d (forward) + 10 S^2 H d (backward)"
    del q, k, v, dout, fws, lse, out, grads
    return res


def layer_step(ctx, lw, chunks, reps: int, dev):
    """One attention layer around the chunk loop on the Wan2.2-shaped rank
    share: the QKV projection (split and rotary embedding fused), the chunked
    forward in the auto schedule, the output projection, each timed on its
    own, and the whole hcms_layer_forward.  The projection GEMM's roofline is
    the bf16 MFMA peak; torch.matmul (hipBLASLt) on the same shapes is shown
    beside it as a reference only."""
    x, w_qkv, w_o = (t.to(dev) for t in inputs.make_layer(lw))
    table = hcms.rope_table(lw.grid, lw.axis_pairs, lw.base)
    S, H, d, D = lw.S, lw.H, lw.d, lw.D
    qkv = tuple(torch.empty((S, H, d), dtype=x.dtype, device=dev) for _ in range(3))
    o = torch.empty((S, H, d), dtype=x.dtype, device=dev)
    y = torch.empty((S, D), dtype=x.dtype, device=dev)
    ws = ctx.workspaces(S, H, d, x.dtype)
    steps = {
        "qkv_projection": lambda: hcms.qkv_projection(x, w_qkv, H, d, table, lw.grid,
                                                      lw.axis_pairs, out=qkv),
        "attention_chunks": lambda: ctx.forward(qkv[0], qkv[1], qkv[2], lw.P, lw.scale, chunks,
                                                out=o, workspaces=ws),
        "output_projection": lambda: hcms.linear(o.view(S, H * d), w_o, out=y),
        "layer": lambda: ctx.layer_forward(x, w_qkv, w_o, lw.P, H, d, lw.scale, chunks, table,
                                           lw.grid, lw.axis_pairs, out=y),
    }
    for fn in steps.values():
        for _ in range(5):
            fn()
    torch.cuda.synchronize()
    res = {"workload": f"{lw.name}: S={S} ({'x'.join(map(str, lw.grid))} latent grid), H={H}, "
                       f"d={d}, D={D}, bf16, chunks {'+'.join(map(str, chunks))}",
           "chunks": list(chunks)}
    fl = lw.flops
    flops = {"qkv_projection": fl["qkv_projection"], "attention_chunks": fl["attention"],
             "output_projection": fl["output_projection"], "layer": sum(fl.values())}
    for name, fn in steps.items():
        q3 = quartiles(time_region(fn, reps))
        res[name] = {"ms": q3, "TFLOPs": round(flops[name] / (q3["median"] * 1e-3) / 1e12, 1)}
    ref = {}
    xr = o.view(S, H * d)
    for name, a, b_ in (("qkv_projection", x, w_qkv), ("output_projection", xr, w_o)):
        out = torch.empty((a.shape[0], b_.shape[0]), dtype=a.dtype, device=dev)
        for _ in range(5):
            torch.matmul(a, b_.t(), out=out)
        ref[name] = round(statistics.median(
            time_region(lambda: torch.matmul(a, b_.t(), out=out), reps)), 4)
        del out
    qp = res["qkv_projection"]
    res["gemm_roofline"] = {
        "bound": "mfma", "achieved": qp["TFLOPs"], "peak": MFMA_BF16_PEAK_TFLOPS,
        "unit": "TFLOP/s", "frac": round(qp["TFLOPs"] / MFMA_BF16_PEAK_TFLOPS, 4),
        "kernel": "linear_kernel<bf16, qkv epilogue>",
        "per_launch": f"2*S*D*3*H*d = {fl['qkv_projection']:.3e} FLOP per launch; median "
                      f"{qp['ms']['median']} ms over {reps} launches"}
    res["reference_torch_matmul_ms"] = ref
    res["note"] = ("TFLOPs of each step count its algorithmic FLOPs (2 per multiply-add; attention "
                   "4 S^2 H d); reference_torch_matmul_ms is hipBLASLt on the plain GEMMs of the "
                   "same shapes, not part of the path")
    del x, w_qkv, w_o, qkv, o, y, table
    return res


def one_chunk_roofline(ctx, w, qd, kd, vd, out, ws, steps: int, warmup: int):
    """The attention roofline of the workload in one chunk of all heads (the
    serial plan: pack, one attention launch, unpack): the timed steps' step
    time minus the step's copy kernels (timed in a second pass with events
    around every kernel), over the launch's FLOPs."""
    sizes = (w.H,)

    def step():
        ctx.forward(qd, kd, vd, w.P, w.scale, sizes, mode=hcms.MODE_SERIAL, out=out, workspaces=ws)

    for _ in range(warmup):
        step()
    main_stream = torch.cuda.current_stream()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record(main_stream)
    for _ in range(steps):
        step()
    t1.record(main_stream)
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / steps
    ctx.set_timing(steps)
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    attn = ctx.kernel_ms(hcms.OP_ATTENTION)
    copies = (sum(ctx.kernel_ms(hcms.OP_PACK)) + sum(ctx.kernel_ms(hcms.OP_UNPACK))) / steps
    ctx.set_timing(0)
    achieved = w.flops / ((ms - copies) * 1e-3) / 1e12
    ev = w.flops / (statistics.mean(attn) * 1e-3) / 1e12
    return {"chunks": list(sizes), "plan": "serial", "ms_per_step": round(ms, 4),
            "achieved": round(achieved, 2), "frac": round(achieved / MFMA_BF16_PEAK_TFLOPS, 4),
            "events_pass_frac": round(ev / MFMA_BF16_PEAK_TFLOPS, 4),
            "avg_launch_ms_events": round(statistics.mean(attn), 4),
            "note": f"{steps} timed steps after {warmup} warm-up steps; achieved = 4 S^2 H d over "
                    f"the step minus its pack and unpack kernels ({copies:.4f} ms)"}


def trace_summary(trace_csv: str, line_path: str) -> str:
    """Markdown summary of a rocprofv3 kernel trace (``--kernel-trace
    --output-format csv``) of one bench.py run, checked against the JSON line
    that same run printed.  The attention dispatches are taken in issue order:
    the first warmup * C are the warm-up steps, the next steps * C the timed
    steps, the next steps * C the pass with events around every kernel (the
    line's roofline), then the plain-launch pass under the fused plan."""
    import csv
    line = None
    with open(line_path) as f:
        for ln in f:
            ln = ln.strip()
            if ln.startswith("{") and '"metric"' in ln:
                line = json.loads(ln)
    if line is None:
        raise SystemExit(f"no bench line in {line_path}")
    cfg = line["config"]
    chunks, S, d = cfg["chunks"], cfg["S"], cfg["d"]
    C, W, K = len(chunks), line["warmup"], line["steps"]
    rows = []
    with open(trace_csv) as f:
        for r in csv.DictReader(f):
            if "attention_dma_kernel" in r["Kernel_Name"] or "attention_kernel" in r["Kernel_Name"]:
                rows.append((int(r["Start_Timestamp"]), int(r["End_Timestamp"]), r["Kernel_Name"]))
    rows.sort()
    flops = [4.0 * S * S * chunks[i % C] * d for i in range(K * C)]

    def pass_stats(first):
        sel = rows[first:first + K * C]
        if len(sel) < K * C:
            return None
        dur = [(e - b) * 1e-6 for b, e, _ in sel]          # ns -> ms
        ach = sum(flops) / (sum(dur) * 1e-3) / 1e12
        per_step = [sum(dur[i * C:(i + 1) * C]) for i in range(K)]
        return {"avg_launch_ms": statistics.mean(dur), "kernel_ms_per_step": statistics.mean(per_step),
                "achieved": ach, "frac": ach / MFMA_BF16_PEAK_TFLOPS, "names": {n for *_, n in sel}}

    timed, events = pass_stats(W * C), pass_stats((W + K) * C)
    rf = line["roofline"]
    out = [f"Bench line: value {line['value']} TFLOP/s, ms_per_step {line['ms_per_step']}, "
           f"roofline achieved {rf['achieved']} TFLOP/s, frac {rf['frac']} "
           f"({cfg['workload']}; warmup {W}, steps {K}).", "",
           f"Attention dispatches in the trace: {len(rows)}.", "",
           "| Pass | Dispatches | Avg launch (ms) | Kernel time per step (ms) | TFLOP/s | frac |",
           "|---|---|---|---|---|---|"]
    for name, st, first in (("timed steps", timed, W * C), ("steps with events (the line's events_pass)",
                                                            events, (W + K) * C)):
        if st:
            out.append(f"| {name} | {first}..{first + K * C - 1} | {st['avg_launch_ms']:.4f} | "
                       f"{st['kernel_ms_per_step']:.4f} | {st['achieved']:.1f} | {st['frac']:.4f} |")
    ev = rf.get("events_pass", {})
    if timed:
        out += ["",
                f"- Attention kernel time per timed step {timed['kernel_ms_per_step']:.4f} ms <= "
                f"the line's ms_per_step {line['ms_per_step']}: "
                f"{timed['kernel_ms_per_step'] <= line['ms_per_step']}.",
                f"- frac from the trace's timed steps {timed['frac']:.4f} against the line's "
                f"{rf['frac']}: {abs(timed['frac'] / rf['frac'] - 1) * 100:.2f} % apart."]
    if events and ev:
        out.append(f"- frac from the trace's events pass {events['frac']:.4f} against the line's "
                   f"events_pass {ev['frac']}: {abs(events['frac'] / ev['frac'] - 1) * 100:.2f} % "
                   f"apart (the events add a few microseconds to each launch they bracket).")
    if timed:
        out.append(f"- Kernels: {', '.join(sorted(timed['names']))}.")
    return "\n".join(out)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=40)
    ap.add_argument("--warmup", type=int, default=150,
                    help="untimed steps; about a second of them lets the clock settle")
    ap.add_argument("--workload", default="wan_p8", choices=sorted(inputs.WORKLOADS))
    ap.add_argument("--chunks", default="2,2,1")
    ap.add_argument("--mode", default="auto", choices=sorted(MODES))
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle baseline")
    ap.add_argument("--no-extras", action="store_true",
                    help="time the step only (for profiler runs)")
    ap.add_argument("--only", choices=("training", "layer"),
                    help="run only that section on the workload and chunks (for profiler runs)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run a plain 1 GiB device copy first (for counter passes)")
    ap.add_argument("--trace-summary", metavar="KERNEL_TRACE_CSV",
                    help="summarise a rocprofv3 kernel trace of a bench run (no GPU needed)")
    ap.add_argument("--bench-line", metavar="FILE",
                    help="with --trace-summary: the output of the traced run (its JSON line)")
    args = ap.parse_args()

    if args.trace_summary:
        print(trace_summary(args.trace_summary, args.bench_line))
        return

    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the hot path "
              "is one GPU's share of HCMS and this library has no multi-GPU exchange.",
              file=sys.stderr)
        sys.exit(2)
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)

    w = inputs.WORKLOADS[args.workload]
    sizes = parse_chunks(args.chunks)
    assert sum(sizes) == w.H, f"chunks {sizes} do not sum to H={w.H}"
    mode = MODES[args.mode]
    hcms.load()
    dev = torch.device("cuda:0")
    if args.copy_calibration:
        copy_calibration(dev)
    if args.only:
        ctx = hcms.Context(max_chunks=max(16, len(sizes)))
        if args.only == "training":
            res = training_step(ctx, w, sizes, max(10, args.steps // 4), dev)
        else:
            lw = inputs.LAYERS["layer_wan_p8"]
            res = layer_step(ctx, lw, lw.chunkings[-1], max(10, args.steps // 2), dev)
        ctx.close()
        print(json.dumps({"only": args.only, args.only: res}), flush=True)
        return
    log(f"workload {w.name}: S={w.S} H={w.H} d={w.d} {w.dtype} P={w.P} chunks={sizes} "
        f"mode={args.mode}")
    q, k, v = inputs.make_qkv(w)
    qd, kd, vd = (x.to(dev) for x in (q, k, v))
    ctx = hcms.Context(max_chunks=max(16, len(sizes)))
    out = torch.empty_like(qd)
    ws = ctx.workspaces(w.S, w.H, w.d, qd.dtype)

    def step(m=mode, chunks=sizes):
        ctx.forward(qd, kd, vd, w.P, w.scale, chunks, mode=m, out=out, workspaces=ws)

    torch.cuda.synchronize()
    sensors = GpuSensors(0)
    clock = {"idle_before_warmup": sensors.sample()}
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    plan = MODE_NAMES[ctx.last_mode]

    # ---- timed region: K steps, nothing but the steps between the events ----
    main_stream = torch.cuda.current_stream()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record(main_stream)
    for _ in range(args.steps):
        step()
    t1.record(main_stream)
    torch.cuda.synchronize()
    clock["after_timed_steps"] = sensors.sample()
    clock["source"] = ("amdsmi metrics table (current_gfxclks averaged over the XCDs, "
                       "current_socket_power, temperature_hotspot), read with the GPU idle before "
                       "the warm-up and right after the timed steps; the table refreshes about "
                       "once a second, so the second reading reflects the warm-up and timed steps "
                       "when they last a second or more (the default run) and may predate them in "
                       "a shorter run")
    ms_per_step = t0.elapsed_time(t1) / args.steps

    # ---- the same K steps again with every kernel bracketed by events on
    # the stream that runs it: per-launch durations for the roofline ----
    ctx.set_timing(args.steps)
    t0.record(main_stream)
    for _ in range(args.steps):
        step()
    t1.record(main_stream)
    torch.cuda.synchronize()
    ms_per_step_events = t0.elapsed_time(t1) / args.steps
    attn_ms = ctx.kernel_ms(hcms.OP_ATTENTION)
    pack_ms = ctx.kernel_ms(hcms.OP_PACK)
    unpack_ms = ctx.kernel_ms(hcms.OP_UNPACK)
    ctx.set_timing(0)

    # ---- under a plan whose launches also carry copies, the same steps once
    # more in the serial plan: the attention launch on its own ----
    plain_ms = None
    if plan == "fused":
        ctx.set_timing(args.steps)
        for _ in range(args.steps):
            step(m=hcms.MODE_SERIAL)
        torch.cuda.synchronize()
        plain_ms = ctx.kernel_ms(hcms.OP_ATTENTION)
        ctx.set_timing(0)

    tflops = w.flops / (ms_per_step * 1e-3) / 1e12
    C = len(sizes)
    launch_flops = [4.0 * w.S * w.S * sizes[i % C] * w.d for i in range(len(attn_ms))]
    avg_attn_ms = statistics.mean(attn_ms)
    achieved_events = sum(launch_flops) / (sum(attn_ms) * 1e-3) / 1e12
    # Copies that ran as kernels of their own (in the fused plan chunk 0's
    # pack and the last unpack; the others rode in the attention launches).
    own_pk = [i for i in range(len(pack_ms)) if plan != "fused" or i % C == 0]
    own_up = [i for i in range(len(unpack_ms)) if plan != "fused" or i % C == C - 1]
    if plan in ("fused", "serial"):
        # One stream, kernels back to back: the timed steps' attention time
        # is the step minus its own copy kernels (their durations from the
        # events pass).  The events around every kernel in that pass
        # lengthen each launch by a few microseconds, so this figure, from
        # the timed region itself, is the roofline's.
        copies_per_step = (sum(pack_ms[i] for i in own_pk) +
                           sum(unpack_ms[i] for i in own_up)) / args.steps
        attn_per_step = ms_per_step - copies_per_step
        achieved = w.flops / (attn_per_step * 1e-3) / 1e12
        how = (f"timed steps: {ms_per_step:.4f} ms per step minus its own copy kernels "
               f"{copies_per_step:.4f} ms (pack of chunk 0 and unpack of the last chunk"
               f"{'' if plan == 'fused' else ', and every other copy'}, from the events pass) = "
               f"{attn_per_step:.4f} ms of attention launches per step, "
               f"{attn_per_step / C:.4f} ms per launch on average")
    else:
        achieved = achieved_events
        how = "the events pass (several streams: the step does not decompose)"
    result = {
        "metric": "attention TFLOP/s (4·S²·H·d) + pipelined vs serial chunk time, 1 MI355X",
        "value": round(tflops, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic: seeded N(0,1)*0.5 Q/K/V, Wan2.2-shaped (no real activations)",
        "config": {
            "workload": f"{w.name}: S={w.S} (36 frames x 1560 tokens), H={w.H} local heads, "
                        f"d={w.d}, {w.dtype}, P={w.P} shards, chunks {'+'.join(map(str, sizes))}, "
                        f"pack+attention+unpack, {plan} schedule",
            "S": w.S, "H": w.H, "d": w.d, "P": w.P, "chunks": list(sizes),
            "mode": args.mode, "plan": plan,
        },
        "roofline": {
            "bound": "mfma",
            "achieved": round(achieved, 2),
            "peak": MFMA_BF16_PEAK_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(achieved / MFMA_BF16_PEAK_TFLOPS, 4),
            "traffic": measured_traffic(w.name, sizes, plan),
            "kernel": "attention_dma_kernel (d = 128, bf16)" + (
                "; in the fused plan each launch also carries the neighbouring chunks' copies "
                "on the CUs its last round leaves idle (attention_dma_kernel<true>)"
                if plan == "fused" else ""),
            "per_launch": f"4*S^2*H_c*d FLOP per chunk launch; achieved from {how}",
            "events_pass": {
                "achieved": round(achieved_events, 2),
                "frac": round(achieved_events / MFMA_BF16_PEAK_TFLOPS, 4),
                "avg_launch_ms": round(avg_attn_ms, 4),
                "note": f"events around every kernel on its stream, a second pass of the "
                        f"{args.steps} steps ({ms_per_step_events:.4f} ms per step with the "
                        f"events), {len(attn_ms)} launches"},
        },
        "gpu_clock": clock,
    }
    if tuple(sizes) != (w.H,):
        result["roofline"]["one_chunk"] = one_chunk_roofline(ctx, w, qd, kd, vd, out, ws,
                                                             args.steps, max(args.warmup, 20))
    if plain_ms:
        plain = sum(launch_flops) / (sum(plain_ms) * 1e-3) / 1e12
        result["roofline"]["plain_launch"] = {
            "achieved": round(plain, 2),
            "frac": round(plain / MFMA_BF16_PEAK_TFLOPS, 4),
            "avg_launch_ms": round(statistics.mean(plain_ms), 4),
            "note": "the same launches without riding copies (serial plan, a third pass of the "
                    "steps): the attention kernel's own roofline; the copies riding in the fused "
                    "launches take part of the power the attention would otherwise clock on",
        }

    if not args.no_extras:
        es = w.elem_bytes
        pk_bytes = [3 * 2 * w.S * sizes[i % C] * w.d * es for i in range(len(pack_ms))]
        up_bytes = [2 * w.S * sizes[i % C] * w.d * es for i in range(len(unpack_ms))]
        # In the fused plan a copy that rides in an attention launch reports
        # that launch's time; the rates then cover the copies that ran alone
        # (chunk 0's pack, the last chunk's unpack: own_pk, own_up above).
        pipe = {"pack_in_step_GBps": round(sum(pk_bytes[i] for i in own_pk) /
                                           (sum(pack_ms[i] for i in own_pk) * 1e-3) / 1e9, 1),
                "unpack_in_step_GBps": round(sum(up_bytes[i] for i in own_up) /
                                             (sum(unpack_ms[i] for i in own_up) * 1e-3) / 1e9, 1)}
        if plan == "fused":
            pipe["in_step_note"] = ("fused plan: rates of the copies that ran as launches of "
                                    "their own (chunk 0's pack, the last unpack); the others "
                                    "rode in the attention launches")

        # ---- layout kernels alone on the Wan-P4, Wan-P8 and Stress shapes:
        # cold (MALL flushed) and warm.  A byte move does not depend on the
        # values, so the buffers are left uninitialised. ----
        scratch = torch.zeros(768 * 2**20 // 4, dtype=torch.float32, device=dev)
        reps = 20
        res = {}
        for lw in (inputs.WORKLOADS[n] for n in ("wan_p4", "wan_p8", "stress")):
            src = torch.empty((lw.S, lw.H, lw.d), dtype=inputs.torch_dtype(lw), device=dev)
            hm = torch.empty((lw.H, lw.S, lw.d), dtype=src.dtype, device=dev)
            nbytes = 2 * src.numel() * src.element_size()
            entry = {"bytes": nbytes}
            for name, fn in (("pack", lambda: hcms.pack(src, lw.P, 0, lw.H, out=hm)),
                             ("unpack", lambda: hcms.unpack(hm, src, lw.P, 0))):
                cold, warm = [], []
                for _ in range(reps):
                    flush_mall(scratch)
                    cold += time_region(fn, 1)
                warm = time_region(fn, reps)
                mc, mw = statistics.median(cold), statistics.median(warm)
                entry[name] = {
                    "GBps_cold": round(nbytes / (mc * 1e-3) / 1e9, 1),
                    "frac_of_hbm_cold": round(nbytes / (mc * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                    "GBps_warm": round(nbytes / (mw * 1e-3) / 1e9, 1),
                    "frac_of_hbm_warm": round(nbytes / (mw * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                    "median_ms_cold": round(mc, 5)}
            res[lw.name] = entry
            del src, hm
        del scratch
        res["note"] = ("one tensor, all heads; bytes = read + write of [S][H][d]; cold = the 256 MB "
                       "MALL holds other (clean) data, warm = back-to-back reps")
        res.update(pipe)
        result["layout"] = res

        # ---- the schedules side by side: serial, Alg. 1, inline, lanes, fused ----
        torch.cuda.synchronize()
        reps = max(20, args.steps // 2)
        cmp = [compare_modes(ctx, w, sizes, reps, dev), compare_modes(ctx, w, (w.H,), reps, dev),
               compare_modes(ctx, w, (1,) * w.H, reps, dev)]
        wp4 = inputs.WORKLOADS["wan_p4"]
        for ch in ((5, 5), (4, 3, 3), (10,)):
            cmp.append(compare_modes(ctx, wp4, ch, reps, dev))
        small = inputs.WORKLOADS["small"]
        for ch in ((3, 3, 2), (2, 2, 2, 2)):
            cmp.append(compare_modes(ctx, small, ch, max(reps, 40), dev))
        result["schedules"] = cmp

        # ---- allocator peak: full workspaces against two chunk slots ----
        result["memory"] = [peak_memory(ctx, w, (1,) * w.H, dev),
                            peak_memory(ctx, inputs.WORKLOADS["stress"], (10, 10, 10, 10), dev)]

        # ---- training: forward with the softmax statistic, then backward ----
        result["training"] = training_step(ctx, w, sizes, max(10, args.steps // 4), dev)

        # ---- the attention layer around the chunk loop (Wan-P8 share) ----
        lw = inputs.LAYERS["layer_wan_p8"]
        result["layer"] = layer_step(ctx, lw, lw.chunkings[-1], max(10, args.steps // 2), dev)

        # ---- the time model over the chunk count (Wan-P8, Wan-P4) ----
        sweeps = [time_model_sweep(ctx, tw, reps, dev) for tw in dict.fromkeys((w, wp4))]
        result["time_model"] = sweeps
        result["adaptive_chunks"] = adaptive_chunks(ctx, sweeps)

    if not args.no_cpu:
        log("timing the oracle on the host ...")
        result["cpu_baseline"] = cpu_baseline(w, q, k, v, args.cpu_seconds)

    ctx.close()
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
