#!/usr/bin/env python3
"""Benchmark of the quantized dequantize-and-multiply hot path on one MI355X.

Default workload (one "step"): one batch-1 decode step of a 32-layer 7B
decoder weight set -- per layer q, k, v, o (4096x4096, 3-bit per-group
codebook, group 128) and gate, up (11008x4096), down (4096x11008) (4-bit
uniform, group 128) -- i.e. 224 quantized GEMVs launched back to back in
layer order and replayed from a HIP graph. Inputs are synthetic and already
resident in HBM when the timed region starts.

Printed (one JSON line): effective HBM GB/s on packed-weight bytes over the
step (value), us per decode step, the roofline of the dominant kernel measured
live (HIP events around a graph of its launches, on the stream they run on),
and the CPU oracle timed on a bounded sample. Extra keys: gemv_configs (the
single 4-bit and 3-bit GEMVs c1, c2, c3 with the plain read of the same bytes)
and prefill_c5 (the MLP prefill GEMM at m = 16, 64, 512 against its roofline).

Other workloads (each prints its own line): --workload c1|c2|c3 (single GEMV
configs, rotated over enough copies to defeat the 256 MB last-level cache),
--workload batch (the same decode step for 1 to 4 sequences decoded together,
one line per batch size), --workload c5 (prefill GEMM, m = 16, 64, 512), --workload c5a8 (the same with int8
per-token activations), --workload q4xgemm (the same MLP prefill in the Q4X format, fp16 and int8
activations), --workload q4x (the paper's Q4X
format on the MLP shapes gate 11008x4096 and down 4096x11008, one line each,
rotated over copies like c1-c3), --workload a8 (c1, c2, c3, the 22016x4096 gate|up
matrix and the Q4X gate matrix with fp16 and with int8 activations, one line each), --workload tp8
(one GPU's share of the decode step at 8-way tensor parallelism, and c2 split 8 ways by
rows; the collectives are not run), --workload floor (plain read of
the same byte counts and empty grids: the floor of a one-launch GEMV) and
--workload counters (the run that the FETCH_SIZE / WRITE_SIZE passes profile).
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

HBM_PEAK_GBS = 8000.0            # MI355X HBM3E, published
FP16_MFMA_PEAK_TFLOPS = 2500.0   # dense fp16 matrix-core peak, published
INT8_MFMA_PEAK_TOPS = 5000.0    # dense int8 matrix-core peak, published
METRIC = "batch-1 qGEMV effective HBM GB/s (% of peak) + µs per 7B decode step"
KERNEL_SOURCES = ["qx_device.h", "gemv_common.h", "gemv.hip"]  # what the measured GEMV kernel is built from


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2505_07531_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def committed_traffic(kernel_key: str):
    """HBM bytes per launch from committed counter summaries, if taken on this kernel source."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        with open(path) as f:
            rec = json.load(f).get(kernel_key)
    except (OSError, ValueError):
        return None
    if not rec or rec.get("source_hash") != kernel_source_hash():
        return None
    return rec.get("bytes_per_launch")


# ----------------------------------------------------------------- workloads
def quantize_and_pack(spec, qx, device):
    q = spec.quantized()
    return qx.PackedWeight.from_quant(q, device=device)


def concat_rows(parts):
    """One quantized matrix whose rows are the rows of `parts` in order (same codes, same
    tables): the GEMV of the result is the GEMVs of the parts, row for row."""
    import qx_inputs as qi
    p0 = parts[0]
    cat = lambda a: None if getattr(p0, a) is None else np.concatenate([getattr(p, a) for p in parts])
    return qi.QuantWeight(sum(p.n for p in parts), p0.k, p0.bits, p0.group, p0.kind, cat("codes"),
                          cat("scales"), cat("zeros"), cat("codebook"))


class DecodeStep:
    """The 224 GEMVs of one decode step, resident on the GPU.

    fused=False launches the 224 GEMVs one by one (q, k, v, o, gate, up, down per
    layer). fused=True packs q|k|v and gate|up, which read the same activation
    vector, as single matrices with the same quantized rows, so a layer is four
    launches (qkv, o, gate|up, down) and the outputs are the same rows.
    """

    def __init__(self, qx, device, plan, quant, fused=False, batch=1):
        import torch
        from qx_inputs import configs
        self.plan = plan
        layers = len(plan) // 7
        self.launches = []  # (PackedWeight, activation key, [(row offset, plan index), ...])
        if fused:
            for l in range(layers):
                b = 7 * l
                groups = [[b, b + 1, b + 2], [b + 3], [b + 4, b + 5], [b + 6]]
                for g in groups:
                    q = concat_rows([quant[i] for i in g]) if len(g) > 1 else quant[g[0]]
                    offs, o = [], 0
                    for i in g:
                        offs.append((o, i))
                        o += quant[i].n
                    self.launches.append((qx.PackedWeight.from_quant(q, device=device),
                                          self.plan[g[0]][1], offs))
        else:
            for i, q in enumerate(quant):
                self.launches.append((qx.PackedWeight.from_quant(q, device=device),
                                      self.plan[i][1], [(0, i)]))
        self.batch = batch
        self.x = {}
        for l in range(layers):
            for t in range(4):
                xv = configs.c4_activation(l, t) if batch == 1 else configs.c4_batch_activations(l, t, batch)
                self.x[(l, t)] = torch.from_numpy(xv).to(device)
        self.y = [torch.empty((batch, pw.desc.n) if batch > 1 else pw.desc.n, dtype=torch.float16,
                              device=device) for pw, _, _ in self.launches]
        self.packed_bytes = sum(spec.packed_bytes for spec, _ in self.plan)
        self.act_bytes = sum(2 * (spec.n + spec.k) for spec, _ in self.plan)
        self.qx = qx

    def output(self, plan_index):
        """Device view of the y of GEMV `plan_index` of the plan ([batch][n] when batch > 1)."""
        for (pw, _, offs), y in zip(self.launches, self.y):
            for off, i in offs:
                if i == plan_index:
                    return y[..., off:off + self.plan[i][0].n]
        raise KeyError(plan_index)

    def launch(self, stream=None):
        qx = self.qx
        for (pw, xi, _), y in zip(self.launches, self.y):
            if self.batch == 1:
                qx.qx_gemv(pw.desc, pw.data, self.x[xi], y, stream)
            else:
                qx.qx_gemm(pw.desc, pw.data, self.batch, self.x[xi], y, stream)


def gated_kernel_durations(launches, reps=3):
    """Per-launch GPU durations (ms) from HIP event pairs around each launch.

    The stream is held behind a sleep kernel on a second stream while every
    launch and event is enqueued, so host enqueue speed cannot stretch the
    measured intervals.
    """
    import torch
    s = torch.cuda.current_stream()
    gate_stream = torch.cuda.Stream()
    out = []
    for _ in range(reps):
        gate = torch.cuda.Event()
        with torch.cuda.stream(gate_stream):
            torch.cuda._sleep(int(2e8))  # ~0.1 s of device cycles
            gate.record(gate_stream)
        s.wait_event(gate)
        evs = []
        for fn in launches:
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            a.record(s)
            fn()
            b.record(s)
            evs.append((a, b))
        torch.cuda.synchronize()
        out.extend(a.elapsed_time(b) for a, b in evs)
    return np.array(out)


def cpu_baseline_decode():
    """The oracle (unpack + fp16 dequant + fp64 matvec from the packed blob) on one matrix of
    each decoder shape -- q (4096x4096 codebook), gate (11008x4096 uniform), down (4096x11008
    uniform) of layer 0 -- scaled by how often each shape occurs in a step (128, 64, 32)."""
    import oracle
    import paper_2505_07531_amd as qx
    from qx_inputs import configs
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        threads = 1
    sample = [("q", 0, 128), ("gate", 2, 64), ("down", 3, 32)]
    items = []
    for name, t, count in sample:
        spec = configs.c4_matrix(0, name)
        q = spec.quantized()
        blob = qx.qx_pack_layout(qx.desc(q.n, q.k, q.bits, q.group, q.kind), q.codes, q.scales,
                                 q.zeros, q.codebook)
        items.append((spec, blob, configs.c4_activation(0, t), count))
    step_s, total, reps = 0.0, 0.0, 3
    for spec, blob, x, count in items:
        times = []
        for _ in range(reps):
            t0 = time.perf_counter()
            w16 = oracle.dequant_packed(blob, spec.n, spec.k, spec.bits, spec.group, spec.kind)
            oracle.gemv(w16, x)
            times.append(time.perf_counter() - t0)
        total += sum(times)
        step_s += float(np.median(times)) * count
    packed = sum(s.packed_bytes for s, _ in configs.c4_plan(32))
    return {"value": round(packed / step_s / 1e9, 4), "unit": "GB/s", "cores": int(threads),
            "kind": "oracle",
            "sample": f"3 GEMVs (layer-0 q, gate, down: unpack + fp16 dequant + fp64 matvec), each "
                      f"timed {reps} times ({total:.1f} s in all); the medians weighted x128/x64/x32 "
                      f"to a full step = "
                      f"{step_s * 1e3:.0f} ms per decode step; numpy elementwise work is "
                      f"single-threaded, BLAS uses the listed threads"}


def quantize_plan(plan):
    t0 = time.time()
    quant = []
    for i, (spec, _) in enumerate(plan):
        quant.append(spec.quantized())
        if (i + 1) % 28 == 0:
            log(f"quantized {i + 1}/{len(plan)} matrices ({time.time() - t0:.0f}s)")
    return quant


def time_graph(launch, stream, steps, warmup):
    """ms per replay of a HIP graph holding the launches made by `launch()`."""
    import torch
    with torch.cuda.stream(stream):
        launch()  # eager run first: fail loudly before capture
        stream.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            launch()
        for _ in range(warmup):
            g.replay()
        stream.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record(stream)
        for _ in range(steps):
            g.replay()
        e1.record(stream)
        torch.cuda.synchronize()
    return e0.elapsed_time(e1) / steps


def bench_decode(args, qx):
    import torch
    from qx_inputs import configs
    dev = torch.device("cuda:0")
    t0 = time.time()
    plan = configs.c4_plan(32)
    quant = quantize_plan(plan)
    fused = DecodeStep(qx, dev, plan, quant, fused=True)
    single = DecodeStep(qx, dev, plan, quant, fused=False)
    del quant
    log(f"workload ready in {time.time() - t0:.0f}s: {fused.packed_bytes / 1e9:.3f} GB packed "
        f"(each of two launch plans)")
    stream = torch.cuda.Stream()
    ms = time_graph(fused.launch, stream, args.steps, args.warmup)
    log(f"fused plan (128 launches): {ms * 1e3:.1f} us per decode step")
    ms_single = time_graph(single.launch, stream, max(5, args.steps // 2), 3)
    log(f"one launch per GEMV (224 launches): {ms_single * 1e3:.1f} us per decode step")

    # dominant kernel: the 4-bit uniform GEMV on the fused gate|up matrices (22016x4096)
    dom = [(pw, xi, y) for (pw, xi, offs), y in zip(fused.launches, fused.y) if pw.desc.n == 22016]
    def launch_dom():
        for pw, xi, y in dom:
            qx.qx_gemv(pw.desc, pw.data, fused.x[xi], y)
    dom_graph_ms = time_graph(launch_dom, stream, 20, 3) / len(dom)
    with torch.cuda.stream(stream):
        durs = gated_kernel_durations([lambda a=a: qx.qx_gemv(a[0].desc, a[0].data, fused.x[a[1]], a[2])
                                       for a in dom], reps=3)
    d0 = dom[0][0].desc
    alg_bytes = (d0.n * d0.k * d0.bits // 8 + d0.n * (d0.k // d0.group) * 4) + 2 * (d0.k + d0.n)
    avg_ms = dom_graph_ms
    achieved = alg_bytes / (avg_ms * 1e-3) / 1e9
    traffic = committed_traffic("gemv_u4_g128_22016x4096")
    value = fused.packed_bytes / (ms * 1e-3) / 1e9
    out = {
        "metric": METRIC, "value": round(value, 2), "unit": "GB/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 6),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f16",
        "data": "synthetic (seeded Philox weights: Laplace attention, Student-t MLP; N(0,1) activations)",
        "config": {"workload": "7B decoder decode step, batch 1: 32 layers x (q,k,v,o 4096x4096 "
                               "3-bit codebook g128; gate,up 11008x4096 and down 4096x11008 4-bit "
                               "uniform g128) = 224 GEMVs; q|k|v and gate|up packed as one matrix "
                               "each (same rows), 128 launches, HIP graph replay",
                   "packed_bytes_per_step": fused.packed_bytes,
                   "activation_bytes_per_step": fused.act_bytes},
        "us_per_step": round(ms * 1e3, 2),
        "pct_of_hbm_peak": round(100 * value / HBM_PEAK_GBS, 2),
        "us_per_step_one_launch_per_gemv": round(ms_single * 1e3, 2),
        "roofline": {"kernel": "gemv_wave_kernel<4, uniform, g128> on the 22016x4096 gate|up "
                               "matrix (32 launches per step)",
                     "bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "traffic": traffic, "bytes_per_launch": alg_bytes,
                     "avg_launch_us": round(avg_ms * 1e3, 3),
                     "avg_launch_us_event_pairs": round(float(np.mean(durs)) * 1e3, 3),
                     "launches_timed": 20 * len(dom)},
    }
    return out


def bench_decode_batch(args, qx):
    """The fused decode step for m = 2, 3, 4 sequences decoded together (one qx_gemm per
    launch); one line per m, and batch 1 (qx_gemv) for reference."""
    import torch
    from qx_inputs import configs
    dev = torch.device("cuda:0")
    plan = configs.c4_plan(32)
    quant = quantize_plan(plan)
    stream = torch.cuda.Stream()
    lines = []
    base_us = None
    for m in (1, 2, 3, 4):
        step = DecodeStep(qx, dev, plan, quant, fused=True, batch=m)
        ms = time_graph(step.launch, stream, args.steps, args.warmup)
        us = ms * 1e3
        base_us = us if m == 1 else base_us
        log(f"decode step, batch {m}: {us:.1f} us")
        lines.append({
            "metric": "decode step tokens/s at batch m (7B decoder, 224 products per step)",
            "value": round(m / (ms * 1e-3), 1), "unit": "tokens/s", "n_gpus": 1,
            "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 6),
            "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f16",
            "data": "synthetic (seeded Philox weights and activations)",
            "config": {"workload": f"7B decoder decode step, batch {m}: the decode7b matrices, "
                                   "q|k|v and gate|up fused, 128 launches of "
                                   + ("qx_gemv" if m == 1 else f"qx_gemm with m={m}")
                                   + ", HIP graph replay",
                       "batch": m, "packed_bytes_per_step": step.packed_bytes},
            "us_per_step": round(us, 2),
            "effective_weight_GBps": round(step.packed_bytes / (ms * 1e-3) / 1e9, 1),
            "step_time_vs_batch1": round(us / base_us, 3),
        })
        del step
        torch.cuda.empty_cache()
    return lines


def bench_tp8_share(args, qx):
    """One GPU's share of the decode step under 8-way tensor parallelism, at its real
    shapes: q|k|v and gate|up split by rows (512 rows of each of q, k, v, 1376 of gate and
    of up), o and down split along k (512, and 11008 / 8 padded to 11 chunks = 1408; these
    are synthetic matrices of the shard shape drawn like o and down), 128 launches per step
    replayed from a HIP graph; and the c2 matrix split 8 ways by rows (1376x4096). The
    all-reduces after o and down, and everything between GPUs, are not run."""
    import torch
    from qx_inputs import configs
    dev = torch.device("cuda:0")
    P, H, F = 8, configs.HIDDEN, configs.MLP
    kd = -(-F // P // 128) * 128
    launches, packed = [], 0
    for l in range(configs.LAYERS):
        qkv = concat_rows([configs.c4_matrix(l, m).quantized(0, H // P) for m in ("q", "k", "v")])
        gu = concat_rows([configs.c4_matrix(l, m).quantized(0, F // P) for m in ("gate", "up")])
        o = configs.MatrixSpec(f"L{l}.o/{P}", H, H // P, "laplace", configs.LAPLACE_B, 5, 2 * l, 3, 128,
                               configs.CODEBOOK).quantized()
        dn = configs.MatrixSpec(f"L{l}.down/{P}", H, kd, "t4", configs.T4_STD, 5, 2 * l + 1, 4, 128,
                                configs.UNIFORM).quantized()
        xs = [configs.c4_activation(l, 0), configs.c4_activation(l, 1)[:H // P], configs.c4_activation(l, 2),
              configs.c4_activation(l, 3)[:kd]]
        for q, x in zip((qkv, o, gu, dn), xs):
            pw = qx.PackedWeight.from_quant(q, device=dev)
            packed += pw.data.numel()
            launches.append((pw, torch.from_numpy(np.ascontiguousarray(x)).to(dev),
                             torch.empty(q.n, dtype=torch.float16, device=dev)))
    def launch():
        for pw, x, y in launches:
            qx.qx_gemv(pw.desc, pw.data, x, y)
    stream = torch.cuda.Stream()
    ms = time_graph(launch, stream, args.steps, args.warmup)
    log(f"tp8 share: {ms * 1e3:.1f} us per step, {packed} packed bytes")
    lines = [{"metric": "one GPU's share of the 7B decode step at 8-way tensor parallelism (us per step)",
              "value": round(ms * 1e3, 2), "unit": "us", "n_gpus": 1, "steps": args.steps,
              "warmup": args.warmup, "ms_per_step": round(ms, 6), "higher_is_better": False,
              "scaling": "strong", "vs_baseline": None, "dtype": "f16",
              "data": "synthetic (seeded Philox weights and activations)",
              "config": {"workload": "7B decoder decode step, batch 1, the share of one of 8 GPUs: per layer "
                                     "q|k|v 1536x4096 and o 4096x512 codebook-3 g128, gate|up 2752x4096 and "
                                     "down 4096x1408 uniform-4 g128 (128 launches, HIP graph replay); "
                                     "collectives not run", "packed_bytes_per_step": packed},
              "effective_weight_GBps": round(packed / (ms * 1e-3) / 1e9, 1)}]
    spec, x = configs.c2()
    q = spec.quantized(0, F // P)
    d = qx.desc(q.n, q.k, q.bits, q.group, q.kind)
    blob = qx.qx_pack_layout(d, q.codes, q.scales, q.zeros, q.codebook)
    base = torch.from_numpy(blob).to(dev)
    copies = [base] + [base.clone() for _ in range(max(2, -(-(512 << 20) // blob.size)) - 1)]
    xd = torch.from_numpy(x).to(dev)
    y = torch.empty(q.n, dtype=torch.float16, device=dev)
    def launch_c2():
        for c in copies:
            qx.qx_gemv(d, c, xd, y)
    ms2 = time_graph(launch_c2, stream, max(3, args.steps // len(copies)), 2) / len(copies)
    gbs = (blob.size + 2 * (q.n + q.k)) / (ms2 * 1e-3) / 1e9
    lines.append({"metric": "batch-1 qGEMV effective HBM GB/s (c2, one of 8 row shards)", "value": round(gbs, 2),
                  "unit": "GB/s", "n_gpus": 1, "steps": len(copies) * max(3, args.steps // len(copies)),
                  "warmup": 2 * len(copies), "ms_per_step": round(ms2, 6), "higher_is_better": True,
                  "scaling": "strong", "vs_baseline": None, "dtype": "f16", "data": "synthetic",
                  "config": {"workload": f"c2 rows 0-{q.n - 1}: {q.n}x{q.k} 3-bit uniform g64, graph of "
                                         f"back-to-back launches over {len(copies)} copies",
                             "packed_bytes": int(blob.size)},
                  "pct_of_hbm_peak": round(100 * gbs / HBM_PEAK_GBS, 2), "avg_launch_us": round(ms2 * 1e3, 3)})
    return lines


def rotated_copies(qx, spec, device, min_total=512 << 20):
    q = spec.quantized()
    d = qx.desc(q.n, q.k, q.bits, q.group, q.kind)
    if q.kind == qx.QX_Q4X:
        blob = qx.qx_pack_q4x(d, q.codes, q.scales, q.selectors, q.codebook)
    else:
        blob = qx.qx_pack_layout(d, q.codes, q.scales, q.zeros, q.codebook)
    import torch
    reps = max(2, -(-min_total // blob.size))
    base = torch.from_numpy(blob).to(device)
    copies = [base] + [base.clone() for _ in range(reps - 1)]
    return d, copies


def bench_single_gemv(args, qx, name, a8=False):
    import torch
    from qx_inputs import configs
    dev = torch.device("cuda:0")
    if name.startswith("q4x."):
        spec, x = configs.q4x_matrix(name[4:]), configs.q4x_activation(name[4:])
    elif name == "gateup":  # the fused gate|up matrix of the decode step, layer 0
        spec = configs.MatrixSpec("gate|up", 2 * configs.MLP, configs.HIDDEN, "t4", configs.T4_STD,
                                  3, 900, 4, 128, configs.UNIFORM)
        x = configs.c4_activation(0, 2)
    else:
        spec, x = getattr(configs, name)()
    gemv = qx.qx_gemv_a8 if a8 else qx.qx_gemv
    d, copies = rotated_copies(qx, spec, dev)
    xd = torch.from_numpy(x).to(dev)
    y = torch.empty(spec.n, dtype=torch.float16, device=dev)
    def launch_all():
        for c in copies:
            gemv(d, c, xd, y)
    reps = max(3, args.steps // len(copies))
    ms = time_graph(launch_all, torch.cuda.Stream(), reps, 2) / len(copies)
    alg = spec.packed_bytes + 2 * (spec.n + spec.k)
    gbs = alg / (ms * 1e-3) / 1e9
    traffic = committed_traffic(f"gemv_{name}")
    act = "int8 activations (per-token RTN, qx_gemv_a8)" if a8 else "fp16 activations"
    return {"metric": f"batch-1 qGEMV effective HBM GB/s ({name}{', A8' if a8 else ''})", "value": round(gbs, 2),
            "unit": "GB/s", "n_gpus": 1, "steps": reps * len(copies), "warmup": 2 * len(copies),
            "ms_per_step": round(ms, 6), "higher_is_better": True, "scaling": "weak",
            "vs_baseline": None, "dtype": "i8" if a8 else "f16", "data": "synthetic",
            "config": {"workload": f"{name}: {spec.n}x{spec.k} {spec.bits}-bit "
                                   f"{['uniform', 'codebook', 'Q4X (4 x 16 matrix codebook, scale + 2-bit selector per group)'][spec.kind]} "
                                   f"g{spec.group}, {act}, graph of back-to-back launches over {len(copies)} copies",
                       "copies": len(copies), "packed_bytes": spec.packed_bytes},
            "pct_of_hbm_peak": round(100 * gbs / HBM_PEAK_GBS, 2),
            "roofline": {"bound": "hbm", "achieved": round(gbs, 2), "peak": HBM_PEAK_GBS,
                         "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": traffic,
                         "avg_launch_us": round(ms * 1e3, 3)}}


def bench_gemm(args, qx, a8=False, q4x=False):
    """c5 prefill: gate, up, down at m = 16, 64, 512. a8: activations quantized per token
    (qx_quantize_a8, once per input, inside the timed region) and qx_gemm_a8. q4x: the same
    MLP shapes in the paper's Q4X format (Table 2 runs Q4X prefill with 8-bit activations)."""
    import torch
    from qx_inputs import configs
    dev = torch.device("cuda:0")
    if q4x:
        specs = {"gate": configs.q4x_matrix("gate"), "down": configs.q4x_matrix("down"),
                 "up": configs.MatrixSpec("q4x.up", configs.MLP, configs.HIDDEN, "t4", configs.T4_STD,
                                          5, 2, 4, 64, configs.Q4X)}
    else:
        specs = {nm: configs.c5_matrix(nm) for nm in ("gate", "up", "down")}
    mats = {nm: quantize_and_pack(specs[nm], qx, dev) for nm in ("gate", "up", "down")}
    # distinct copies of the three matrices, >= 512 MB in all, so that the codes of one
    # set are not still in the 256 MB last-level cache when they are read again
    set_bytes = sum(mats[nm].nbytes for nm in mats)
    nsets = max(2, -(-(512 << 20) // set_bytes))
    sets = [{nm: mats[nm].data for nm in mats}]
    sets += [{nm: mats[nm].data.clone() for nm in mats} for _ in range(nsets - 1)]
    lines = []
    for m in configs.C5_M:
        xin, xdn = configs.c5_activations(m)
        xi, xd = torch.from_numpy(xin).to(dev), torch.from_numpy(xdn).to(dev)
        ys = {nm: torch.empty((m, mats[nm].desc.n), dtype=torch.float16, device=dev) for nm in mats}
        qi_, si_ = torch.empty(xi.shape, dtype=torch.int8, device=dev), torch.empty(m, dtype=torch.float32, device=dev)
        qd_, sd_ = torch.empty(xd.shape, dtype=torch.int8, device=dev), torch.empty(m, dtype=torch.float32, device=dev)
        def launch_all():
            for st in sets:
                if a8:
                    qx.qx_quantize_a8(m, xi.shape[1], xi, qi_, si_)
                    qx.qx_quantize_a8(m, xd.shape[1], xd, qd_, sd_)
                    for nm in ("gate", "up", "down"):
                        dn = nm == "down"
                        qx.qx_gemm_a8(mats[nm].desc, st[nm], m, qd_ if dn else qi_, sd_ if dn else si_, ys[nm])
                    continue
                for nm in ("gate", "up", "down"):
                    qx.qx_gemm(mats[nm].desc, st[nm], m, xd if nm == "down" else xi, ys[nm])
        # ms for the three GEMMs
        t = time_graph(launch_all, torch.cuda.Stream(), 3, 1) / nsets
        flops = 2.0 * m * sum(mats[nm].desc.n * mats[nm].desc.k for nm in mats)
        byts = sum(specs[nm].packed_bytes for nm in mats) + m * 90_624
        tf = flops / (t * 1e-3) / 1e12
        gbs = byts / (t * 1e-3) / 1e9
        int8_cores = a8 and not q4x  # Q4X levels are fp16: its A8 products run on the fp16 matrix cores
        peak = INT8_MFMA_PEAK_TOPS if int8_cores else FP16_MFMA_PEAK_TFLOPS
        hbm_t, mfma_t = byts / (HBM_PEAK_GBS * 1e9), flops / (peak * 1e12)
        bound = "hbm" if hbm_t >= mfma_t else "mfma"
        frac = (hbm_t if bound == "hbm" else mfma_t) / (t * 1e-3)
        unit = "TOP/s" if int8_cores else "TFLOP/s"
        fmt_name = "Q4X (4 x 16 matrix codebook, scale + 2-bit selector per group of 64)" if q4x else "3-bit uniform g64"
        lines.append({"metric": f"prefill qGEMM{' Q4X' if q4x else ''}{' W·A8' if a8 else ''} (gate+up+down, m={m})",
                      "value": round(tf, 3), "unit": unit, "n_gpus": 1, "steps": 3 * nsets,
                      "warmup": nsets, "ms_per_step": round(t, 6), "higher_is_better": True,
                      "scaling": "weak", "vs_baseline": None, "dtype": "i8" if int8_cores else "f16",
                      "data": "synthetic",
                      "config": {"workload": f"{'Q4X ' if q4x else 'c5 '}MLP prefill GEMM m={m}, {fmt_name}, "
                                             + ("int8 per-token activations (quantized in the timed "
                                                "region), " if a8 else "")
                                             + f"graph over {nsets} copies of the three matrices"},
                      "roofline": {"bound": bound, "achieved": round(gbs if bound == "hbm" else tf, 2),
                                   "peak": HBM_PEAK_GBS if bound == "hbm" else peak,
                                   "unit": "GB/s" if bound == "hbm" else unit,
                                   "frac": round(frac, 4), "traffic": None}})
    return lines


def read_floor_us(nbytes: int, stream) -> float:
    """us per launch of a plain coalesced read of `nbytes` (16 B per thread), cold: rotated
    over copies >= 512 MB in a graph of back-to-back launches (the floor of a one-launch
    GEMV of that many bytes)."""
    import torch
    from paper_2505_07531_amd import probe
    dev = torch.device("cuda:0")
    nbytes = -(-nbytes // 16) * 16
    reps = max(2, -(-(512 << 20) // nbytes))
    bufs = [torch.ones(nbytes, dtype=torch.uint8, device=dev) for _ in range(reps)]
    sink = torch.zeros(4, dtype=torch.int32, device=dev)
    def launch_all():
        for b in bufs:
            probe.qxp_read(b, sink)
    us = time_graph(launch_all, stream, 5, 2) / reps * 1e3
    del bufs
    torch.cuda.empty_cache()
    return us


def gemv_config_summaries(args, qx):
    """c1, c2, c3 (batch-1 GEMV, rotated copies, graph-timed) next to the plain read of the
    same bytes: us, GB/s on packed bytes + x + y, % of 8 TB/s, % of the read's rate."""
    import torch
    out = {}
    stream = torch.cuda.Stream()
    for name in ("c1", "c2", "c3"):
        line = bench_single_gemv(args, qx, name)
        us = line["ms_per_step"] * 1e3
        alg = line["config"]["packed_bytes"]
        floor = read_floor_us(alg, stream)
        out[name] = {"workload": line["config"]["workload"], "us": round(us, 3), "GBps": line["value"],
                     "pct_of_hbm_peak": line["pct_of_hbm_peak"], "read_floor_us": round(floor, 3),
                     "pct_of_read_floor": round(100 * floor / us, 1), "bytes": alg}
        log(f"{name}: {us:.2f} us ({line['pct_of_hbm_peak']:.1f} % of 8 TB/s), read floor {floor:.2f} us")
    return out


def prefill_summary(args, qx):
    """c5 (prefill GEMM on the MLP shapes, gate + up + down) at m = 16, 64, 512."""
    out = {}
    for line in bench_gemm(args, qx):
        m = int(line["metric"].split("m=")[1].rstrip(")"))
        rf = line["roofline"]
        out[f"m{m}"] = {"us": round(line["ms_per_step"] * 1e3, 2), "TFLOPs": line["value"],
                        "bound": rf["bound"], "achieved": rf["achieved"], "unit": rf["unit"],
                        "frac_of_bound": rf["frac"]}
        log(f"c5 m={m}: {line['ms_per_step'] * 1e3:.1f} us, {rf['frac'] * 100:.1f} % of the {rf['bound']} roof")
    return out


def bench_kernel_counters(args, qx):
    """Workload for counter passes: the dominant kernel (4-bit uniform GEMV on the fused
    22016x4096 gate|up matrix of layer 0) launched 20 times, then a 256 MiB device-to-device
    copy launched 5 times as the known-size reference for FETCH_SIZE / WRITE_SIZE."""
    import torch
    from qx_inputs import configs
    dev = torch.device("cuda:0")
    q = concat_rows([configs.c4_matrix(0, "gate").quantized(), configs.c4_matrix(0, "up").quantized()])
    pw = qx.PackedWeight.from_quant(q, device=dev)
    x = torch.from_numpy(configs.c4_activation(0, 2)).to(dev)
    y = torch.empty(pw.desc.n, dtype=torch.float16, device=dev)
    for _ in range(20):
        qx.qx_gemv(pw.desc, pw.data, x, y)
    a = torch.ones(256 << 20, dtype=torch.uint8, device=dev)
    b = torch.empty_like(a)
    for _ in range(5):
        b.copy_(a)
    torch.cuda.synchronize()
    return {"workload": "counters", "gemv_launches": 20, "gemv_packed_bytes": pw.nbytes,
            "gemv_x_y_bytes": 2 * (pw.desc.k + pw.desc.n), "copy_launches": 5,
            "copy_bytes_each_way": int(a.numel())}


def bench_floor(args, qx):
    """The floor of a one-launch GEMV: a plain coalesced read of the same number of
    bytes (16 B per thread, cold: rotated over copies >= 512 MB, graph-timed), and an
    empty grid of the decode kernels' block counts."""
    import torch
    from paper_2505_07531_amd import probe
    from qx_inputs import configs
    dev = torch.device("cuda:0")
    sink = torch.zeros(4, dtype=torch.int32, device=dev)
    sizes = {"q|k|v": 3 * configs.c4_matrix(0, "q").packed_bytes,
             "o": configs.c4_matrix(0, "o").packed_bytes,
             "gate|up": 2 * configs.c4_matrix(0, "gate").packed_bytes,
             "down": configs.c4_matrix(0, "down").packed_bytes}
    for name in ("c1", "c2", "c3"):
        sizes[name] = getattr(configs, name)()[0].packed_bytes
    stream = torch.cuda.Stream()
    reads = []
    for name, nbytes in sizes.items():
        reps = max(2, -(-(512 << 20) // nbytes))
        bufs = [torch.ones(nbytes, dtype=torch.uint8, device=dev) for _ in range(reps)]
        def launch_all():
            for b in bufs:
                probe.qxp_read(b, sink)
        us = time_graph(launch_all, stream, 5, 2) / reps * 1e3
        reads.append({"matrix": name, "bytes": nbytes, "us": round(us, 3),
                      "gbs": round(nbytes / (us * 1e-6) / 1e9, 1)})
        log(f"read {name}: {nbytes} B in {us:.3f} us")
        del bufs
    empty = {}
    for blocks in (1, 512, 1536, 2752):
        def launch_empty():
            for _ in range(100):
                probe.qxp_empty(blocks, sink)
        empty[str(blocks)] = round(time_graph(launch_empty, stream, 5, 2) / 100 * 1e3, 3)
    return {"workload": "floor", "read": reads, "empty_grid_us_by_blocks": empty,
            "note": "per launch, graph of back-to-back launches; 256 threads per block"}


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="decode7b",
                    choices=["decode7b", "batch", "c1", "c2", "c3", "c5", "c5a8", "q4x", "q4xgemm", "a8",
                             "tp8", "counters", "floor"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-configs", action="store_true",
                    help="decode7b only: skip the c1-c3 GEMV and c5 prefill keys")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only: the library has no multi-GPU path "
              f"(asked for --gpus {args.gpus}).", file=sys.stderr)
        sys.exit(2)
    import torch
    import paper_2505_07531_amd as qx
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    qx.load()
    log(f"device: {torch.cuda.get_device_name(0)}")
    if args.workload == "decode7b":
        out = bench_decode(args, qx)
        if not args.no_configs:
            out["gemv_configs"] = gemv_config_summaries(args, qx)
            out["prefill_c5"] = prefill_summary(args, qx)
        if not args.no_cpu_baseline:
            t0 = time.time()
            out["cpu_baseline"] = cpu_baseline_decode()
            log(f"cpu baseline in {time.time() - t0:.0f}s")
        else:
            out["cpu_baseline"] = None
        props = torch.cuda.get_device_properties(0)
        out["device"] = {"name": props.name, "arch": getattr(props, "gcnArchName", ""),
                         "compute_units": props.multi_processor_count,
                         "memory_gb": round(props.total_memory / 1e9, 1)}
        print(json.dumps(out), flush=True)
    elif args.workload == "counters":
        print(json.dumps(bench_kernel_counters(args, qx)), flush=True)
    elif args.workload == "floor":
        print(json.dumps(bench_floor(args, qx)), flush=True)
    elif args.workload == "tp8":
        for line in bench_tp8_share(args, qx):
            print(json.dumps(line), flush=True)
    elif args.workload == "batch":
        for line in bench_decode_batch(args, qx):
            print(json.dumps(line), flush=True)
    elif args.workload == "q4xgemm":
        for a8 in (False, True):
            for line in bench_gemm(args, qx, a8=a8, q4x=True):
                print(json.dumps(line), flush=True)
    elif args.workload == "c5a8":
        for line in bench_gemm(args, qx, a8=True):
            print(json.dumps(line), flush=True)
    elif args.workload == "c5":
        for line in bench_gemm(args, qx):
            print(json.dumps(line), flush=True)
    elif args.workload == "a8":
        for name in ("c1", "c2", "c3", "gateup", "q4x.gate"):
            for a8 in (False, True):
                print(json.dumps(bench_single_gemv(args, qx, name, a8)), flush=True)
    elif args.workload == "q4x":
        for name in ("q4x.gate", "q4x.down"):
            print(json.dumps(bench_single_gemv(args, qx, name)), flush=True)
    else:
        print(json.dumps(bench_single_gemv(args, qx, args.workload)), flush=True)


if __name__ == "__main__":
    main()
