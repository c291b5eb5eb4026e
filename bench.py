"""Benchmark of the INT8 encoder-decoder hot path on one MI355X.

One step = one whole translation of the batch-1 latency workload: a seeded
synthetic 12-encoder / 2-decoder model (d_model 256, 4 heads, FFN 1024,
shared vocabulary 32000, int8 weights with per-channel scales), one source of
30 tokens, encoder + exactly 30 greedy decode steps (embedding, int8 linear
layers, int8 self/cross attention with the int8 key/value cache, fused
logits + arg-max), replayed from a captured hipGraph, inputs already in HBM.

Prints one JSON line: decoded tokens per second (value), ms per sentence,
the roofline of the dominant kernel (the decoder's fused logits + arg-max
kernel over the 8.19 MB int8 embedding, HBM bound, launched alone through
mnmt_qlinear on one int8 row), the int8 GEMM throughput of the largest
quantized-linear sweep shape against the i8 matrix-core peak, and the CPU
oracle timed on the host as a baseline.

--counters runs only the roofline kernel (50 launches) and a 256 MiB device
copy, for rocprofv3 --pmc passes; --ingest-counters FETCH.csv WRITE.csv turns
the two passes' counter_collection files into profiles/counters.json (HBM
bytes per launch, scaled by what the same counters read for the copy).
"""
from __future__ import annotations

import argparse
import ctypes as C
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E
I8_PEAK_TOPS = 5000.0  # MI355X dense int8 matrix-core peak


def _events_ms(torch, fn, reps, stream):
    """Average ms per call of fn() over reps back-to-back calls on `stream`."""
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        fn()
    e1.record(stream)
    e1.synchronize()
    return e0.elapsed_time(e1) / reps


ROOF_TAG = "step_logits_raw_b1"
ROOF_KERNEL = "k_step_logits<256, true, 2, true>"
COPY_BYTES = 256 << 20


def _warm(torch, fn, seconds=0.05):
    """Untimed calls for about ``seconds`` of wall time (at least 3): the GPU's
    clocks settle under sustained load (a 60 us GEMM measured right after an
    idle phase runs up to 20% slower)."""
    t0 = time.perf_counter()
    n = 0
    while n < 3 or time.perf_counter() - t0 < seconds:
        fn()
        n += 1
        if n % 16 == 0:
            torch.cuda.synchronize()
    torch.cuda.synchronize()


def _graph_launch_ms(torch, fn, launches=200, replays=5):
    """Mean time per launch (ms) of fn() captured `launches` times back to back
    in one graph and replayed `replays` times between two events on the
    replaying stream: each launch's duration plus its gap to the next, as the
    kernel runs inside the decoder's captured step graph."""
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for _ in range(launches):
            fn()
    s = torch.cuda.current_stream()
    for _ in range(3):
        g.replay()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(s)
    for _ in range(replays):
        g.replay()
    e1.record(s)
    e1.synchronize()
    return e0.elapsed_time(e1) / (launches * replays)


def _source_hash():
    h = hashlib.sha256()
    for f in ("decode_step.hip", "canon.hpp", "blocks.hpp", "chain.hpp", "internal.h"):
        with open(os.path.join(ROOT, "paper_2306_04235_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def _traffic(kernel_tag):
    """HBM bytes per launch from committed rocprofv3 counter runs, if they were
    taken on the current kernel source (else None)."""
    path = os.path.join(ROOT, "profiles", "counters.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        data = json.load(f)
    rec = data.get(kernel_tag)
    if not rec or rec.get("source_hash") != _source_hash():
        return None
    return rec.get("hbm_bytes_per_launch")


def _roofline_kernel(torch, np, mnmt, WL, G, info, blob, dev, stream):
    """The roofline kernel as a closure, and its algorithmic bytes per launch:
    the int8 embedding [V, d] (in the fragment order the decoder reads it in,
    the same V·d bytes), the fp32 output scales [V], one int8 row, and the
    8-byte arg-max partial of every block (the store pattern of the batch-1
    decode step)."""
    from synth.modelfile import read_model

    dims = WL.Dims(info.d_model, info.n_heads, info.d_ffn, info.n_enc, info.n_dec, info.vocab)
    alg_bytes = WL.logits_gemv_bytes(dims) + info.d_model + 8 * mnmt.argmax_partials(info.vocab)
    _, tens = read_model(blob)
    x = torch.randint(-127, 128, (1, info.d_model), dtype=torch.int8, device=dev)
    E = mnmt.mnmt_pack_weights(torch.from_numpy(np.array(tens["emb.w"])).to(dev), stream=stream)
    c_out = torch.from_numpy(np.array(tens["emb.s"])).to(dev)  # the values do not affect the timing
    slot = torch.zeros((1, mnmt.argmax_partials(info.vocab)), dtype=torch.int64, device=dev)
    V, epi = info.vocab, mnmt.EPI_ARGMAX_PARTIAL_PACKED

    def fn():
        mnmt.mnmt_qlinear(x, E, c_out, None, epi, out=slot, stream=stream, n_out=V)

    return fn, alg_bytes


def _trace_avg_us(kernel_tag):
    """Average kernel-trace duration (us) of the roofline kernel from the
    committed rocprofv3 summary, if it was taken on the current kernel source."""
    path = os.path.join(ROOT, "profiles", "counters.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f).get(kernel_tag + "_trace")
    if not rec or rec.get("source_hash") != _source_hash():
        return None
    return rec.get("avg_us")


def counters_run():
    """Short run for rocprofv3 --pmc: the roofline kernel 50 times, then a
    256 MiB device-to-device copy (the counters' calibration) 3 times."""
    import numpy as np
    import torch

    from paper_2306_04235_amd import mnmt, workload as WL
    from synth import generate as G

    dev = torch.device("cuda:0")
    blob = G.build_model(G.WORKLOADS["mobile"].model)
    model = mnmt.Model(blob)
    stream = torch.cuda.current_stream()
    fn, _ = _roofline_kernel(torch, np, mnmt, WL, G, model.info, blob, dev, stream)
    for _ in range(50):
        fn()
    src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    model.close()
    print("counters run done", flush=True)


GEMM_TAG = "qgemm_4096x256x32000"
GEMM_COUNTERS = ("SQ_INSTS_VALU_MFMA_MOPS_I8", "SQ_VALU_MFMA_BUSY_CYCLES", "GRBM_GUI_ACTIVE", "SQ_BUSY_CYCLES")


def _gemm_source_hash():
    h = hashlib.sha256()
    for f in ("gemm.hip", "qlinear.hip", "blocks.hpp", "canon.hpp", "internal.h"):
        with open(os.path.join(ROOT, "paper_2306_04235_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def _gemm_case(torch, dev):
    """The largest sweep shape (4096 x 256 x 32000, int8 requantizing
    epilogue) as a closure over random operands, and M, K, N."""
    from paper_2306_04235_amd import mnmt

    M, K, N = 4096, 256, 32000
    Xg = torch.randint(-127, 128, (M, K), dtype=torch.int8, device=dev)
    Wg = torch.randint(-127, 128, (N, K), dtype=torch.int8, device=dev)
    sc = torch.full((N,), 1e-4, dtype=torch.float32, device=dev)
    bi = torch.zeros(N, dtype=torch.float32, device=dev)
    Yg = torch.empty((M, N), dtype=torch.int8, device=dev)
    stream = torch.cuda.current_stream()
    return (lambda: mnmt.mnmt_qlinear(Xg, Wg, sc, bi, mnmt.EPI_I8, out=Yg, stream=stream)), (M, K, N)


def beam_counters_run():
    """Short run for one rocprofv3 --pmc pass over the base beam workload:
    one eager translation (every kernel a dispatch of its own)."""
    import torch

    from paper_2306_04235_amd import mnmt
    from synth import generate as G

    dev = torch.device("cuda:0")
    w = G.WORKLOADS["base_beam"]
    m = mnmt.Model(G.build_model(w.model))
    src, lens = G.workload_inputs(w)
    sess = mnmt.Session(m, w.batch, w.s_max, w.steps, w.beam)
    sess.translate(torch.from_numpy(src).to(dev), torch.from_numpy(lens).to(dev), beam=w.beam, max_steps=w.steps,
                   alpha=w.alpha, use_graph=False)
    torch.cuda.synchronize()
    sess.status()
    print("beam counters run done", flush=True)


def gemm_counters_run():
    """Short run for one rocprofv3 --pmc pass over the GEMM: 5 launches, then
    20 more (the counters are taken per dispatch)."""
    import torch

    g, _ = _gemm_case(torch, torch.device("cuda:0"))
    for _ in range(25):
        g()
    torch.cuda.synchronize()
    print("gemm counters run done", flush=True)


def ingest_gemm_counters(csv_path, command):
    """MFMA work and utilization of the GEMM's kernel from one counter pass
    (GEMM_COUNTERS) into profiles/counters.json: i8 ops = MOPS_I8 * 512 per
    dispatch (against 2MKN); the MFMA busy share = the MFMA busy cycles
    (summed over the 1024 SIMDs) over 1024 x the GPU-active cycles of one XCD
    (the file sums GRBM_GUI_ACTIVE over the 8 XCDs), rocprofv3's MfmaUtil;
    medians over the last 20 dispatches."""
    import csv

    vals, dur = {}, {}
    with open(csv_path) as f:
        for row in csv.DictReader(f):
            if "k_gemm" not in row["Kernel_Name"]:
                continue
            key = (row["Kernel_Name"], row["Counter_Name"])
            vals.setdefault(key, {}).setdefault(int(row["Dispatch_Id"]), 0.0)
            vals[key][int(row["Dispatch_Id"])] += float(row["Counter_Value"])
            dur[int(row["Dispatch_Id"])] = (int(row["End_Timestamp"]) - int(row["Start_Timestamp"])) * 1e-9
    kernels = {k for k, _ in vals}
    if len(kernels) != 1:
        raise SystemExit(f"expected one GEMM kernel, found {sorted(kernels)}")
    kname = kernels.pop()

    def med(c):
        v = [x for _, x in sorted(vals[(kname, c)].items())][-20:]
        return sorted(v)[len(v) // 2]

    M, K, N = 4096, 256, 32000
    mops, busy, gui = med("SQ_INSTS_VALU_MFMA_MOPS_I8"), med("SQ_VALU_MFMA_BUSY_CYCLES"), med("GRBM_GUI_ACTIVE")
    gui_xcd = gui / 8
    d = sorted(dur[i] for i in sorted(dur)[-20:])[10]
    rec = {"source_hash": _gemm_source_hash(), "kernel": kname, "i8_ops_per_launch": mops * 512,
           "alg_ops": 2 * M * K * N, "mfma_busy_cycles_per_simd": busy / 1024, "gpu_active_cycles_per_xcd": gui_xcd,
           "duration_us": round(d * 1e6, 2),
           "mfma_busy_frac": round(busy / 1024 / gui_xcd, 4), "command": command}
    path = os.path.join(ROOT, "profiles", "counters.json")
    data = {}
    if os.path.exists(path):
        with open(path) as f:
            data = json.load(f)
    data[GEMM_TAG] = rec
    with open(path, "w") as f:
        json.dump(data, f, indent=1)
    print(json.dumps(rec))


def _gemm_counters():
    path = os.path.join(ROOT, "profiles", "counters.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f).get(GEMM_TAG)
    if not rec or rec.get("source_hash") != _gemm_source_hash():
        return None
    return {k: rec[k] for k in ("mfma_busy_frac", "i8_ops_per_launch", "duration_us")}


def ingest_counters(fetch_csv, write_csv, command):
    """profiles/counters.json from the FETCH_SIZE and WRITE_SIZE passes."""
    import csv

    def per_kernel(path, counter):
        vals = {}
        with open(path) as f:
            for row in csv.DictReader(f):
                if row["Counter_Name"] != counter:
                    continue
                vals.setdefault(row["Kernel_Name"], []).append(float(row["Counter_Value"]))
        return vals

    out = {}
    for counter, path in (("FETCH_SIZE", fetch_csv), ("WRITE_SIZE", write_csv)):
        vals = per_kernel(path, counter)
        roof = [v for k, v in vals.items() if "k_step_logits" in k]
        others = {k: v for k, v in vals.items() if "k_step_logits" not in k and "mnmt" not in k}
        copy_name, copy_vals = max(others.items(), key=lambda kv: max(kv[1]))
        factor = COPY_BYTES / max(copy_vals)  # bytes per counter unit
        per_launch = sorted(roof[0])[len(roof[0]) // 2] * factor  # median over the launches
        out[counter] = {"per_launch_bytes": per_launch, "bytes_per_unit": factor, "copy_kernel": copy_name,
                        "copy_counter": max(copy_vals), "launches": len(roof[0])}
    rec = {"source_hash": _source_hash(), "kernel": ROOF_KERNEL,
           "hbm_bytes_per_launch": round(out["FETCH_SIZE"]["per_launch_bytes"] + out["WRITE_SIZE"]["per_launch_bytes"]),
           "fetch": out["FETCH_SIZE"], "write": out["WRITE_SIZE"], "command": command}
    path = os.path.join(ROOT, "profiles", "counters.json")
    data = {}
    if os.path.exists(path):
        with open(path) as f:
            data = json.load(f)
    data[ROOF_TAG] = rec
    os.makedirs(os.path.dirname(path), exist_ok=True)
    with open(path, "w") as f:
        json.dump(data, f, indent=1)
    print(json.dumps(rec))


def ingest_trace(stats_csv, command):
    """The roofline kernel's average kernel-trace duration (rocprofv3
    --kernel-trace --stats of a bench.py run, its kernel_stats.csv) into
    profiles/counters.json, keyed by the kernel sources' hash like the
    counters."""
    import csv

    calls, total_ns = 0, 0.0
    with open(stats_csv) as f:
        for row in csv.DictReader(f):
            if ROOF_KERNEL in row["Name"].replace("mnmt::(anonymous namespace)::", ""):
                calls += int(row["Calls"])
                total_ns += float(row["TotalDurationNs"])
    if not calls:
        raise SystemExit(f"{ROOF_KERNEL} not in {stats_csv}")
    rec = {"source_hash": _source_hash(), "kernel": ROOF_KERNEL, "avg_us": round(total_ns / calls / 1e3, 4),
           "calls": calls, "command": command}
    path = os.path.join(ROOT, "profiles", "counters.json")
    data = {}
    if os.path.exists(path):
        with open(path) as f:
            data = json.load(f)
    data[ROOF_TAG + "_trace"] = rec
    with open(path, "w") as f:
        json.dump(data, f, indent=1)
    print(json.dumps(rec))


def _host_cpu():
    try:
        with open("/proc/cpuinfo") as f:
            for ln in f:
                if ln.startswith("model name"):
                    return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(workload, min_seconds=10.0):
    """The oracle (scalar C, one thread) translating the workload's batch
    repeatedly for about min_seconds; also returns its output, which the GPU
    translations must equal."""
    import oracle
    from synth import generate as G

    m = oracle.Model(G.build_model(workload.model))
    src, lens = G.workload_inputs(workload)
    n, t0 = 0, time.perf_counter()
    while True:
        ref = m.greedy(src, lens, workload.steps)
        n += 1
        el = time.perf_counter() - t0
        if el >= min_seconds and n >= 2:
            break
    rec = {"value": n * workload.steps * workload.batch / el, "unit": "tokens/s", "cores": 1, "kind": "oracle",
           "host_cpu": _host_cpu(), "host_cpus_visible": os.cpu_count(),
           "sample": f"{n} sentences of the same workload (batch 1, 30 source tokens, 30 greedy steps), "
                     f"{el:.1f} s, single-threaded scalar C"}
    return rec, ref


def oracle_greedy(workload):
    import oracle
    from synth import generate as G

    src, lens = G.workload_inputs(workload)
    return oracle.Model(G.build_model(workload.model)).greedy(src, lens, workload.steps)


def check_tokens(what, got_out, got_len, ref):
    """Exit non-zero unless the GPU's tokens and lengths equal the oracle's."""
    import numpy as np

    if not (np.array_equal(got_out, ref[0]) and np.array_equal(got_len, ref[1])):
        print(f"bench.py: {what}: the GPU output differs from the oracle's; no figure is reported",
              file=sys.stderr, flush=True)
        sys.exit(3)


def memory_read_gbs(torch, mnmt, dev):
    """Read bandwidth of the probe kernel: a 64 MiB buffer read 32 times per
    launch (per XCD 8 MiB, twice its L2: the data streams from the 256 MB
    last-level cache) and a 4 GiB buffer read once (HBM).  Median of 5 timed
    launches after 2 untimed ones, each between two events."""
    import numpy as np

    sink = torch.empty(mnmt.DEBUG_READ_BLOCKS, dtype=torch.int32, device=dev)
    out = {}
    for name, nbytes, reps in (("llc_64MiB", 64 << 20, 32), ("hbm_4GiB", 4 << 30, 1)):
        x = torch.ones(nbytes // 4, dtype=torch.int32, device=dev)
        ts = []
        for i in range(7):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            mnmt.mnmt_debug_read(x, sink, reps)
            e1.record()
            e1.synchronize()
            if i >= 2:
                ts.append(e0.elapsed_time(e1))
        out[name] = round(nbytes * reps / (float(np.median(ts)) * 1e-3) / 1e9, 1)
        del x
    torch.cuda.synchronize()
    return out


def qlinear_sweep(torch, mnmt, G, dev, reps=100):
    """The quantized-linear sweep: X int8 [M, K] x W int8 [N, K], int32
    accumulation, folded per-channel requant to int8, for M in {1, 4, 64, 256,
    4096} and (K, N) in {(256, 1024), (1024, 256), (512, 2048), (256, 32000)}.
    Each shape: 3 untimed launches, then ``reps`` back to back between two
    events (launch gaps included).  Roofline per shape: the larger of the i8
    matrix-core time 2MKN / 5.0 POP/s and the memory time of its algorithmic
    bytes (X, W, 8 B of constants per column, the int8 output) at 8 TB/s."""
    stream = torch.cuda.current_stream()
    mark = torch.empty(1, device=dev)
    rows = []
    for K, N in G.SWEEP_KN:
        for M in G.SWEEP_M:
            X, W, mult, bias = (torch.from_numpy(a).to(dev) for a in G.sweep_case(M, K, N))
            mark.fill_(float(M))  # a fill kernel separates the shapes in a kernel trace
            Y = torch.empty((M, N), dtype=torch.int8, device=dev)
            g = lambda: mnmt.mnmt_qlinear(X, W, mult, bias, mnmt.EPI_I8, out=Y, stream=stream)  # noqa: E731
            _warm(torch, g)
            ms = _events_ms(torch, g, reps, stream)
            ops = 2.0 * M * K * N
            nbytes = M * K + N * K + 8 * N + M * N
            t_mfma = ops / (I8_PEAK_TOPS * 1e12)
            t_mem = nbytes / (HBM_PEAK_GBS * 1e9)
            t_roof = _sweep_roofline_us(M, K, N) * 1e-6
            rows.append({"M": M, "K": K, "N": N, "us": round(ms * 1e3, 3), "tops": round(ops / (ms * 1e-3) / 1e12, 2),
                         "gbs": round(nbytes / (ms * 1e-3) / 1e9, 1), "bound": "mfma" if t_mfma >= t_mem else "hbm",
                         "roof_us": round(t_roof * 1e6, 3), "frac": round(t_roof / (ms * 1e-3), 4)})
            print(f"sweep M={M} K={K} N={N}: {ms * 1e3:.2f} us, roofline {rows[-1]['bound']} "
                  f"{t_roof * 1e6:.2f} us, frac {rows[-1]['frac']:.3f}", file=sys.stderr, flush=True)
    return rows


def _sweep_roofline_us(M, K, N):
    ops = 2.0 * M * K * N
    nbytes = M * K + N * K + 8 * N + M * N
    return max(ops / (I8_PEAK_TOPS * 1e12), nbytes / (HBM_PEAK_GBS * 1e9)) * 1e6


def sweep_trace_summary(trace_csv, command):
    """Per-shape kernel durations of ``--sweep`` from a rocprofv3 kernel trace
    (the fill kernel before each shape splits the dispatches), as markdown."""
    import csv

    with open(trace_csv) as f:
        recs = sorted(csv.DictReader(f), key=lambda r: int(r["Start_Timestamp"]))
    groups = []
    for r in recs:
        name = r["Kernel_Name"]
        if "Fill" in name or "fill" in name:
            groups.append([])
        elif groups and "mnmt::" in name:
            groups[-1].append((name, (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3))
    from synth import generate as G

    shapes = [(M, K, N) for K, N in G.SWEEP_KN for M in G.SWEEP_M]
    if len(groups) != len(shapes):
        raise SystemExit(f"expected {len(shapes)} shape groups, found {len(groups)}")
    out = ["| M | K | N | kernel(s) | launches | mean µs | roofline µs | frac |", "|---:|---:|---:|---|---:|---:|---:|---:|"]
    for (M, K, N), g in zip(shapes, groups):
        names = sorted({n.replace("void ", "").replace("mnmt::(anonymous namespace)::", "").split("(")[0] for n, _ in g})
        timed = g[-100:]  # one kernel per call: the timed launches are the last 100
        calls = len(timed)
        mean_us = sum(d for _, d in timed) / max(1, calls)
        roof = _sweep_roofline_us(M, K, N)
        out.append(f"| {M} | {K} | {N} | `{'`, `'.join(names)}` | {calls} | {mean_us:.2f} | {roof:.2f} | {roof / mean_us:.3f} |")
    print(f"Command: `{command}`\n" if command else "", end="")
    print("\n".join(out))


# Beam side measurements: (workload, weight bits); 4-bit models are loaded
# with their weights packed only, so every kernel reads the packed rows.
BEAM_RUNS = {"mobile_beam": ("mobile_beam", 8), "mobile_beam_w4_packed": ("mobile_beam", 4),
             "base_beam": ("base_beam", 8)}


def beam_throughput(torch, mnmt, G, dev, names=tuple(BEAM_RUNS), reps=3, check=True):
    """The two batched beam-search workloads (mobile: 64 sentences, base: 128;
    beam 4, length penalty 0.6), and the mobile one with packed 4-bit weights,
    each translation one captured graph, inputs resident on the device: one
    untimed translation, then ``reps`` timed back to back, then 10 more each
    alone between two events (median, p10, p90).
    The last translation's shortest sentence is compared with the oracle, and
    a composite roofline (the sum over phases of max(ops / i8 peak, bytes /
    HBM peak), paper_2306_04235_amd.workload.beam_roofline_s) over the steps
    the batch ran gives the fraction."""
    import dataclasses

    import numpy as np

    from paper_2306_04235_amd import workload as WL

    res = {}
    for name in names:
        wname, bits = BEAM_RUNS[name]
        w = G.WORKLOADS[wname]
        mcfg = w.model if bits == 8 else dataclasses.replace(w.model, name=w.model.name + "-w4", w_bits=4)
        blob = G.build_model(mcfg)
        m = mnmt.Model(blob, flags=mnmt.LOAD_PACKED_4BIT_ONLY if bits == 4 else 0)
        src, lens = G.workload_inputs(w)
        ts, tl = torch.from_numpy(src).to(dev), torch.from_numpy(lens).to(dev)
        sess = mnmt.Session(m, w.batch, w.s_max, w.steps, w.beam)
        outs = (torch.empty((w.batch, w.steps), dtype=torch.int32, device=dev),
                torch.empty(w.batch, dtype=torch.int32, device=dev),
                torch.empty(w.batch, dtype=torch.float32, device=dev))
        run = lambda: sess.translate(ts, tl, beam=w.beam, max_steps=w.steps, alpha=w.alpha,  # noqa: E731
                                     use_graph=True, out=outs)
        run()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(reps):
            run()
        torch.cuda.synchronize()
        el = (time.perf_counter() - t0) / reps
        # per-batch distribution: each translation alone between two events
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(10)]
        for e0, e1 in ev:
            e0.record()
            run()
            e1.record()
            e1.synchronize()
        one = np.sort([e0.elapsed_time(e1) for e0, e1 in ev])
        sess.status()
        toks = int(outs[1].sum().item())
        out_np, len_np = outs[0].cpu().numpy(), outs[1].cpu().numpy()
        if check:  # the shortest source against the oracle
            import oracle

            i = int(np.argmin(lens))
            om = oracle.Model(blob)
            ref = om.beam(src[i:i + 1], lens[i:i + 1], w.beam, w.steps, w.alpha)
            check_tokens(f"{name} sentence {i}", out_np[i:i + 1], len_np[i:i + 1], ref)
        steps_run = int(len_np.max())
        m_dims = WL.Dims(m.info.d_model, m.info.n_heads, m.info.d_ffn, m.info.n_enc, m.info.n_dec, m.info.vocab)
        roof = WL.beam_roofline_s(m_dims, lens, w.beam, steps_run, I8_PEAK_TOPS * 1e12, HBM_PEAK_GBS * 1e9)
        res[name] = {"workload": w.name + ("" if bits == 8 else "-w4-packed"), "arena_bytes": m.arena.numel(),
                     "ms_per_batch": round(el * 1e3, 3), "sentences_per_s": round(w.batch / el, 1),
                     "output_tokens_per_s": round(toks / el, 1), "batch": w.batch, "beam": w.beam,
                     "max_steps": w.steps, "steps_run": steps_run,
                     "ms_per_batch_alone": {"median": round(float(np.median(one)), 3), "p10": round(float(one[1]), 3),
                                            "p90": round(float(one[8]), 3), "runs": len(one)},
                     "composite_roofline": {"ms": round(roof["seconds"] * 1e3, 4),
                                            "frac": round(roof["seconds"] / el, 4),
                                            "parts_ms": {k: round(v["seconds"] * 1e3, 4)
                                                         for k, v in roof["parts"].items()}}}
        sess.close()
        m.close()
    return res


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-paper-shapes", action="store_true", help="skip the paper-shape side measurements")
    ap.add_argument("--no-beam", action="store_true", help="skip the batched beam-search side measurements")
    ap.add_argument("--beam-only", nargs="?", const="all", choices=("all", *BEAM_RUNS),
                    help="only the batched beam-search measurements (for profiling), optionally one workload")
    ap.add_argument("--sweep", action="store_true", help="only the quantized-linear sweep (20 shapes, I8 epilogue)")
    ap.add_argument("--counters", action="store_true", help="only the roofline kernel and the copy (for --pmc)")
    ap.add_argument("--ingest-counters", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"))
    ap.add_argument("--ingest-trace", metavar="KERNEL_STATS_CSV",
                    help="record the roofline kernel's kernel-trace average from a rocprofv3 --stats file")
    ap.add_argument("--ingest-command", default="")
    ap.add_argument("--sweep-trace", metavar="KERNEL_TRACE_CSV", help="summarize a kernel trace of --sweep")
    ap.add_argument("--gemm-counters", action="store_true",
                    help="only the 4096x256x32000 GEMM, 25 launches (for one --pmc pass of " + " ".join(GEMM_COUNTERS)
                    + ")")
    ap.add_argument("--beam-counters", action="store_true",
                    help="only one eager translation of the base beam workload (for a --pmc pass)")
    ap.add_argument("--ingest-gemm-counters", metavar="COUNTER_CSV",
                    help="record the GEMM's MFMA counters from a --gemm-counters pass")
    args = ap.parse_args()
    if args.ingest_gemm_counters:
        ingest_gemm_counters(args.ingest_gemm_counters, args.ingest_command)
        return
    if args.sweep_trace:
        sweep_trace_summary(args.sweep_trace, args.ingest_command)
        return
    if args.ingest_trace:
        ingest_trace(args.ingest_trace, args.ingest_command)
        return
    if args.ingest_counters:
        ingest_counters(*args.ingest_counters, args.ingest_command)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported (the batch-1 path does not "
              "shard; larger batches shard by sentence, see the design notes)", file=sys.stderr)
        sys.exit(2)
    if args.counters:
        counters_run()
        return
    if args.gemm_counters:
        gemm_counters_run()
        return
    if args.beam_counters:
        beam_counters_run()
        return

    import numpy as np
    import torch

    from paper_2306_04235_amd import mnmt, workload as WL
    from synth import generate as G

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    if args.sweep:
        print(json.dumps({"qlinear_sweep": qlinear_sweep(torch, mnmt, G, dev)}), flush=True)
        return
    if args.beam_only:
        names = tuple(BEAM_RUNS) if args.beam_only == "all" else (args.beam_only,)
        print(json.dumps({"beam_throughput": beam_throughput(torch, mnmt, G, dev, names)}), flush=True)
        return
    w = G.WORKLOADS["mobile"]
    blob = G.build_model(w.model)
    model = mnmt.Model(blob)
    info = model.info
    src, lens = G.workload_inputs(w)
    tsrc = torch.from_numpy(src).to(dev)
    tlen = torch.from_numpy(lens).to(dev)
    sess = mnmt.Session(model, w.batch, w.s_max, w.steps, 1)
    stream = torch.cuda.current_stream()
    outs = (torch.empty((w.batch, w.steps), dtype=torch.int32, device=dev),
            torch.empty(w.batch, dtype=torch.int32, device=dev), torch.empty(w.batch, dtype=torch.float32, device=dev))

    def step(o=None):
        sess.translate(tsrc, tlen, beam=1, max_steps=w.steps, use_graph=True, out=o or outs)

    # the oracle's translation of the same sentence, which the timed ones must equal
    if args.no_cpu_baseline:
        ref = oracle_greedy(w)
    else:
        cpu_rec, ref = cpu_baseline(w)
    for _ in range(args.warmup):
        step()
    # every timed translation writes its own outputs, all compared afterwards
    touts = [(torch.empty((w.batch, w.steps), dtype=torch.int32, device=dev),
              torch.empty(w.batch, dtype=torch.int32, device=dev),
              torch.empty(w.batch, dtype=torch.float32, device=dev)) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        step(touts[k])
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    sess.status()  # raises if a chained kernel's wait gave up during the timed translations
    for k, o in enumerate(touts):
        check_tokens(f"timed translation {k}", o[0].cpu().numpy(), o[1].cpu().numpy(), ref)
    outs = touts[-1]
    tokens = int(outs[1].sum().item()) * args.steps
    ms_per_sentence = elapsed * 1e3 / (args.steps * w.batch)
    dims = WL.Dims(info.d_model, info.n_heads, info.d_ffn, info.n_enc, info.n_dec, info.vocab)
    sent_bytes = WL.greedy_sentence_bytes(dims, int(lens[0]), w.steps)
    sent_gbs = sent_bytes / (ms_per_sentence * 1e-3) / 1e9
    sentence_roofline = {"bound": "hbm", "alg_bytes": sent_bytes, "achieved": round(sent_gbs, 1),
                         "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(sent_gbs / HBM_PEAK_GBS, 4)}

    # Latency distribution (outside the timed region): 50 translations, each
    # between two events on the stream.
    lat = []
    cur = torch.cuda.current_stream()
    for _ in range(50):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(cur)
        step()
        e1.record(cur)
        e1.synchronize()
        lat.append(e0.elapsed_time(e1))
        check_tokens("latency translation", outs[0].cpu().numpy(), outs[1].cpu().numpy(), ref)
    sess.status()
    lat_ms = {"median": round(float(np.median(lat)), 4), "p10": round(float(np.percentile(lat, 10)), 4),
              "p90": round(float(np.percentile(lat, 90)), 4), "runs": len(lat)}

    # Dominant kernel: the decoder's fused logits + arg-max over the int8
    # embedding (batch 1), launched alone on one int8 row.
    fn, alg_bytes = _roofline_kernel(torch, np, mnmt, WL, G, info, blob, dev, None)  # the current stream
    for _ in range(10):
        fn()
    kern_ms = _graph_launch_ms(torch, fn)
    achieved = alg_bytes / (kern_ms * 1e-3) / 1e9
    roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": _traffic(ROOF_TAG),
                "kernel": ROOF_KERNEL + " (fused logits + arg-max, M=1 K=256 N=32000)",
                "alg_bytes_per_launch": alg_bytes, "avg_us": round(kern_ms * 1e3, 3),
                "data": "the 8.19 MB embedding stays in the last-level cache across back-to-back launches; "
                        "peak is the HBM figure, see llc_read_gbs for the cache's measured rate"}
    trace = _trace_avg_us(ROOF_TAG)
    if trace:
        roofline["trace_avg_us"] = trace
        roofline["trace_frac"] = round(alg_bytes / (trace * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)
    mem = memory_read_gbs(torch, mnmt, dev)
    roofline["llc_read_gbs"] = mem["llc_64MiB"]
    roofline["hbm_read_gbs"] = mem["hbm_4GiB"]
    roofline["frac_of_measured_llc"] = round(achieved / mem["llc_64MiB"], 4)

    # Largest quantized-linear sweep shape on the matrix cores.
    g, (M, K, N) = _gemm_case(torch, dev)
    _warm(torch, g)
    gemm_ms = _events_ms(torch, g, 20, stream)
    tops = 2.0 * M * K * N / (gemm_ms * 1e-3) / 1e12
    qgemm = {"shape": [M, K, N], "epilogue": "i8 requant", "tops": round(tops, 1), "peak": I8_PEAK_TOPS,
             "frac": round(tops / I8_PEAK_TOPS, 4), "avg_us": round(gemm_ms * 1e3, 2)}
    gc = _gemm_counters()  # committed MFMA counters of the same kernel source, if any
    if gc:
        qgemm["counters"] = gc

    # The paper's own MobileNMT-10MB / 20MB shapes on the same batch-1 path
    # (context beside the paper's phone latencies, not the headline workload),
    # and the workload model with 4-bit linear weights (the paper's W-E-A
    # 4-8-8 setting) loaded packed only.
    import dataclasses

    paper = {}
    mob4 = dataclasses.replace(G.MOBILE, name="mobile-12-2-w4-packed", w_bits=4)
    for cfg in () if args.no_paper_shapes else (G.PAPER_10MB, G.PAPER_20MB, mob4):
        flags = mnmt.LOAD_PACKED_4BIT_ONLY if cfg is mob4 else 0
        pblob = G.build_model(cfg)
        pm = mnmt.Model(pblob, flags=flags)
        if cfg is mob4:
            psrc, plen = src, lens
        else:
            psrc, plen = G.make_sources(cfg.vocab, 1, [30], seed=2010 + cfg.d_model, s_max=30)
        ps = mnmt.Session(pm, 1, 30, 30, 1)
        pt, pl = torch.from_numpy(psrc).to(dev), torch.from_numpy(plen).to(dev)
        pouts = (torch.empty((1, 30), dtype=torch.int32, device=dev), torch.empty(1, dtype=torch.int32, device=dev),
                 torch.empty(1, dtype=torch.float32, device=dev))
        for _ in range(5):
            ps.translate(pt, pl, beam=1, max_steps=30, use_graph=True, out=pouts)
        torch.cuda.synchronize()
        p0 = time.perf_counter()
        for _ in range(20):
            ps.translate(pt, pl, beam=1, max_steps=30, use_graph=True, out=pouts)
        torch.cuda.synchronize()
        pe = time.perf_counter() - p0
        paper[cfg.name] = {"ms_per_sentence": round(pe * 1e3 / 20, 4),
                           "tokens_per_s": round(int(pouts[1].sum().item()) * 20 / pe, 1),
                           "arena_bytes": int(pm.arena.numel())}
        if cfg is mob4:  # the same sentence as the headline, checked against the oracle
            import oracle

            ps.status()
            r4 = oracle.Model(pblob).greedy(psrc, plen, 30)
            check_tokens("4-bit translations", pouts[0].cpu().numpy(), pouts[1].cpu().numpy(), r4)
        ps.close()
        pm.close()

    line = {
        "metric": "decoded tokens/sec at batch 1 (greedy, 30-token sentences)",
        "value": round(tokens / elapsed, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(elapsed * 1e3 / args.steps, 4),
        "ms_per_sentence": round(ms_per_sentence, 4),
        "latency_ms_per_sentence": lat_ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int8",
        "data": "synthetic",
        "config": {"workload": w.name, "batch": w.batch, "src_len": int(lens[0]), "greedy_steps": w.steps,
                   "d_model": info.d_model, "heads": info.n_heads, "ffn": info.d_ffn, "enc_layers": info.n_enc,
                   "dec_layers": info.n_dec, "vocab": info.vocab, "graph": True},
        "roofline": roofline,
        "sentence_roofline": sentence_roofline,
        "qgemm": qgemm,
        "paper_shapes_b1_greedy30": paper,
    }
    if not args.no_beam:
        line["beam_throughput"] = beam_throughput(torch, mnmt, G, dev)
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_rec
    print(json.dumps(line), flush=True)
    sess.close()
    model.close()


if __name__ == "__main__":
    main()
