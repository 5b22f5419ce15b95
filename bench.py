"""Benchmark: one VSC layer (rule-book build + forward) on MI355X.

Workload (default): 8 voxelised surfaces on a 128^3 grid, ~100k active sites
each (~900k in total), VSC 3^3, 64 -> 64 planes, bf16 features and weights,
fp32 accumulation, bf16 output, fp32 bias.  A step is one pass of the whole
hot path on resident inputs: build the rule book (site map, neighbour probe,
per-offset compaction) and run the forward multiply-add.

Prints one JSON line:
  value      active sites per second over whole steps (build + forward)
  roofline   the forward kernel (the dominant one) against the bf16 dense
             matrix-core peak, from HIP events around each forward launch
  phases     rule book and forward per step: means, 10/50/90th percentiles,
             and medians of a few extra steps run after evicting the caches
  cpu_baseline  the oracle on one sample of the same workload, host cores

Other modes (not the benchmark line): --workload with a multi-layer stack
(VSC levels joined by SC) times the whole stack; --peaks measures a plain
device copy and a library bf16 GEMM as achievable-peak references; --ops
times sparse pooling, DC and the gradients (one JSON line per op).
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAKS = {  # MI355X published dense peaks
    "bf16": 2500.0,    # TFLOP/s
    "f32": 157.3,      # TFLOP/s
    "hbm": 8000.0,     # GB/s
}


def _args():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--workload", default="surf128x8_vsc3_c64_bf16")
    p.add_argument("--variant", default="matched", choices=["matched", "literal"])
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-samples", type=int, default=2,
                   help="samples of the batch the single-thread oracle baseline runs on")
    p.add_argument("--calib-copy-mb", type=int, default=0,
                   help="run one plain device copy of this many MiB (counter calibration)")
    p.add_argument("--peaks", action="store_true",
                   help="measure a device copy and a bf16 library GEMM instead")
    p.add_argument("--cold-steps", type=int, default=10,
                   help="extra steps after a cache-evicting write each (reported apart)")
    p.add_argument("--ops", action="store_true",
                   help="time pooling, DC and the gradients instead")
    p.add_argument("--stack-sync", action="store_true",
                   help="stack mode: wait for each SC build's output count on the host "
                        "instead of chaining the next build on the device-side count")
    return p.parse_args()


def knobs():
    """The library's environment switches as set for this run (None = default)."""
    return {k: os.environ.get(k) for k in ("SPCONV_RULEBOOK", "SPCONV_FORCE_PATH",
                                           "SPCONV_HASH_LAYOUT", "SPCONV_TEST_HASH_SLOTS")}


def kernel_source_hash():
    h = hashlib.sha256()
    for f in ("forward.hip", "forward_kernels.h", "forward_w0.hip", "forward_types.h"):
        with open(os.path.join(ROOT, "paper_1706_01307_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def load_traffic(kernel, workload):
    """HBM bytes per launch from a committed rocprofv3 counter summary, or
    None when absent or taken on a different kernel source."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel}_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as fh:
        t = json.load(fh)
    if t.get("source_hash") != kernel_source_hash():
        return None
    return t.get("hbm_bytes_per_launch")


def cpu_model():
    """The host CPU's model name (from /proc/cpuinfo), or None."""
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def forward_kernel(c_in, c_out, bf16, n):
    """The forward kernel the library picks for these channel counts (the
    library's own dispatch rule): the matrix cores for bf16 C_in of 32 / 64 /
    96 / 128 or fp32 C_in of 16 ... 128 with C_out a multiple of 16, else the
    one-plane-group kernel for at most 4 input planes on at least 2048 rows
    (C_out a multiple of 16), else one lane per output element."""
    mfma_cin = (32, 64, 96, 128) if bf16 else (16, 32, 64, 96, 128)
    if c_out % 16 == 0 and c_in in mfma_cin:
        return "k_fwd_mfma"
    if c_in <= 4 and n >= 2048 and c_out % 16 == 0:
        return "k_fwd_lowc"
    return "k_fwd_vec"


def cpu_baseline(wl, x_bits, w_bits, bias, n_samples):
    """The oracle (std::map rule book + double-precision forward, both
    parallel over output rows on OpenMP threads) timed on this host: the whole
    workload on every thread OpenMP is given, and the first samples of the
    batch on one thread (a bounded slice; its rate is reported per site)."""
    import oracle
    in_dt = oracle.BF16 if wl.dtype == "bf16" else oracle.F32
    f = [1] + [3] * wl.d

    def run(rows):
        t0 = time.perf_counter()
        rb = oracle.Rulebook(oracle.VSC, wl.coords[rows], wl.spatial_size, f)
        t1 = time.perf_counter()
        rb.forward(x_bits[rows], w_bits, bias, in_dt=in_dt)
        t2 = time.perf_counter()
        return t1 - t0, t2 - t1

    threads = oracle.set_threads(0)
    n = len(wl.coords)
    tb, tf = run(np.arange(n))
    sample = np.nonzero(wl.coords[:, 0] < n_samples)[0]
    oracle.set_threads(1)
    try:
        sb, sf = run(sample)
    finally:
        oracle.set_threads(threads)
    return {"value": n / (tb + tf), "unit": "active sites/s", "cores": threads,
            "kind": "oracle", "cpu_model": cpu_model(), "host_cpus": os.cpu_count(),
            "sample": f"the whole workload ({n} sites) on {threads} OpenMP threads: rule book "
                      f"{tb:.2f} s + forward {tf:.2f} s",
            "single_thread": {"value": len(sample) / (sb + sf), "unit": "active sites/s",
                              "cores": 1,
                              "sample": f"samples 0..{n_samples - 1} of the batch "
                                        f"({len(sample)} sites) on one thread: rule book "
                                        f"{sb:.2f} s + forward {sf:.2f} s"}}


def main():
    a = _args()
    if a.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU only; --gpus must be 1"}))
        sys.exit(2)
    import torch
    import paper_1706_01307_amd as spc
    from paper_1706_01307_amd import _lib, inputs

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    lib = _lib.load()
    dev = torch.device("cuda:0")
    if a.peaks:
        measure_peaks(torch, dev)
        return
    if a.ops:
        run_ops(a, torch, dev, spc, inputs)
        return
    wl = inputs.make_workload(a.workload, variant=a.variant)
    if len(wl.layers) > 1:
        run_stack(a, wl, torch, dev, lib, _lib, inputs)
        return
    layer = wl.layers[0]
    assert layer.kind == "vsc", "bench times a single VSC layer or a stack"
    N, D = len(wl.coords), wl.d + 1
    K = layer.f ** wl.d
    Cin, Cout = layer.c_in, layer.c_out
    bf16 = wl.dtype == "bf16"

    xf = inputs.normal_f32((N, Cin), seed=11)
    wf = inputs.normal_f32((K, Cin, Cout), std=1.0 / np.sqrt(K * Cin), seed=12)
    bias = inputs.normal_f32((Cout,), std=0.1, seed=13)
    if bf16:
        x_bits, w_bits = inputs.to_bf16_bits(xf), inputs.to_bf16_bits(wf)
        xt = torch.from_numpy(x_bits.view(np.int16)).view(torch.bfloat16).to(dev)
        wt = torch.from_numpy(w_bits.view(np.int16)).view(torch.bfloat16).to(dev)
        in_dt = out_dt = _lib.BF16
        yt = torch.empty((N, Cout), dtype=torch.bfloat16, device=dev)
    else:
        x_bits, w_bits = xf, wf
        xt, wt = torch.from_numpy(xf).to(dev), torch.from_numpy(wf).to(dev)
        in_dt = out_dt = _lib.F32
        yt = torch.empty((N, Cout), dtype=torch.float32, device=dev)
    bt = torch.from_numpy(bias).to(dev)
    ct = torch.from_numpy(np.ascontiguousarray(wl.coords)).to(dev).contiguous()

    size = np.array(wl.spatial_size, np.int32)
    fa = np.array([1] + [layer.f] * wl.d, np.int32)
    sa = np.ones(D, np.int32)
    stream = torch.cuda.current_stream()
    sp = ctypes.c_void_p(stream.cuda_stream)
    h = ctypes.c_void_p()
    args_build = (_lib.VSC, D, ctypes.c_void_p(ct.data_ptr()), N, size.ctypes.data,
                  fa.ctypes.data, sa.ctypes.data, _lib.BUILD_ASYNC, sp, ctypes.byref(h))
    xp, wp, bp, ypt = (ctypes.c_void_p(t.data_ptr()) for t in (xt, wt, bt, yt))

    def step(evs=None, split=True):
        if evs and split:
            evs[0].record(stream)
        _lib.check(lib.spconv_build_rulebook(*args_build), "build")
        if evs:
            evs[1].record(stream)
        _lib.check(lib.spconv_vsc_forward(h, in_dt, xp, wp, bp, out_dt, ypt, Cin, Cout, sp),
                   "forward")
        if evs:
            evs[2].record(stream)
        lib.spconv_rulebook_destroy(h)

    if a.calib_copy_mb:
        src = torch.ones(a.calib_copy_mb << 18, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    # correctness gate on this exact input before timing: a synchronous build
    # must succeed and its rule book must satisfy the VSC invariants
    rb = spc.build_rulebook(spc.VSC, ct, wl.spatial_size, fa)
    off = rb.pair_off
    k = np.diff(off)
    assert k[K // 2] == N and np.array_equal(k, k[::-1]), "rule book invariants failed"
    sum_k = int(off[-1])
    rb.close()

    for _ in range(a.warmup):
        step()
    torch.cuda.synchronize()

    # the timed steps: events around the forward only (its duration is the
    # roofline's denominator); the build's share comes from the same steps
    # run again untimed with an event before the build as well
    evt = [[None] + [torch.cuda.Event(enable_timing=True) for _ in range(2)]
           for _ in range(a.steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    host = 0.0
    for i in range(a.steps):
        h0 = time.perf_counter()
        step(evt[i], split=False)
        host += time.perf_counter() - h0
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    fwd_t = np.array([e[1].elapsed_time(e[2]) for e in evt])
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(a.steps)]
    for i in range(a.steps):
        step(evs[i])
    torch.cuda.synchronize()
    rb_t = np.array([e[0].elapsed_time(e[1]) for e in evs])
    rb_ms, fwd_ms = float(rb_t.mean()), float(fwd_t.mean())
    ms_per_step = (t1 - t0) * 1e3 / a.steps

    def pct(v):
        return [float(x) for x in np.percentile(v, [10, 50, 90])]

    # cold caches (outside the timed region): before each of a few steps a
    # 1 GiB write evicts L2 and the 256 MB Infinity Cache
    flush = torch.empty(1 << 28, dtype=torch.float32, device=dev)
    cold = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(a.cold_steps)]
    for i in range(a.cold_steps):
        flush.fill_(float(i))
        step(cold[i])
    torch.cuda.synchronize()
    del flush
    cold_rb = np.array([e[0].elapsed_time(e[1]) for e in cold])
    cold_fwd = np.array([e[1].elapsed_time(e[2]) for e in cold])

    # a last asynchronous build, checked for device-side errors
    _lib.check(lib.spconv_build_rulebook(*args_build), "build")
    _lib.check(lib.spconv_rulebook_status(h), "build status")
    lib.spconv_rulebook_destroy(h)

    flops = 2.0 * sum_k * Cin * Cout
    tflops = flops / (fwd_ms * 1e-3) / 1e12
    dt = "bf16" if bf16 else "f32"
    peak = PEAKS[dt]
    kernel = forward_kernel(Cin, Cout, bf16, N)
    traffic = load_traffic(kernel, a.workload)
    # forward algorithmic bytes: features in/out, gather map, weights, bias
    esz = 2 if bf16 else 4
    fwd_bytes = N * Cin * esz + N * Cout * esz + 4 * K * N + K * Cin * Cout * esz + 4 * Cout

    # rule-book algorithmic bytes (the unit cost the survey fixes for a VSC
    # build): coordinates read (4 D N), a hash table of cap = 2^ceil(log2 2N)
    # 8-byte slots initialised, one 12-byte insert per site, one 12-byte
    # key + value probe per site and non-centre offset, the pairs written
    # (8 per pair) and the K + 1 offsets
    cap = 1 << max(0, (2 * N - 1).bit_length())
    rb_bytes = (4 * D * N + 8 * cap + 12 * N + 12 * (K - 1) * N + 8 * sum_k + 8 * (K + 1))
    # what this build itself must write: gather map, pairs, schedule, offsets
    rb_out_bytes = 4 * K * N + 8 * sum_k + 4 * N + 8 * (K + 1)

    headline = a.workload == "surf128x8_vsc3_c64_bf16"
    out = {
        "metric": ("VSC layer active sites/sec + effective TFLOP/s (3^3, C=64, 128^3 surfaces)"
                   if headline else "VSC layer active sites/sec + effective TFLOP/s"),
        "value": N / (ms_per_step * 1e-3),
        "unit": "active sites/s",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": dt,
        "data": "synthetic",
        "config": {"workload": a.workload, "variant": a.variant, "batch": wl.batch,
                   "grid": wl.size, "active_sites": N, "sum_k": sum_k, "K": K,
                   "c_in": Cin, "c_out": Cout, "out_dtype": dt},
        "knobs": knobs(),
        "effective_tflops": tflops,
        "sites_per_s_rulebook_reuse": N / (fwd_ms * 1e-3),
        "host_enqueue_ms_per_step": host * 1e3 / a.steps,
        "phases_ms": {"rulebook": rb_ms, "forward": fwd_ms},
        "rulebook_io": {"algorithmic_bytes": rb_bytes,
                        "GBps": rb_bytes / (rb_ms * 1e-3) / 1e9, "peak_GBps": PEAKS["hbm"],
                        "frac": rb_bytes / (rb_ms * 1e-3) / 1e9 / PEAKS["hbm"],
                        "output_bytes": rb_out_bytes,
                        "output_GBps": rb_out_bytes / (rb_ms * 1e-3) / 1e9},
        "phases_ms_p10_p50_p90": {"rulebook": pct(rb_t), "forward": pct(fwd_t),
                                  "build_and_forward": pct(rb_t + fwd_t)},
        "cold_caches_ms_median": ({"steps": a.cold_steps,
                                   "rulebook": float(np.median(cold_rb)),
                                   "forward": float(np.median(cold_fwd))}
                                  if a.cold_steps > 0 else None),
        "roofline": ({"bound": "mfma", "kernel": kernel, "achieved": tflops, "peak": peak,
                      "unit": "TFLOP/s", "frac": tflops / peak, "traffic": traffic,
                      "algorithmic_bytes": fwd_bytes}
                     if kernel == "k_fwd_mfma" else
                     {"bound": "hbm", "kernel": kernel,
                      "achieved": fwd_bytes / (fwd_ms * 1e-3) / 1e9, "peak": PEAKS["hbm"],
                      "unit": "GB/s", "frac": fwd_bytes / (fwd_ms * 1e-3) / 1e9 / PEAKS["hbm"],
                      "traffic": traffic, "algorithmic_bytes": fwd_bytes}),
    }
    if not a.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl, x_bits, w_bits, bias, a.cpu_samples)
    print(json.dumps(out), flush=True)


def measure_peaks(torch, dev):
    """Achievable references on this GPU: a 1 GiB device-to-device copy
    (HBM read + write) and an 8192^3 bf16 GEMM through the vendor library."""
    def timed(fn, reps):
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps * 1e-3
    nb = 1 << 30
    src = torch.ones(nb // 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    t_copy = timed(lambda: dst.copy_(src), 20)
    del src, dst
    n = 8192
    a = torch.randn((n, n), dtype=torch.bfloat16, device=dev).contiguous()
    b = torch.randn((n, n), dtype=torch.bfloat16, device=dev).contiguous()
    t_mm = timed(lambda: torch.matmul(a, b), 10)
    print(json.dumps({
        "copy_GBps": 2 * nb / t_copy / 1e9, "copy_bytes": nb,
        "bf16_gemm_TFLOPs": 2 * n ** 3 / t_mm / 1e12, "gemm_shape": [n, n, n],
        "spec": {"hbm_GBps": PEAKS["hbm"], "bf16_TFLOPs": PEAKS["bf16"]}}), flush=True)


def run_stack(a, wl, torch, dev, lib, _lib, inputs):
    """A stack of layers: VSC levels joined by strided SC layers.  One VSC
    rule book per level serves all its VSC layers (Section 4: layers on the
    same sites share it).  By default every build after the first is chained
    on the last SC book (its output sites and device-side count) and feature
    buffers are sized by the books' row bounds, so a step enqueues all its
    work without the host waiting; --stack-sync instead reads each SC book's
    output count on the host before the next level.  A step = every build +
    every forward + releases."""
    D = wl.d + 1
    bf16 = wl.dtype == "bf16"
    esz = 2 if bf16 else 4
    tdt = torch.bfloat16 if bf16 else torch.float32
    dt_code = _lib.BF16 if bf16 else _lib.F32
    N0 = len(wl.coords)
    ct = torch.from_numpy(np.ascontiguousarray(wl.coords)).to(dev).contiguous()
    params = []
    for j, L in enumerate(wl.layers):
        K = L.f ** wl.d
        wf = inputs.normal_f32((K, L.c_in, L.c_out), std=1.0 / np.sqrt(K * L.c_in), seed=100 + j)
        bf = inputs.normal_f32((L.c_out,), std=0.1, seed=200 + j)
        if bf16:
            wt = torch.from_numpy(inputs.to_bf16_bits(wf).view(np.int16)).view(torch.bfloat16).to(dev)
        else:
            wt = torch.from_numpy(wf).to(dev)
        params.append((wt, torch.from_numpy(bf).to(dev)))
    xf = inputs.normal_f32((N0, wl.layers[0].c_in), seed=11)
    if bf16:
        x0 = torch.from_numpy(inputs.to_bf16_bits(xf).view(np.int16)).view(torch.bfloat16).to(dev)
    else:
        x0 = torch.from_numpy(xf).to(dev)
    stream = torch.cuda.current_stream()
    sp = ctypes.c_void_p(stream.cuda_stream)
    chain = not a.stack_sync
    info = []

    def rows_out(h):
        if chain:
            nb_in, nb_out = ctypes.c_int64(), ctypes.c_int64()
            _lib.check(lib.spconv_rulebook_bounds(h, ctypes.byref(nb_in), ctypes.byref(nb_out)),
                       "bounds")
            return nb_out.value
        n_out = ctypes.c_int64()
        _lib.check(lib.spconv_rulebook_query(h, None, ctypes.byref(n_out), None, None, None),
                   "query")
        return n_out.value

    # per-layer arguments that do not change from step to step
    size0 = np.array(wl.spatial_size, np.int32)
    largs = []
    for j, L in enumerate(wl.layers):
        f = np.array([1] + [L.f] * wl.d, np.int32)
        s = np.array([1] + [L.s] * wl.d, np.int32)
        wt, bt = params[j]
        largs.append((f, s, f.ctypes.data, s.ctypes.data,
                      _lib.VSC if L.kind == "vsc" else _lib.SC,
                      _lib.BUILD_ASYNC if (chain or L.kind == "vsc") else 0,
                      lib.spconv_vsc_forward if L.kind == "vsc" else lib.spconv_sc_forward,
                      ctypes.c_void_p(wt.data_ptr()), ctypes.c_void_p(bt.data_ptr())))
    coords0 = ctypes.c_void_p(ct.data_ptr())

    def step(record=False):
        coords, N, size = coords0, N0, size0
        x, rb, parent, handles = x0, None, None, []
        for j, L in enumerate(wl.layers):
            _, _, fp, spp, kind, flags, fwd, wp, bp = largs[j]
            h = rb if L.kind == "vsc" else None
            if h is None:
                h = ctypes.c_void_p()
                if chain and parent is not None:
                    _lib.check(lib.spconv_build_rulebook_on(parent, kind, fp, spp, flags, sp,
                                                            ctypes.byref(h)), "build on")
                else:
                    _lib.check(lib.spconv_build_rulebook(kind, D, coords, N, size.ctypes.data,
                                                         fp, spp, flags, sp,
                                                         ctypes.byref(h)), "build")
                handles.append(h)
            y = torch.empty((rows_out(h), L.c_out), dtype=tdt, device=dev)
            _lib.check(fwd(h, dt_code, ctypes.c_void_p(x.data_ptr()), wp, bp,
                           dt_code, ctypes.c_void_p(y.data_ptr()), L.c_in, L.c_out, sp),
                       "forward")
            if L.kind == "vsc":
                rb = h
            else:
                rb, parent = None, h
                if not chain:
                    osz = np.zeros(D, np.int32)
                    _lib.check(lib.spconv_rulebook_query(h, None, None, None, osz.ctypes.data,
                                                         None), "query")
                    oc = ctypes.c_void_p()
                    _lib.check(lib.spconv_rulebook_out_coords(h, ctypes.byref(oc)),
                               "out coords")
                    coords, N, size = oc, y.shape[0], osz
            if record:
                n_in, n_out = ctypes.c_int64(), ctypes.c_int64()
                off = np.zeros(L.f ** wl.d + 1, np.int64)
                _lib.check(lib.spconv_rulebook_query(h, ctypes.byref(n_in), ctypes.byref(n_out),
                                                     None, None, off.ctypes.data), "query")
                info.append({"layer": j, "kind": L.kind, "n_in": n_in.value,
                             "n_out": n_out.value, "c_in": L.c_in, "c_out": L.c_out,
                             "sum_k": int(off[-1])})
            x = y
        for h in handles:
            lib.spconv_rulebook_destroy(h)
        return x

    step(record=True)                     # sizes and pair counts (untimed)
    for _ in range(a.warmup):
        step()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    host = 0.0
    for _ in range(a.steps):
        h0 = time.perf_counter()
        step()
        host += time.perf_counter() - h0
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / a.steps
    flops = sum(2.0 * r["sum_k"] * r["c_in"] * r["c_out"] for r in info)
    print(json.dumps({
        "metric": "layer-stack forward active input sites/sec (all builds + forwards)",
        "value": N0 / (ms * 1e-3), "unit": "active sites/s", "n_gpus": 1, "steps": a.steps,
        "warmup": a.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": wl.dtype, "data": "synthetic",
        "config": {"workload": wl.name, "variant": a.variant, "batch": wl.batch,
                   "grid": wl.size, "active_sites": N0, "layers": info,
                   "builds": "chained on device counts" if chain else "host waits per SC"},
        "knobs": knobs(),
        "effective_tflops": flops / (ms * 1e-3) / 1e12,
        "host_enqueue_ms_per_step": host * 1e3 / a.steps,
        "bytes_features": int(sum(r["n_in"] * r["c_in"] * esz + r["n_out"] * r["c_out"] * esz
                                  for r in info))}), flush=True)


def run_ops(a, torch, dev, spc, inputs):
    """Pooling, DC, gradients and the fused block epilogue on the workloads
    they belong to, one JSON line each: the level-0 sites of the 4 x 256^3
    encoder (2^3 stride-2 SC: pooling, DC, the SC gradients) and the
    8 x 128^3 headline VSC layer (its input and weight gradients, and its
    forward with batch-norm affine + residual + ReLU fused).  Each line gives the mean time per call from
    HIP events on the stream the library runs on, and achieved / peak for the
    bound that applies (algorithmic bytes or FLOPs per call)."""
    stream = torch.cuda.current_stream()

    def timed(fn):
        for _ in range(a.warmup):
            fn()
        torch.cuda.synchronize()
        e = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        e[0].record(stream)
        for _ in range(a.steps):
            fn()
        e[1].record(stream)
        torch.cuda.synchronize()
        return e[0].elapsed_time(e[1]) / a.steps

    def feats(n, c, seed):
        f = inputs.normal_f32((n, c), seed=seed)
        return torch.from_numpy(inputs.to_bf16_bits(f).view(np.int16)).view(torch.bfloat16).to(dev)

    def weights(K, ci, co, seed):
        f = inputs.normal_f32((K, ci, co), std=1.0 / np.sqrt(K * ci), seed=seed)
        return torch.from_numpy(inputs.to_bf16_bits(f).view(np.int16)).view(torch.bfloat16).to(dev)

    def emit(op, workload, ms, bound, achieved, unit, peak, extra):
        print(json.dumps({"op": op, "workload": workload, "ms_per_call": ms,
                          "calls": a.steps, "dtype": "bf16",
                          "roofline": {"bound": bound, "achieved": achieved, "peak": peak,
                                       "unit": unit, "frac": achieved / peak},
                          **extra}), flush=True)

    # ---- encoder level 0: 2^3 stride-2 SC on 4 x 256^3 surfaces
    wl = inputs.make_workload("surf256x4_unet_enc_bf16", variant=a.variant)
    ct = torch.from_numpy(np.ascontiguousarray(wl.coords)).to(dev)
    n_in = len(wl.coords)
    f2 = [1, 2, 2, 2]
    rb = spc.build_rulebook(spc.SC, ct, wl.spatial_size, f2, f2, transpose=True)
    n_out, K = rb.n_out, rb.K
    sum_k = int(rb.pair_off[-1])
    C = 32
    x = feats(n_in, C, 21)
    y = torch.empty((n_out, C), dtype=torch.bfloat16, device=dev)
    for mode, name in ((spc.POOL_MAX, "max_pool_2x2x2_s2"), (spc.POOL_AVG, "avg_pool_2x2x2_s2")):
        ms = timed(lambda: spc.pool_forward(rb, x, mode, out=y))
        nbytes = n_in * C * 2 + n_out * C * 2 + 4 * K * n_out
        emit(name, "surf256x4 level 0", ms, "hbm", nbytes / (ms * 1e-3) / 1e9, "GB/s",
             PEAKS["hbm"], {"n_in": n_in, "n_out": n_out, "C": C, "algorithmic_bytes": nbytes})
    # DC 2^3 stride 2 (decoder upsampling, 64 -> 32 planes), SC input gradient
    ci, co = 64, 32
    xd = feats(n_out, ci, 22)
    wd = weights(K, ci, co, 23)
    yd = torch.empty((n_in, co), dtype=torch.bfloat16, device=dev)
    ms = timed(lambda: spc.dc_forward(rb, xd, wd, out=yd))
    fl = 2.0 * sum_k * ci * co
    # f = s: every output row takes one input row through one W^i (37 FLOP per
    # byte at 64 -> 32 planes, far below the matrix-core ridge): HBM-bound.
    # Algorithmic bytes: inputs once, outputs once, the two pair columns, W.
    dc_bytes = n_out * ci * 2 + n_in * co * 2 + 8 * sum_k + K * ci * co * 2
    emit("dc_2x2x2_s2_c64_c32", "surf256x4 level 0", ms, "hbm", dc_bytes / (ms * 1e-3) / 1e9,
         "GB/s", PEAKS["hbm"], {"n_in": n_out, "n_out": n_in, "sum_k": sum_k,
                                "algorithmic_bytes": dc_bytes,
                                "effective_tflops": fl / (ms * 1e-3) / 1e12})
    wsc = weights(K, co, ci, 24)                 # SC(32 -> 64) weights
    dysc = feats(n_out, ci, 25)
    dxsc = torch.empty((n_in, co), dtype=torch.bfloat16, device=dev)
    ms = timed(lambda: spc.backward_data(rb, spc.OP_SC, dysc, wsc, out=dxsc))
    emit("sc_input_grad_2x2x2_s2_c32_c64", "surf256x4 level 0", ms, "hbm",
         dc_bytes / (ms * 1e-3) / 1e9, "GB/s", PEAKS["hbm"],
         {"sum_k": sum_k, "algorithmic_bytes": dc_bytes,
          "effective_tflops": fl / (ms * 1e-3) / 1e12})
    xsc = feats(n_in, co, 26)
    ms = timed(lambda: spc.backward_weight(rb, spc.OP_SC, xsc, dysc, co, ci))
    emit("sc_weight_grad_2x2x2_s2_c32_c64", "surf256x4 level 0", ms, "mfma",
         fl / (ms * 1e-3) / 1e12, "TFLOP/s", PEAKS["bf16"], {"sum_k": sum_k})
    rb.close()
    del x, y, xd, yd, dysc, dxsc, xsc

    # ---- headline VSC layer: input and weight gradients
    wl = inputs.make_workload("surf128x8_vsc3_c64_bf16", variant=a.variant)
    ct = torch.from_numpy(np.ascontiguousarray(wl.coords)).to(dev)
    N = len(wl.coords)
    rb = spc.build_rulebook(spc.VSC, ct, wl.spatial_size, [1, 3, 3, 3])
    sum_k = int(rb.pair_off[-1])
    C = 64
    w = weights(27, C, C, 31)
    dy = feats(N, C, 32)
    xv = feats(N, C, 33)
    dx = torch.empty((N, C), dtype=torch.bfloat16, device=dev)
    fl = 2.0 * sum_k * C * C
    ms = timed(lambda: spc.backward_data(rb, spc.OP_VSC, dy, w, out=dx))
    emit("vsc_input_grad_3x3x3_c64", "surf128x8", ms, "mfma", fl / (ms * 1e-3) / 1e12,
         "TFLOP/s", PEAKS["bf16"], {"active_sites": N, "sum_k": sum_k})
    ms = timed(lambda: spc.backward_weight(rb, spc.OP_VSC, xv, dy, C, C))
    emit("vsc_weight_grad_3x3x3_c64", "surf128x8", ms, "mfma", fl / (ms * 1e-3) / 1e12,
         "TFLOP/s", PEAKS["bf16"], {"active_sites": N, "sum_k": sum_k})

    # forward with the block epilogue (batch-norm affine, residual, ReLU) fused,
    # against the plain forward and against the forward followed by the same
    # epilogue as separate torch passes
    scale = torch.from_numpy(inputs.normal_f32((C,), seed=34)).to(dev)
    shift = torch.from_numpy(inputs.normal_f32((C,), std=0.5, seed=35)).to(dev)
    res = feats(N, C, 36)
    y = torch.empty((N, C), dtype=torch.bfloat16, device=dev)
    ms = timed(lambda: spc.forward_fused(rb, xv, w, scale, shift, res, True, out=y))
    ms_plain = timed(lambda: spc.vsc_forward(rb, xv, w, shift, out=y))

    def separate():
        spc.vsc_forward(rb, xv, w, None, out=y)
        y.copy_(torch.relu(torch.addcmul(shift, y.float(), scale) + res.float()))
    ms_sep = timed(separate)
    emit("vsc_fused_bn_res_relu_3x3x3_c64", "surf128x8", ms, "mfma", fl / (ms * 1e-3) / 1e12,
         "TFLOP/s", PEAKS["bf16"],
         {"active_sites": N, "sum_k": sum_k, "plain_forward_ms": ms_plain,
          "forward_then_torch_epilogue_ms": ms_sep})
    rb.close()

    # ---- the low-channel path: one input plane (pen strokes), VSC 3x3,
    # 1 -> 32 fp32 on 1,024 grids of 64^2 (the one-plane kernel k_fwd_lowc;
    # HBM-bound: features, gather map and output each move once)
    coords = inputs.pen_strokes(1024, 64, seed=31, target=400)
    n = len(coords)
    ct = torch.from_numpy(coords).to(dev)
    rb = spc.build_rulebook(spc.VSC, ct, [1024, 64, 64], [1, 3, 3])
    K, sum_k = rb.K, int(rb.pair_off[-1])
    ci, co = 1, 32
    x1 = torch.from_numpy(inputs.normal_f32((n, ci), seed=32)).to(dev)
    w1 = torch.from_numpy(inputs.normal_f32((K, ci, co), std=1.0 / 3, seed=33)).to(dev)
    b1 = torch.from_numpy(inputs.normal_f32((co,), std=0.1, seed=34)).to(dev)
    y1 = torch.empty((n, co), dtype=torch.float32, device=dev)
    ms = timed(lambda: spc.vsc_forward(rb, x1, w1, b1, out=y1))
    nbytes = n * ci * 4 + n * co * 4 + 4 * K * n + K * ci * co * 4 + 4 * co
    emit("vsc_lowc_3x3_c1_c32_f32", "pen 1024 x 64^2", ms, "hbm", nbytes / (ms * 1e-3) / 1e9,
         "GB/s", PEAKS["hbm"], {"dtype": "f32", "kernel": "k_fwd_lowc", "active_sites": n,
                                "sum_k": sum_k, "algorithmic_bytes": nbytes})
    rb.close()


if __name__ == "__main__":
    main()
