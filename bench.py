#!/usr/bin/env python3
"""Benchmark of the CNN forward contraction on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
                    [--out-dtype fp32|bf16] [--eager] [--no-cpu-baseline] [--no-configs]
                    [--plan KERNEL:TK:TP:TC] [--copy-bytes N] [--cold]

A step is one forward convolution Out = conv(In, Ker) of the workload
(default: the largest, the strided 3x3 layer Nb=64, Nc=128, Nk=256, 28x28
outputs, stride 2, bf16 In and Ker, fp32 accumulation and fp32 Out) through
the C ABI, on inputs already resident in device memory, with the plan
cnn_plan_find measures to be fastest (cnn_fwd runs it; cnn_fwd_plan_ws with
a workspace allocated beforehand if that plan needs one).  The K timed
steps are captured into one HIP graph and replayed, so host launch cost
does not pace a kernel of a few microseconds (--eager launches each step
from the host instead).  Before them, W untimed steps run and then further
untimed replays until at least one second has passed, so that the timed
steps see the GPU's sustained clocks ("warmup" in the JSON line is W,
"untimed_steps" all the untimed steps that ran).  The timed region is
bracketed by torch.cuda.synchronize().

Prints ONE JSON line: the metric (conv TFLOP/s = 2 Nb Nk Nc Nr Ns Nw Nh /
seconds per step), the roofline of the convolution kernel (HIP events on
the stream it runs on, algorithmic bytes or flops per launch; HBM-bound
kernels also against the bandwidth of a 256 MiB device copy measured in
the same run, "frac_of_copy"), the fp64
CPU oracle timed on this host as a baseline, and under "configs" the same
figures for every workload (each with its own oracle baseline on a bounded
sample).
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

PEAK_TFLOPS = {"bf16": 2516.6, "f32": 157.3}   # dense MFMA, MI355X datasheet
PEAK_HBM_GBS = 8000.0                           # HBM3E, MI355X datasheet
DEFAULT_WORKLOAD = "conv3x3_s2_b64"


# The HBM counters are taken per workload on the kernel of a fixed plan; its
# code comes from its family's source, the shared headers and the launch
# path, not from the other families' sources or the plan selector.
FAMILY_SOURCE = {"rows": "k_rows.hip", "srows": "k_srows.hip", "gemm1": "k_gemm1.hip",
                 "smallc": "k_smallc.hip", "igemm": "k_igemm.hip",
                 "splitc": ("k_igemm.hip", "k_cslice.hip"),
                 "pointwise": "k_igemm2.hip", "igemm_pipe": "k_igemm2.hip",
                 "igemm_rawk": "k_igemm2.hip", "igemm_dma": "k_igemm3.hip",
                 "igemm_wide": "k_igemm4.hip", "direct": "k_direct.hip"}
NOT_COUNTED = ("cnn_select.cpp",)


def kernel_source_hash(family: str) -> str:
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2105_13480_amd", "csrc")
    for f in sorted(os.listdir(csrc)):
        own = FAMILY_SOURCE.get(family, ())
        own = (own,) if isinstance(own, str) else own
        if (f.startswith("k_") and f not in own) or f in NOT_COUNTED:
            continue
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(f.encode() + b"\0" + fh.read())
    with open(os.path.join(ROOT, "include", "cnn.h"), "rb") as fh:
        h.update(b"cnn.h\0" + fh.read())
    return h.hexdigest()[:16]


def measured_traffic(workload: str, mode: str, family: str, variant: int):
    """HBM bytes per launch from the committed rocprofv3 counter summary,
    if it was taken on the same instantiation and the current sources of
    the plan's kernel (else None)."""
    path = os.path.join(ROOT, "profiles", "hbm_traffic.json")
    try:
        with open(path) as fh:
            data = json.load(fh)
    except (OSError, ValueError):
        return None
    rec = data.get(f"{workload}/{mode}")
    if not rec or rec.get("source_hash") != kernel_source_hash(family) or \
            rec.get("family") != family or rec.get("variant") != variant:
        return None
    return rec.get("hbm_bytes_per_launch")


KERNELS = {"direct": 1, "igemm": 2, "pointwise": 3, "smallc": 4, "igemm_pipe": 5,
           "igemm_dma": 6, "igemm_wide": 7, "igemm_rawk": 8, "rows": 10, "gemm1": 11,
           "srows": 12, "splitc": 13}


def forced_plan(spec: str, w, mode: str):
    """Plan for --plan KERNEL[:TK:TP:TC] (e.g. igemm_pipe:64:256:16)."""
    from paper_2105_13480_amd import cnn
    parts = spec.split(":")
    kern = KERNELS[parts[0]]
    tk, tp, tc = (int(x) for x in parts[1:4]) if len(parts) >= 4 else (0, 0, 0)
    prob = cnn.problem(*w.dims())
    if len(parts) < 5:
        return cnn.plan_tiles(prob, cnn.DTYPES[mode], kern, tk, tp, tc)
    # with a variant, TP may be the plan's (balanced) tile: find the variant's
    # largest tile among the instantiated sizes
    want = int(parts[4])
    for tp_max in [tp] + [32 * m for m in range(1, 17)]:
        try:
            pl = cnn.plan_tiles(prob, cnn.DTYPES[mode], kern, tk, tp_max, tc)
        except cnn.CnnError:
            continue
        if pl.variant == want:
            return pl
    # several instantiations may implement one tiling: the candidate itself
    for pl in cnn.plan_candidates(prob, cnn.DTYPES[mode]):
        if pl.kernel == kern and pl.variant == want and (tp in (0, pl.tp)):
            return pl
    raise SystemExit(f"--plan {spec}: no tiling resolves to variant {want}")


def copy_calibration(nbytes: int, steps: int):
    """Device-to-device copy of a known size (torch), for scaling the HBM
    byte counters of rocprofv3 (FETCH_SIZE / WRITE_SIZE)."""
    import torch
    n = nbytes // 4
    a = torch.ones(n, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    t_w = time.perf_counter()
    while time.perf_counter() - t_w < 0.5:  # sustained clocks
        for _ in range(8):
            b.copy_(a)
        torch.cuda.synchronize()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    ev0.record()
    for _ in range(steps):
        b.copy_(a)
    ev1.record()
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / steps
    print(json.dumps({"copy_bytes": n * 4, "ms_per_copy": round(ms, 5),
                      "GB_per_s_read_plus_write": round(2 * n * 4 / (ms * 1e-3) / 1e9, 1)}),
          flush=True)


def copy_gbs(nbytes: int = 1 << 28, steps: int = 20) -> float:
    """HBM bandwidth of a large device copy (bytes read plus written per
    second, HIP events, after half a second of untimed copies): the
    attainable side of the roofline beside the 8 TB/s datasheet figure."""
    import torch
    a = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    t_w = time.perf_counter()
    while time.perf_counter() - t_w < 0.5:
        for _ in range(8):
            b.copy_(a)
        torch.cuda.synchronize()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    ev0.record()
    for _ in range(steps):
        b.copy_(a)
    ev1.record()
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / steps
    del a, b
    return 2.0 * nbytes / (ms * 1e-3) / 1e9


def _counter_medians(csv_dir: str, counter: str):
    """{kernel name: (dispatches, median value in KiB)} of one rocprofv3
    --pmc pass (its *counter_collection.csv)."""
    import csv
    import glob
    import statistics
    vals = {}
    for path in glob.glob(os.path.join(csv_dir, "**", "*counter_collection.csv"), recursive=True):
        with open(path) as fh:
            for r in csv.DictReader(fh):
                if r["Counter_Name"] == counter:
                    vals.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]))
    return {k: (len(v), statistics.median(v)) for k, v in vals.items()}


def summarize_counters(pmc_dir: str, workload: str, mode: str, copy_bytes: int, commands,
                       family: str, variant: int):
    """Write profiles/hbm_traffic.json from four rocprofv3 --pmc passes under
    pmc_dir: conv_fetch / conv_write (FETCH_SIZE / WRITE_SIZE of this bench
    with a forced plan) and copy_fetch / copy_write (the same counters on a
    device copy of copy_bytes, whose true traffic is known).  Counter KiB are
    scaled by true / counted bytes of the copy."""
    cf = _counter_medians(os.path.join(pmc_dir, "copy_fetch"), "FETCH_SIZE")
    cw = _counter_medians(os.path.join(pmc_dir, "copy_write"), "WRITE_SIZE")
    kf = _counter_medians(os.path.join(pmc_dir, "conv_fetch"), "FETCH_SIZE")
    kw = _counter_medians(os.path.join(pmc_dir, "conv_write"), "WRITE_SIZE")
    copy_f = max((v for k, v in cf.items() if "copyBuffer" in k), key=lambda x: x[0])[1]
    copy_w = max((v for k, v in cw.items() if "copyBuffer" in k), key=lambda x: x[0])[1]
    f_scale = copy_bytes / (copy_f * 1024.0)
    w_scale = copy_bytes / (copy_w * 1024.0)
    conv = [k for k in kf if "cnnlib::conv_" in k]
    name = max(conv, key=lambda k: kf[k][0])
    fetch = kf[name][1] * 1024.0 * f_scale
    write = kw[name][1] * 1024.0 * w_scale
    path = os.path.join(ROOT, "profiles", "hbm_traffic.json")
    try:
        with open(path) as fh:
            data = json.load(fh)
    except (OSError, ValueError):
        data = {}
    data[f"{workload}/{mode}"] = {
        "kernel": name, "dispatches": kf[name][0],
        "fetch_kib_median": kf[name][1], "write_kib_median": kw[name][1],
        "copy_bytes": copy_bytes, "copy_fetch_kib": copy_f, "copy_write_kib": copy_w,
        "fetch_scale": round(f_scale, 4), "write_scale": round(w_scale, 4),
        "hbm_fetch_bytes": round(fetch), "hbm_write_bytes": round(write),
        "hbm_bytes_per_launch": round(fetch + write),
        "family": family, "variant": variant, "source_hash": kernel_source_hash(family),
        "commands": commands}
    with open(path, "w") as fh:
        json.dump(data, fh, indent=1, sort_keys=True)
    print(json.dumps(data[f"{workload}/{mode}"]))


def _device_inputs(w, mode):
    import numpy as np
    import torch

    from paper_2105_13480_amd import inputs

    In, Ker = inputs.make_inputs(w)
    if In.dtype == np.uint16:
        dIn = torch.from_numpy(In.view(np.int16)).view(torch.bfloat16).cuda()
        dKer = torch.from_numpy(Ker.view(np.int16)).view(torch.bfloat16).cuda()
    else:
        dIn, dKer = torch.from_numpy(In).cuda(), torch.from_numpy(Ker).cuda()
    out_dt = torch.bfloat16 if mode == "bf16_obf16" else torch.float32
    dOut = torch.empty((w.Nb, w.Nk, w.Nw, w.Nh), dtype=out_dt, device="cuda")
    return dIn, dKer, dOut


def time_workload(w, mode: str, steps: int, warmup: int, eager: bool, plan_spec: str = "",
                  find: bool = True):
    """(ms per step by the host clock, kernel ms per step by HIP events on the
    launching stream, the plan, untimed steps run)."""
    import torch

    from paper_2105_13480_amd import cnn

    dIn, dKer, dOut = _device_inputs(w, mode)
    cap_stream = torch.cuda.Stream()
    if plan_spec:
        plan = forced_plan(plan_spec, w, mode)
        selection = "forced"
    elif find:  # time every candidate once, before the timed region
        plan, _ = cnn.plan_find(dIn, dKer, dOut, w.sw, w.sh, stream=cap_stream)
        torch.cuda.synchronize()
        selection = "find"
    else:  # the selector's own choice
        plan = cnn.plan(cnn.problem(*w.dims()), cnn.DTYPES[mode])
        selection = "model"
    ws = None
    if plan.ws_bytes > 0:  # allocated here, before the timed region
        ws = torch.empty(plan.ws_bytes, dtype=torch.uint8, device="cuda")

        def step():
            cnn.fwd_plan_ws(dIn, dKer, dOut, plan, ws, w.sw, w.sh)
    elif selection != "find":
        def step():
            cnn.fwd_plan(dIn, dKer, dOut, plan, w.sw, w.sh)
    else:
        # cnn_fwd runs the cached plan: the fastest workspace-free candidate
        # of the search (the one returned here), or the model's choice
        assert cnn.plan_lookup(cnn.problem(*w.dims()), cnn.DTYPES[mode]).variant == plan.variant

        def step():
            cnn.fwd(dIn, dKer, dOut, w.sw, w.sh)

    with torch.cuda.stream(cap_stream):
        for _ in range(2):
            step()
    torch.cuda.synchronize()
    done = 2

    graph = None
    if not eager:
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=cap_stream):
            for _ in range(steps):
                step()
    # Untimed: at least `warmup` steps (whole replays of the timed graph),
    # and at least one second of them, so that the GPU clocks have reached
    # their sustained state before the timed region.
    t_w = time.perf_counter()
    while time.perf_counter() - t_w < 1.0 or done < warmup:
        if graph is not None:
            graph.replay()
            done += steps
        else:
            step()
            done += 1
        if done % (10 * steps) < (steps if graph is not None else 1):
            torch.cuda.synchronize()  # keep the host within a few replays of the GPU
    torch.cuda.synchronize()

    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record()
    if graph is not None:
        graph.replay()
    else:
        for _ in range(steps):
            step()
    ev1.record()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_per_step = (t1 - t0) * 1e3 / steps
    kernel_ms = ev0.elapsed_time(ev1) / steps
    del graph
    plan.selection = selection
    return ms_per_step, kernel_ms, plan, done


def roofline(w, mode: str, plan, kms: float):
    """Roofline of the step's kernels from their event time: HBM-bound below
    the ridge (algorithmic bytes per launch over 8 TB/s), else MFMA-bound."""
    prec = "f32" if mode == "f32" else "bf16"
    alg_bytes = plan.compulsory_bytes
    ai = w.flops / alg_bytes
    ridge = PEAK_TFLOPS[prec] * 1e12 / (PEAK_HBM_GBS * 1e9)
    k_tflops = w.flops / (kms * 1e-3) / 1e12
    if ai < ridge:
        achieved = alg_bytes / (kms * 1e-3) / 1e9
        return {"bound": "hbm", "achieved": round(achieved, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBS, 4)}
    return {"bound": "mfma", "achieved": round(k_tflops, 2), "peak": PEAK_TFLOPS[prec],
            "unit": "TFLOP/s", "frac": round(k_tflops / PEAK_TFLOPS[prec], 4)}


def cold_time(w, mode: str, reps: int = 30):
    """Median time of one cnn_fwd call (HIP events around it on its stream)
    with cold caches: a 1 GiB scratch tensor is written before each call,
    outside the timed region, which evicts In, Ker and Out from the L2s and
    the 256 MB MALL.  Also the median of single calls without the flush
    (same timing method), for comparison.  Returns (cold_ms, warm_ms)."""
    import statistics

    import numpy as np
    import torch

    from paper_2105_13480_amd import cnn, inputs

    In, Ker = inputs.make_inputs(w)
    if In.dtype == np.uint16:
        dIn = torch.from_numpy(In.view(np.int16)).view(torch.bfloat16).cuda()
        dKer = torch.from_numpy(Ker.view(np.int16)).view(torch.bfloat16).cuda()
    else:
        dIn, dKer = torch.from_numpy(In).cuda(), torch.from_numpy(Ker).cuda()
    out_dt = torch.bfloat16 if mode == "bf16_obf16" else torch.float32
    dOut = torch.empty((w.Nb, w.Nk, w.Nw, w.Nh), dtype=out_dt, device="cuda")
    scratch = torch.empty(1 << 28, dtype=torch.float32, device="cuda")
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    cnn.fwd(dIn, dKer, dOut, w.sw, w.sh)  # the plan cnn_plan_find cached
    cold, warm = [], []
    for flush, acc in ((True, cold), (False, warm)):
        for _ in range(reps):
            if flush:
                scratch.fill_(1.0)
            torch.cuda.synchronize()
            e0.record()
            cnn.fwd(dIn, dKer, dOut, w.sw, w.sh)
            e1.record()
            torch.cuda.synchronize()
            acc.append(e0.elapsed_time(e1))
    del scratch
    return statistics.median(cold), statistics.median(warm)


def cpu_baseline(w, budget_s: float = 10.0, threads: int = 0):
    """fp64 oracle on this host's cores (or `threads` of them): the whole
    workload, or a prefix of its batch for large ones, repeated until about
    `budget_s` seconds."""
    import oracle
    from paper_2105_13480_amd import inputs

    In, Ker = inputs.make_inputs(w)
    prev = oracle.set_threads(threads) if threads else None
    try:
        per_image = w.flops / w.Nb
        cores = oracle.threads()
        nb = w.Nb
        # keep one pass under ~1/3 of the budget at ~4 GFLOP/s per thread
        while nb > 1 and per_image * nb > budget_s / 3 * 4e9 * cores:
            nb //= 2
        sub = In[:nb]
        oracle.conv(sub, Ker[:1], w.sw, w.sh)  # load + warm
        passes, t0 = 0, time.perf_counter()
        while True:
            oracle.conv(sub, Ker, w.sw, w.sh)
            passes += 1
            el = time.perf_counter() - t0
            if el >= budget_s or passes >= 50:
                break
    finally:
        if prev:
            oracle.set_threads(prev)
    flops = per_image * nb * passes
    return {"value": round(flops / el / 1e12, 6), "unit": "TFLOP/s", "cores": cores,
            "kind": "oracle",
            "sample": f"{nb} of {w.Nb} images of {w.name}, full Nk/Nc/spatial extent, "
                      f"{passes} passes in {el:.1f} s (fp64 seven-loop direct convolution)"}


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=0,
                    help="untimed steps before the timed ones (at least one second of untimed "
                         "steps runs in any case, for sustained GPU clocks)")
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--out-dtype", choices=["fp32", "bf16"], default="fp32")
    ap.add_argument("--eager", action="store_true")
    ap.add_argument("--cold", action="store_true",
                    help="also time single calls with cold caches (a 1 GiB write before each)")
    ap.add_argument("--model-plan", action="store_true",
                    help="use the selector's model plan instead of timing the candidates")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-configs", action="store_true",
                    help="time the headline workload only (no per-workload list)")
    ap.add_argument("--all", action="store_true",
                    help="per-workload list with both output dtypes (table on stderr)")
    ap.add_argument("--plan", default="",
                    help="force a tiling, KERNEL[:TK:TP:TC[:VARIANT]], KERNEL one of "
                         + "/".join(KERNELS))
    ap.add_argument("--copy-bytes", type=int, default=0,
                    help="only time a device copy of this many bytes (counter calibration)")
    ap.add_argument("--summarize-counters", default="",
                    help="write profiles/hbm_traffic.json from rocprofv3 --pmc passes in this "
                         "directory (conv_fetch, conv_write, copy_fetch, copy_write); no GPU")
    ap.add_argument("--commands", default="",
                    help="with --summarize-counters: the commands that made the passes")
    args = ap.parse_args()
    if args.steps < 1:
        raise SystemExit("--steps must be at least 1")
    if args.warmup < 0:
        raise SystemExit("--warmup must be at least 0")

    if args.summarize_counters:
        from paper_2105_13480_amd import inputs as _inputs
        w = _inputs.BY_NAME[args.workload]
        mode = "f32" if w.dtype == "f32" else ("bf16" if args.out_dtype == "fp32" else "bf16_obf16")
        parts = args.plan.split(":")
        if len(parts) < 5:
            raise SystemExit("--summarize-counters needs --plan KERNEL:TK:TP:TC:VARIANT "
                             "(the plan the passes ran)")
        summarize_counters(args.summarize_counters, w.name, mode, args.copy_bytes,
                           [c for c in args.commands.split(";;") if c], parts[0], int(parts[4]))
        return

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py: this library runs on one GPU only; the contraction shards along the "
              "batch with no exchange, but no multi-GPU path is implemented (use --gpus 1)",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2105_13480_amd import cnn, inputs

    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        sys.exit(1)
    cnn.lib()  # fail loudly if the HIP library is missing
    if args.copy_bytes:
        copy_calibration(args.copy_bytes, args.steps)
        return

    def mode_of(w, out_dtype):
        return "f32" if w.dtype == "f32" else ("bf16" if out_dtype == "fp32" else "bf16_obf16")

    def plan_fields(pl):
        d = pl.as_dict()
        out = {k: d[k] for k in ("kernel", "variant", "tk", "tp", "tc", "grid")}
        if pl.kernel == cnn.K_SPLITC:
            out["kc"] = pl.kc
        out["workspace_bytes"] = pl.ws_bytes
        out["model_us"] = round(pl.model_us, 2)
        return out

    w = inputs.BY_NAME[args.workload]
    mode = mode_of(w, args.out_dtype)
    print(f"bench: {w.name} {mode}: plan search and {args.steps} timed steps", file=sys.stderr,
          flush=True)
    ms, kms, plan, untimed = time_workload(w, mode, args.steps, args.warmup, args.eager,
                                           args.plan, find=not args.model_plan)
    model = cnn.plan(cnn.problem(*w.dims()), cnn.DTYPES[mode])

    prec = "f32" if mode == "f32" else "bf16"
    tflops = w.flops / (ms * 1e-3) / 1e12
    roof = roofline(w, mode, plan, kms)
    roof["traffic"] = measured_traffic(w.name, mode, plan.as_dict()["kernel"], plan.variant)
    try:  # Eq. (3) at the XCD / L2 level for the timed plan (a prediction)
        roof["model_hbm_bytes"] = round(sum(cnn.hbm_bytes(plan, 8, 4 << 20)))
    except cnn.CnnError:
        roof["model_hbm_bytes"] = None
    roof["algorithmic_bytes_per_launch"] = plan.compulsory_bytes
    roof["eq1_bytes_per_launch"] = plan.eq1_bytes
    roof["kernel_ms"] = round(kms, 5)
    roof["pct_mfma_peak"] = round(100.0 * w.flops / (kms * 1e-3) / 1e12 / PEAK_TFLOPS[prec], 2)
    # the same algorithmic rate against the measured copy bandwidth
    copy_bw = copy_gbs()
    roof["copy_gbs"] = round(copy_bw, 1)
    if roof["bound"] == "hbm":
        roof["frac_of_copy"] = round(roof["achieved"] / copy_bw, 4)

    line = {
        "metric": "conv TFLOP/s (2*Nb*Nk*Nc*Nr*Ns*Nw*Nh/s) + % MFMA peak, 1 MI355X",
        "value": round(tflops, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "untimed_steps": untimed,
        "ms_per_step": round(ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": prec,
        "data": "synthetic (seeded uniform In, He-normal Ker)",
        "config": {"workload": w.name, "Nb": w.Nb, "Nc": w.Nc, "Nk": w.Nk, "Nw": w.Nw,
                   "Nh": w.Nh, "Nr": w.Nr, "Ns": w.Ns, "sw": w.sw, "sh": w.sh,
                   "in_dtype": w.dtype, "acc_dtype": "f32",
                   "out_dtype": "bf16" if mode == "bf16_obf16" else "f32",
                   "launch": "eager" if args.eager else "hipgraph",
                   "plan": plan_fields(plan),
                   "plan_selection": plan.selection,
                   "model_plan": plan_fields(model)},
        "pct_mfma_peak": round(100.0 * tflops / PEAK_TFLOPS[prec], 2),
        "roofline": roof,
    }
    if args.cold:
        c_ms, w_ms = cold_time(w, mode)
        line["cold"] = {"ms_median": round(c_ms, 5), "ms_warm_single": round(w_ms, 5),
                        "reps": 30, "flush_bytes": 1 << 30,
                        "note": "one cnn_fwd call between HIP events; caches flushed by a "
                                "1 GiB write before each call (warm: no flush)"}
    if not args.no_cpu_baseline:
        print("bench: oracle baseline on the host's cores", file=sys.stderr, flush=True)
        line["cpu_baseline"] = cpu_baseline(w, budget_s=10.0)

    if not args.no_configs and not args.plan:
        configs = []
        out_dtypes = ["fp32", "bf16"] if args.all else [args.out_dtype]
        for ww in inputs.WORKLOADS:
            for od in out_dtypes:
                md = mode_of(ww, od)
                if od == "bf16" and md == "f32":
                    continue
                print(f"bench: {ww.name} {md}", file=sys.stderr, flush=True)
                m2, k2, p2, u2 = time_workload(ww, md, min(args.steps, 100), 0, args.eager,
                                               find=not args.model_plan)
                pr = "f32" if md == "f32" else "bf16"
                mdl = cnn.plan(cnn.problem(*ww.dims()), cnn.DTYPES[md])
                rec = {"workload": ww.name, "out_dtype": "bf16" if md == "bf16_obf16" else "f32",
                       "ms": round(k2, 5), "TFLOP_per_s": round(ww.flops / (k2 * 1e-3) / 1e12, 2),
                       "pct_mfma_peak": round(100 * ww.flops / (k2 * 1e-3) / 1e12 / PEAK_TFLOPS[pr], 2),
                       "roofline": roofline(ww, md, p2, k2),
                       "plan": plan_fields(p2), "model_plan": plan_fields(mdl),
                       "model_plan_ms_ratio": None}
                rec["roofline"]["traffic"] = measured_traffic(ww.name, md, p2.as_dict()["kernel"],
                                                              p2.variant)
                rec["roofline"]["model_hbm_bytes"] = round(p2.hbm_bytes)
                if rec["roofline"]["bound"] == "hbm":
                    rec["roofline"]["frac_of_copy"] = round(rec["roofline"]["achieved"] / copy_bw, 4)
                if (mdl.kernel, mdl.variant, mdl.tp, mdl.kc) != (p2.kernel, p2.variant, p2.tp, p2.kc):
                    # the model's own choice, timed the same way
                    _, k3, _, _ = time_workload(ww, md, min(args.steps, 100), 0, args.eager,
                                                find=False)
                    rec["model_plan_ms_ratio"] = round(k3 / k2, 3)
                else:
                    rec["model_plan_ms_ratio"] = 1.0
                if not args.no_cpu_baseline and od == out_dtypes[0]:
                    cb = cpu_baseline(ww, budget_s=2.0)
                    rec["cpu_baseline"] = {k: cb[k] for k in ("value", "unit", "cores", "sample")}
                    if ww.name == "tiny3x3_f32":
                        c1 = cpu_baseline(ww, budget_s=2.0, threads=1)
                        rec["cpu_baseline_1thread"] = {k: c1[k] for k in ("value", "unit", "cores", "sample")}
                configs.append(rec)
                print(f"{ww.name:18s} {md:10s} kernel {k2 * 1e3:9.2f} us  "
                      f"{rec['TFLOP_per_s']:8.1f} TF/s  {rec['pct_mfma_peak']:5.1f}% peak  "
                      f"roofline {rec['roofline']['bound']} {rec['roofline']['frac']:.3f}  "
                      f"plan {p2.as_dict()['kernel']} v{p2.variant} tk{p2.tk} tp{p2.tp} tc{p2.tc}"
                      + (f" kc{p2.kc}" if p2.kernel == cnn.K_SPLITC else "")
                      + f"  model/find {rec['model_plan_ms_ratio']}",
                      file=sys.stderr, flush=True)
                if args.cold:
                    c_ms, w_ms = cold_time(ww, md)
                    print(f"{ww.name:18s} {md:10s} single call: cold {c_ms * 1e3:9.2f} us, "
                          f"warm {w_ms * 1e3:9.2f} us", file=sys.stderr, flush=True)
        line["configs"] = configs

    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
