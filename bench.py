"""Benchmark of the OaA FFT convolution layer on one MI355X.

One step = one training step of one layer through the C ABI: forward (kernel
spectra, input block spectra, per-bin contraction over C, inverse transform +
overlap-add + crop), backward-data (gradient window spectra, contraction over
K with the kernel spectra of the same step, inverse + block crop) and
backward-filter (contraction over the batch and all blocks with the block and
window spectra of the same step, inverse + crop). Inputs are seeded synthetic
arrays already resident in HBM when the timed region starts.

Prints ONE JSON line. value = direct-convolution-equivalent TFLOP/s of the
whole step, 3 * 2*B*K*C*M^2*n^2 / (ms per step). A "roofline" object gives
the dominant kernel's achieved rate from HIP events recorded around each of
its launches inside the timed region, and "cpu_baseline" the fp64 oracle
timed on a bounded sample of the same layer on the host cores.
"""

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0        # MI355X HBM3E
FP32_MFMA_PEAK_TFLOPS = 157.3  # MI355X dense fp32 matrix
PROFILE_DIR = os.path.join(ROOT, "profiles")
PARITY_TOL = 2e-5              # max|err| / max|ref| against the fp64 oracle


def stage_work(ly, geo):
    """Algorithmic bytes (HBM) and flops per launch of each stage.

    Contractions: "flops" is the method's own count, 8 real flops per
    complex multiply-add over all F = L(L/2+1) stored bins of every tile,
    8 B P C K F per launch; "flops_exec" is what the matrix-core engine
    executes, 6 real flops per complex multiply-add (Gauss's three real
    products) over the unique_bins(L) bins that are not conjugates of
    others.

    "bound": the roofline a stage is measured against: the matrix cores for
    the tiled contractions of many channels (min(C, K) >= 32), HBM for the
    transforms, the streaming contraction of few channels and the fused
    few-channel kernels (whose algorithmic bytes are their inputs and
    outputs: the input or gradient planes, the spectra they read, the
    planes or partial sums they write)."""
    B, C, K, N, n, M = ly.B, ly.C, ly.K, ly.N, ly.n, ly.M
    F, P, S, L = geo["F"], geo["P"], geo["split"], geo["L"]
    BP = B * P
    cplx = 8
    Fu = (L // 2 + 1) ** 2 + (L // 2 - 1) ** 2
    alg_flops = 8.0 * BP * C * K * F
    exec_flops = 6.0 * BP * C * K * Fu
    # the transforms' outputs count the same unique bins (the others are
    # conjugates that no later stage reads)
    prod = dict(flops=alg_flops, flops_exec=exec_flops, bound="mfma" if min(C, K) >= 32 else "hbm")
    if geo.get("fused"):
        fused = dict(flops=alg_flops, flops_exec=exec_flops, bound="hbm")
        return {
            "w_spectrum": dict(bytes=K * C * n * n * 4 + Fu * C * K * cplx),
            "x_spectrum": dict(bytes=B * C * N * N * 4 + Fu * C * BP * cplx),
            "fwd_inverse": dict(fused, bytes=(Fu * C * BP + Fu * C * K) * cplx + B * K * M * M * 4),
            "bwd_data_product": dict(fused, bytes=B * K * M * M * 4 + Fu * C * K * cplx + B * C * N * N * 4),
            "bwd_filter_product": dict(fused, bytes=B * K * M * M * 4 + Fu * C * BP * cplx + S * Fu * C * K * cplx),
            "bwd_filter_inverse": dict(bytes=S * Fu * C * K * cplx + K * C * n * n * 4),
        }
    return {
        "w_spectrum": dict(bytes=K * C * n * n * 4 + Fu * C * K * cplx),
        "x_spectrum": dict(bytes=B * C * N * N * 4 + Fu * C * BP * cplx),
        "g_spectrum": dict(bytes=B * K * M * M * 4 + Fu * K * BP * cplx),
        "fwd_product": dict(prod, bytes=(Fu * C * K + Fu * C * BP + Fu * K * BP) * cplx),
        "fwd_inverse": dict(bytes=Fu * K * BP * cplx + B * K * M * M * 4),
        "bwd_data_product": dict(prod, bytes=(Fu * C * K + Fu * K * BP + Fu * C * BP) * cplx),
        "bwd_data_inverse": dict(bytes=Fu * C * BP * cplx + B * C * N * N * 4),
        "bwd_filter_product": dict(prod, bytes=(Fu * C * BP + Fu * K * BP + S * Fu * C * K) * cplx),
        "bwd_filter_inverse": dict(bytes=S * Fu * C * K * cplx + K * C * n * n * 4),
    }


def traffic_key(workload, geo, stage):
    method = "/oas" if geo.get("method") else ""
    return f"{workload}@{geo['L']}:{geo['b']}{method}/{stage}"


SHARED_SOURCES = ("oaa_plan.cpp", "oaa_internal.hpp", "tile_common.hpp", "fft_core.hpp", "twiddle.hpp",
                  "buffer_io.hpp")


def source_digest(fname):
    """Digest of a kernel's source file(s) ("a.hip+b.hip" for a stage of two
    kernels) together with the headers they share and the plan code that
    picks their launch shape."""
    h = hashlib.sha256()
    for f in tuple(fname.split("+")) + SHARED_SOURCES:
        h.update(open(os.path.join(ROOT, "paper_1601_06815_amd", "csrc", f), "rb").read())
    return h.hexdigest()[:16]


KERNEL_FILES = (("big_", "k_big_fft.hip"), ("overlap_gather", "k_big_fft.hip"), ("fused_", "k_fused.hip"),
                ("cgemm_", "k_cgemm.hip"), ("narrow_", "k_narrow.hip"), ("irfft2_fold", "k_fold_fft.hip"),
                ("irfft2_overlap", "k_fold_fft.hip"), ("tile_rfft2", "k_tile_fft.hip"),
                ("window_", "k_tile_fft.hip"), ("irfft2_crop", "k_tile_fft.hip"))


def source_for_kernels(kernels):
    """Source file(s) of a stage's kernel(s), "name" or "name+name"."""
    files = []
    for k in kernels.split("+"):
        f = next((f for prefix, f in KERNEL_FILES if k.startswith(prefix)), None)
        if f and f not in files:
            files.append(f)
    return "+".join(files)


def _profile_record(fname, workload, geo, stage):
    """A committed per-stage counter record (profiles/<fname>), or None if
    absent or taken on a different version of the kernel's source."""
    path = os.path.join(PROFILE_DIR, fname)
    if not os.path.exists(path):
        return None
    try:
        rec = json.load(open(path)).get(traffic_key(workload, geo, stage))
    except (ValueError, OSError):
        return None
    if not rec or not rec.get("kernel"):
        return None
    if rec.get("source_sha256") != source_digest(source_for_kernels(rec["kernel"])):
        return None
    return rec


def measured_traffic(workload, geo, stage):
    """HBM bytes per launch from committed rocprofv3 counter runs of the same
    workload and tiling, or None if absent or stale."""
    rec = _profile_record("traffic.json", workload, geo, stage)
    return None if rec is None else rec.get("bytes_per_launch")


def measured_mfma(workload, geo, stage):
    """Matrix-core counters of a contraction stage (busy fraction and fp32
    MFMA flops per launch) from committed rocprofv3 runs, or None."""
    rec = _profile_record("mfma.json", workload, geo, stage)
    if rec is None:
        return None
    return {k: rec[k] for k in ("mfma_busy", "mfma_f32_flops", "mfma_xf32_flops", "mfma_bf16_flops") if k in rec}


def cpu_baseline(ly, x, w, g, budget_s=20.0):
    """The fp64 oracle on the host on a sample of whole images (all channels,
    all kernels, all three passes), grown until about budget_s of work."""
    import numpy as np
    import oracle
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        cores = os.cpu_count() or 1
    b, spent, flops = 0, 0.0, 0.0
    per_img = 3 * ly.direct_flops() / ly.B
    while b < ly.B and spent < budget_s:
        xs, gs = np.asarray(x[b:b + 1], np.float64), np.asarray(g[b:b + 1], np.float64)
        t0 = time.perf_counter()
        oracle.conv_forward(xs, w)
        oracle.conv_backward_data(gs, w, ly.N)
        oracle.conv_backward_filter(xs, gs, ly.n)
        spent += time.perf_counter() - t0
        flops += per_img
        b += 1
        if spent * (ly.B / b) < budget_s * 0.5 and b == ly.B:
            break
    return {"value": flops / spent / 1e12, "unit": "TFLOP/s (direct-conv equivalent, fp64)",
            "cores": int(cores), "kind": "oracle",
            "sample": f"{b} of {ly.B} images, all {ly.C} channels and {ly.K} kernels, forward + "
                      f"backward_data + backward_filter, {spent:.1f} s"}


STAGE_ORDER = ["w_spectrum", "x_spectrum", "fwd_product", "fwd_inverse", "g_spectrum", "bwd_data_product",
               "bwd_data_inverse", "bwd_filter_product", "bwd_filter_inverse"]
LIB_KERNELS = ("tile_rfft2_kernel", "window_rfft2_kernel", "window_rows_rfft2_kernel", "irfft2_", "cgemm_", "narrow_",
               "big_rfft2", "big_irfft2", "overlap_gather", "fused_")


def stage_sequence(geo):
    """The stage of each kernel launch of one training step, in launch order
    (the fused passes launch one kernel per pass; the two-step overlap-add at
    L = 128, planes of more than two tiles, adds a gather kernel)."""
    if geo.get("fused"):
        return ["w_spectrum", "x_spectrum", "fwd_inverse", "bwd_data_product", "bwd_filter_product",
                "bwd_filter_inverse"]
    seq = list(STAGE_ORDER)
    if geo["L"] >= 128 and geo["P"] > 2:
        twice = "bwd_data_inverse" if geo.get("method") else "fwd_inverse"
        seq.insert(seq.index(twice), twice)
    return seq


def _per_stage(dispatches, seq, steps):
    """Group the last `steps` steps' dispatches [(kernel, {counter: value})]
    by stage: {stage: (kernels, {counter: mean per step})}."""
    n = len(seq)
    dispatches = dispatches[-steps * n:]
    out = {}
    for j in range(steps):
        for i, stage in enumerate(seq):
            k, vals = dispatches[j * n + i]
            ks, acc = out.setdefault(stage, ([], {}))
            if k not in ks:
                ks.append(k)
            for c, v in vals.items():
                acc[c] = acc.get(c, 0.0) + v / steps
    return {st: ("+".join(ks), acc) for st, (ks, acc) in out.items()}


def _short_kernel(name):
    name = name.replace("void oaa::(anonymous namespace)::", "")
    return name.split("(oaa::")[0]


def _dispatch_values(run_dir, counter):
    """Per-dispatch values of one counter from a rocprofv3 csv run, library
    kernels only, in dispatch order: [(kernel, value), ...]."""
    import csv
    import glob
    rows = list(csv.DictReader(open(glob.glob(os.path.join(run_dir, "**", "*counter_collection.csv"),
                                              recursive=True)[0])))
    per = {}
    for r in rows:
        if r["Counter_Name"] != counter:
            continue
        d = int(r["Dispatch_Id"])
        per[d] = (_short_kernel(r["Kernel_Name"]), per.get(d, ("", 0.0))[1] + float(r["Counter_Value"]))
    return [per[d] for d in sorted(per)]


def summarize_pmc(layer, fetch_dir, write_dir, cal_fetch_dir, cal_write_dir, steps=2, method="oaa"):
    """HBM bytes per launch of each stage from FETCH_SIZE and WRITE_SIZE runs of
    `bench.py --layer <layer> --method <method> --steps 2 --warmup 1
    --no-cpu-baseline`, calibrated against runs of
    `bench.py --copy-calibration 1024`; prints the table and records the
    figures in profiles/traffic.json."""
    from paper_1601_06815_amd import binding
    from paper_1601_06815_amd.workloads import LAYERS
    ly = LAYERS[layer]
    m = binding.METHOD_OVERLAP_SAVE if method == "oas" else binding.METHOD_OVERLAP_ADD
    h = binding.oaa_plan_create_method(ly.B, ly.C, ly.K, ly.N, ly.n, 0, 0, m)
    geo = binding.oaa_plan_geometry(h)
    binding.oaa_plan_destroy(h)
    copy_bytes = 1024 * (1 << 20)
    cf = [v for k, v in _dispatch_values(cal_fetch_dir, "FETCH_SIZE")]
    cw = [v for k, v in _dispatch_values(cal_write_dir, "WRITE_SIZE")]
    # a plain copy reads and writes copy_bytes; counters are in KiB
    f_factor = copy_bytes / (sorted(cf)[len(cf) // 2] * 1024)
    w_factor = copy_bytes / (sorted(cw)[len(cw) // 2] * 1024)
    seq = stage_sequence(geo)
    fetch = _per_stage([(k, {"v": v}) for k, v in _dispatch_values(fetch_dir, "FETCH_SIZE")
                        if k.startswith(LIB_KERNELS)], seq, steps)
    write = _per_stage([(k, {"v": v}) for k, v in _dispatch_values(write_dir, "WRITE_SIZE")
                        if k.startswith(LIB_KERNELS)], seq, steps)
    work = stage_work(ly, geo)
    path = os.path.join(PROFILE_DIR, "traffic.json")
    db = json.load(open(path)) if os.path.exists(path) else {}
    db["_calibration"] = {"copy_bytes_each_way": copy_bytes, "fetch_factor": round(f_factor, 4),
                          "write_factor": round(w_factor, 4),
                          "note": "bytes = counter KiB x 1024 x factor; factors from a plain device copy"}
    name = "overlap-save, h" if geo.get("method") else "b"
    print(f"## {layer}, L={geo['L']} {name}={geo['b']} (mean over the last {steps} steps)")
    print(f"{'stage':20s} {'kernel':48s} {'fetch MB':>9s} {'write MB':>9s} {'total MB':>9s} {'algo MB':>9s} {'ratio':>6s}")
    for stage in [st for st in STAGE_ORDER if st in fetch]:
        kern = fetch[stage][0]
        fb = fetch[stage][1]["v"] * 1024 * f_factor
        wb = write[stage][1]["v"] * 1024 * w_factor
        algo = work[stage]["bytes"]
        print(f"{stage:20s} {kern[:48]:48s} {fb / 1e6:9.1f} {wb / 1e6:9.1f} {(fb + wb) / 1e6:9.1f} "
              f"{algo / 1e6:9.1f} {(fb + wb) / algo:6.2f}")
        db[traffic_key(layer, geo, stage)] = {
            "kernel": kern, "fetch_bytes": int(fb), "write_bytes": int(wb), "bytes_per_launch": int(fb + wb),
            "source_sha256": source_digest(source_for_kernels(kern))}
    with open(path, "w") as f:
        json.dump(db, f, indent=1, sort_keys=True)
        f.write("\n")


def summarize_counters(layer, run_dir, steps=2, method="oaa"):
    """Per-stage values of every counter in a rocprofv3 --pmc run of
    `bench.py --layer <layer> --method <method> --steps 2 --warmup 1
    --no-cpu-baseline` (mean over the last `steps` steps). For the
    contractions, the matrix-core figures (MfmaUtil: busy cycles of the
    MFMA units over active cycles of all SIMDs; MfmaFlopsF32 and the XF32 /
    BF16 MFMA op counts) are recorded in profiles/mfma.json."""
    import csv
    import glob
    from paper_1601_06815_amd import binding
    from paper_1601_06815_amd.workloads import LAYERS
    ly = LAYERS[layer]
    m = binding.METHOD_OVERLAP_SAVE if method == "oas" else binding.METHOD_OVERLAP_ADD
    h = binding.oaa_plan_create_method(ly.B, ly.C, ly.K, ly.N, ly.n, 0, 0, m)
    geo = binding.oaa_plan_geometry(h)
    binding.oaa_plan_destroy(h)
    rows = list(csv.DictReader(open(glob.glob(os.path.join(run_dir, "**", "*counter_collection.csv"),
                                              recursive=True)[0])))
    names = sorted({r["Counter_Name"] for r in rows})
    per = {}
    for r in rows:
        d = int(r["Dispatch_Id"])
        k = _short_kernel(r["Kernel_Name"])
        if not k.startswith(LIB_KERNELS):
            continue
        e = per.setdefault(d, {"kernel": k})
        e[r["Counter_Name"]] = e.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
    disp = [per[d] for d in sorted(per)]
    seq = stage_sequence(geo)
    if not geo.get("fused") and not any(d["kernel"].startswith(("cgemm_", "narrow_")) for d in disp):
        seq = [st for st in seq if not st.endswith("_product")]  # a run filtered to the transform kernels
    staged = _per_stage([(d["kernel"], {c: v for c, v in d.items() if c != "kernel"}) for d in disp],
                        seq, steps)
    work = stage_work(ly, geo)
    name = "overlap-save, h" if geo.get("method") else "b"
    print(f"## {layer}, L={geo['L']} {name}={geo['b']} (mean over the last {steps} steps)")
    print(f"{'stage':20s} {'kernel':44s} " + " ".join(f"{c[:24]:>24s}" for c in names))
    path = os.path.join(PROFILE_DIR, "mfma.json")
    db = json.load(open(path)) if os.path.exists(path) else {}
    for stage in [st for st in STAGE_ORDER if st in staged]:
        kern, vals = staged[stage]
        mean = {c: vals.get(c, 0.0) for c in names}
        print(f"{stage:20s} {kern[:44]:44s} " + " ".join(f"{mean[c]:24.4g}" for c in names))
        if work[stage].get("bound") == "mfma" and "MfmaUtil" in mean:
            rec = {"kernel": kern, "mfma_busy": round(mean["MfmaUtil"] / 100.0, 4),
                   "source_sha256": source_digest(source_for_kernels(kern))}
            if "MfmaFlopsF32" in mean:
                rec["mfma_f32_flops"] = mean["MfmaFlopsF32"]
            for c, key in (("SQ_INSTS_VALU_MFMA_MOPS_XF32", "mfma_xf32_flops"),
                           ("SQ_INSTS_VALU_MFMA_MOPS_BF16", "mfma_bf16_flops")):
                if c in mean:
                    rec[key] = mean[c] * 512
            db[traffic_key(layer, geo, stage)] = rec
    if any("MfmaUtil" in d for d in disp):
        with open(path, "w") as f:
            json.dump(db, f, indent=1, sort_keys=True)
            f.write("\n")


def summarize_stats(run_dir):
    """Short table from a rocprofv3 --kernel-trace --stats csv run."""
    import csv
    import glob
    rows = list(csv.DictReader(open(glob.glob(os.path.join(run_dir, "**", "*kernel_stats.csv"), recursive=True)[0])))
    print(f"{'kernel':64s} {'calls':>6s} {'avg us':>9s} {'min us':>9s} {'max us':>9s} {'% time':>7s}")
    for r in rows:
        print(f"{_short_kernel(r['Name'])[:64]:64s} {int(r['Calls']):6d} {float(r['AverageNs']) / 1e3:9.1f} "
              f"{float(r['MinNs']) / 1e3:9.1f} {float(r['MaxNs']) / 1e3:9.1f} {float(r['Percentage']):7.2f}")


PASS_STAGES = {
    "fwd": ("w_spectrum", "x_spectrum", "fwd_product", "fwd_inverse"),
    "bwd_data": ("g_spectrum", "bwd_data_product", "bwd_data_inverse"),
    "bwd_filter": ("bwd_filter_product", "bwd_filter_inverse"),
}
REPORT_LAYERS = ("tiny", "plane224_n3", "plane224_n5", "plane224_n8", "first224", "mid56", "large128")


def oracle_pass_ms(ly, x, w, g, pas, budget_s):
    """Host time of one pass of the fp64 oracle over the whole layer,
    extrapolated from as many whole images as fit in about budget_s (at
    least one); small layers: median of five runs."""
    import numpy as np
    import oracle

    def run(b0, b1):
        xs = np.asarray(x[b0:b1], np.float64)
        gs = None if g is None else np.asarray(g[b0:b1], np.float64)
        t0 = time.perf_counter()
        if pas == "fwd":
            oracle.conv_forward(xs, w)
        elif pas == "bwd_data":
            oracle.conv_backward_data(gs, w, ly.N)
        else:
            oracle.conv_backward_filter(xs, gs, ly.n)
        return time.perf_counter() - t0

    if ly.direct_flops() < 1e9:
        times = sorted(run(0, ly.B) for _ in range(5))
        return times[2] * 1e3, f"median of 5, all {ly.B} images"
    spent, b = 0.0, 0
    while b < ly.B and (b == 0 or spent < budget_s):
        spent += run(b, b + 1)
        b += 1
    return spent / b * ly.B * 1e3, f"{b} of {ly.B} images, scaled"


def config_report(args):
    """Per config and pass: ms (median of 20 after 3 warm-ups, and the mean of
    the first 10), direct-convolution-equivalent TFLOP/s, each stage's share
    and roofline fraction, and the fp64 oracle's host time."""
    import numpy as np
    import torch
    from paper_1601_06815_amd import binding
    from paper_1601_06815_amd.workloads import LAYERS, make_inputs

    dev = torch.device("cuda:0")
    rows = []
    for name in REPORT_LAYERS:
        ly = LAYERS[name]
        x, w, g = make_inputs(ly, seed=0, want_g="bwd_data" in ly.passes)
        plan = binding.Plan(ly.B, ly.C, ly.K, ly.N, ly.n, device=dev, tiling="auto")
        geo = plan.geometry
        work = stage_work(ly, geo)
        xd, wd = torch.from_numpy(x).to(dev), torch.from_numpy(w).to(dev)
        gd = None if g is None else torch.from_numpy(g).to(dev)
        y = torch.empty((ly.B, ly.K, ly.M, ly.M), dtype=torch.float32, device=dev)
        dx, dw = torch.empty_like(xd), torch.empty_like(wd)
        # the passes as a training step runs them: backward_data reuses the
        # kernel spectra of the forward pass, backward_filter the input and
        # gradient spectra of the two before it
        calls = {"fwd": lambda: plan.forward(xd, wd, y),
                 "bwd_data": lambda: plan.backward_data(gd, None, dx),
                 "bwd_filter": lambda: plan.backward_filter(None, None if plan.caches_grad_spectra else gd, dw)}
        for pas in ly.passes:
            call = calls[pas]
            for _ in range(3):
                call()
            torch.cuda.synchronize()
            ts = []
            plan.set_timing(True)
            plan.stage_times()
            for _ in range(20):
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                call()
                e1.record()
                torch.cuda.synchronize()
                ts.append(e0.elapsed_time(e1))
            st = plan.stage_times()
            plan.set_timing(False)
            med, mean10 = float(np.median(ts)), float(np.mean(ts[:10]))
            # the same pass replayed from a HIP graph (launch overheads removed)
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph):
                call()
            graph.replay()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            for _ in range(20):
                graph.replay()
            e1.record()
            torch.cuda.synchronize()
            ms_graph = e0.elapsed_time(e1) / 20
            del graph
            stages = {}
            for sname, (ms, cnt) in st.items():
                if not cnt or sname not in PASS_STAGES[pas]:
                    continue
                sm = ms / cnt
                wk = work[sname]
                frac_exec = None
                if "flops" in wk and min(ly.C, ly.K) >= 64:
                    frac = wk["flops"] / (sm * 1e-3) / 1e12 / FP32_MFMA_PEAK_TFLOPS
                    frac_exec = wk["flops_exec"] / (sm * 1e-3) / 1e12 / FP32_MFMA_PEAK_TFLOPS
                    bound = "mfma"
                else:
                    frac = wk["bytes"] / (sm * 1e-3) / 1e9 / HBM_PEAK_GBS
                    bound = "hbm"
                stages[sname] = {"ms": sm, "share": sm / med, "bound": bound, "frac": frac, "frac_exec": frac_exec}
            cpu_ms, cpu_note = oracle_pass_ms(ly, x, w, g, pas, args.cpu_budget / 4)
            row = {"layer": name, "pass": pas, "L": geo["L"], "b": geo["b"], "ms_median": med, "ms_mean10": mean10,
                   "ms_graph": ms_graph,
                   "tflops_direct_eq": ly.direct_flops() / (med * 1e-3) / 1e12, "stages": stages,
                   "oracle_ms": cpu_ms, "oracle_sample": cpu_note, "speedup_vs_oracle": cpu_ms / med}
            rows.append(row)
            print(f"[report] {name} {pas}: {med:.4f} ms", file=sys.stderr, flush=True)
        del plan
        torch.cuda.empty_cache()

    print("| layer | pass | (L, b) | ms median | ms mean of 10 | ms graph replay | direct-eq TFLOP/s "
          "| stages: share, roofline fraction | fp64 oracle ms (host) | GPU / oracle |")
    print("|---|---|---|---|---|---|---|---|---|---|")
    for r in rows:
        # layers whose data stays in L2 and whose stages last a few
        # microseconds are bound by launch latency: no roofline fraction
        small = LAYERS[r["layer"]].direct_flops() < 1e9
        st = "; ".join(f"{k} {v['share'] * 100:.0f} %" + ("" if small else f", {v['frac'] * 100:.0f} % {v['bound']}")
                       + ("" if small or v.get("frac_exec") is None else f" ({v['frac_exec'] * 100:.0f} % executed)")
                       for k, v in r["stages"].items())
        if small:
            st += " (latency-bound)"
        print(f"| {r['layer']} | {r['pass']} | ({r['L']}, {r['b']}) | {r['ms_median']:.4f} | {r['ms_mean10']:.4f} "
              f"| {r['ms_graph']:.4f} | {r['tflops_direct_eq']:.2f} | {st} | {r['oracle_ms']:.1f} ({r['oracle_sample']}) "
              f"| {r['speedup_vs_oracle']:.0f}× |")
    r8 = next(r for r in rows if r["layer"] == "plane224_n8")
    xs = r8["stages"].get("x_spectrum", {"share": 0.0})["share"]
    print()
    print(f"224 x 224 plane, 8 x 8 kernel, forward: block division, padding and block transforms take "
          f"{xs * 100:.1f} % of the pass here (one fused kernel); the paper reports 1.6 % for tiling and "
          f"padding alone (Section 3.2).")
    print(f"Same layer: {r8['speedup_vs_oracle']:.0f}x the fp64 oracle on the host; the paper reports up to "
          f"16.3x for OaA over its own single-threaded spatial convolution (Abstract), on hardware it does "
          f"not state: context, not a target.")
    if args.report_out:
        with open(args.report_out, "w") as f:
            json.dump(rows, f, indent=1)
            f.write("\n")


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--layer", default="large128")
    ap.add_argument("--contraction", default="auto", choices=["auto", "valu", "mfma", "narrow", "fused"])
    ap.add_argument("--tiling", default="auto",
                    help="auto: the library's block size (fewer, larger blocks where that cuts work); "
                         "paper: blocks of the kernel's size n; L:b an explicit transform side and block")
    ap.add_argument("--method", default="oaa", choices=["oaa", "oas"],
                    help="oaa: the paper's overlap-and-add tiling; oas: the output-tiled alternative "
                         "(overlap-and-save forward, overlap-add of gradient blocks)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=20.0)
    ap.add_argument("--stages-out", default=None, help="also write per-stage timings as JSON here")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB (for counter calibration) and exit")
    ap.add_argument("--summarize-pmc", nargs=4, metavar=("FETCH_DIR", "WRITE_DIR", "CAL_FETCH_DIR", "CAL_WRITE_DIR"),
                    help="host only: HBM traffic per stage of --layer from rocprofv3 FETCH_SIZE/WRITE_SIZE runs")
    ap.add_argument("--report", action="store_true",
                    help="per config and pass: ms, direct-equivalent TFLOP/s, stage shares and roofline fractions, "
                         "oracle host time (a table, not the JSON line)")
    ap.add_argument("--report-out", default=None, help="with --report: also write the rows as JSON here")
    ap.add_argument("--summarize-counters", metavar="DIR",
                    help="host only: per-stage counter values of --layer from a rocprofv3 --pmc run "
                         "(records matrix-core figures in profiles/mfma.json)")
    ap.add_argument("--summarize-stats", metavar="DIR",
                    help="host only: table of a rocprofv3 --kernel-trace --stats run")
    ap.add_argument("--lib", default=None,
                    help="run the library built at this path instead of the in-tree one (to compare builds)")
    args = ap.parse_args()
    if args.summarize_pmc:
        summarize_pmc(args.layer, *args.summarize_pmc, method=args.method)
        return
    if args.summarize_stats:
        summarize_stats(args.summarize_stats)
        return
    if args.summarize_counters:
        summarize_counters(args.layer, args.summarize_counters, method=args.method)
        return

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(the layer would shard along the batch, with one all-reduce of dw).", file=sys.stderr)
        sys.exit(2)
    if args.lib:
        from paper_1601_06815_amd import binding
        binding.use_library(args.lib)
    if args.report:
        config_report(args)
        return

    import numpy as np
    import torch
    from paper_1601_06815_amd import binding
    from paper_1601_06815_amd.workloads import LAYERS, make_inputs

    dev = torch.device("cuda:0")
    if args.copy_calibration:
        n = args.copy_calibration * (1 << 20) // 4
        a = torch.ones(n, dtype=torch.float32, device=dev)
        b = torch.empty_like(a)
        for _ in range(5):
            torch.mul(a, 1.0, out=b)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes_each_way": n * 4, "launches": 5}))
        return

    ly = LAYERS[args.layer]
    t0 = time.perf_counter()
    x, w, g = make_inputs(ly, seed=0)
    print(f"[bench] inputs for {ly.name} drawn in {time.perf_counter() - t0:.1f} s", file=sys.stderr, flush=True)
    which = {"auto": binding.CONTRACTION_AUTO, "valu": binding.CONTRACTION_VALU,
             "mfma": binding.CONTRACTION_MFMA, "narrow": binding.CONTRACTION_NARROW,
             "fused": binding.CONTRACTION_FUSED}[args.contraction]
    tiling = args.tiling if args.tiling in ("auto", "paper") else tuple(int(v) for v in args.tiling.split(":"))
    method = binding.METHOD_OVERLAP_SAVE if args.method == "oas" else binding.METHOD_OVERLAP_ADD
    if method == binding.METHOD_OVERLAP_SAVE and isinstance(tiling, tuple):
        tiling = (tiling[0], 0)
    plan = binding.Plan(ly.B, ly.C, ly.K, ly.N, ly.n, device=dev, contraction=which, tiling=tiling, method=method)
    geo = plan.geometry
    xd, wd, gd = (torch.from_numpy(a).to(dev) for a in (x, w, g))
    y = torch.empty((ly.B, ly.K, ly.M, ly.M), dtype=torch.float32, device=dev)
    dx = torch.empty_like(xd)
    dw = torch.empty_like(wd)

    def step():
        plan.forward(xd, wd, y)
        plan.backward_data(gd, None, dx)
        plan.backward_filter(None, None if plan.caches_grad_spectra else gd, dw)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    print(f"[bench] warmup done ({args.warmup} steps)", file=sys.stderr, flush=True)

    plan.set_timing(True)
    plan.stage_times()  # clear
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    ev0.record()
    for _ in range(args.steps):
        step()
    ev1.record()
    torch.cuda.synchronize()
    ms_total = ev0.elapsed_time(ev1)
    stages = plan.stage_times()
    plan.set_timing(False)
    ms_step = ms_total / args.steps
    print(f"[bench] timed {args.steps} steps: {ms_step:.3f} ms/step", file=sys.stderr, flush=True)

    # the same step captured once in a HIP graph and replayed (no per-stage
    # events): what a training loop that replays its step would see
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    graph.replay()
    torch.cuda.synchronize()
    ev0.record()
    for _ in range(args.steps):
        graph.replay()
    ev1.record()
    torch.cuda.synchronize()
    ms_graph = ev0.elapsed_time(ev1) / args.steps
    del graph
    print(f"[bench] graph replays: {ms_graph:.3f} ms/step", file=sys.stderr, flush=True)

    direct = 3 * ly.direct_flops()
    value = direct / (ms_step * 1e-3) / 1e12
    work = stage_work(ly, geo)
    per_stage = {}
    for name, (ms, cnt) in stages.items():
        if cnt:
            per_stage[name] = {"ms_per_launch": ms / cnt, "launches": cnt}
    dom = max(per_stage, key=lambda k: per_stage[k]["ms_per_launch"] * per_stage[k]["launches"])
    avg_s = per_stage[dom]["ms_per_launch"] * 1e-3
    wk = work[dom]
    if wk.get("bound") == "mfma":
        achieved = wk["flops"] / avg_s / 1e12
        executed = wk["flops_exec"] / avg_s / 1e12
        roof = {"bound": "mfma", "achieved": achieved, "peak": FP32_MFMA_PEAK_TFLOPS, "unit": "TFLOP/s",
                "frac": achieved / FP32_MFMA_PEAK_TFLOPS,
                "flops_counted": "8 B P C K F: 8 real flops per complex multiply-add over all L(L/2+1) "
                                 "stored bins of every tile",
                "executed": {"achieved": executed, "frac": executed / FP32_MFMA_PEAK_TFLOPS,
                             "flops_counted": "6 real flops per complex multiply-add (three real matrix-core "
                                              "products) over the bins that are not conjugates of others"},
                "counters": measured_mfma(ly.name, geo, dom)}
    else:
        achieved = wk["bytes"] / avg_s / 1e9
        roof = {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": achieved / HBM_PEAK_GBS}
    roof["traffic"] = measured_traffic(ly.name, geo, dom)
    roof["kernel"] = dom
    roof["ms_per_launch"] = per_stage[dom]["ms_per_launch"]
    for name, st in per_stage.items():
        wk = work[name]
        s = st["ms_per_launch"] * 1e-3
        st["gbs_algorithmic"] = wk["bytes"] / s / 1e9
        if "flops" in wk:
            st["tflops"] = wk["flops"] / s / 1e12
            st["tflops_executed"] = wk["flops_exec"] / s / 1e12

    # sampled parity of the timed outputs against the oracle
    import oracle
    rng = np.random.default_rng(0)
    S = 24
    iy = [rng.integers(0, s, S) for s in (ly.B, ly.K, ly.M, ly.M)]
    ix = [rng.integers(0, s, S) for s in (ly.B, ly.C, ly.N, ly.N)]
    iw = [rng.integers(0, s, S) for s in (ly.K, ly.C, ly.n, ly.n)]
    yh, dxh, dwh = y.cpu().numpy(), dx.cpu().numpy(), dw.cpu().numpy()
    errs = {}
    for key, got, ref in (("y", yh[tuple(iy)], oracle.conv_forward_at(x, w, *iy)),
                          ("dx", dxh[tuple(ix)], oracle.conv_backward_data_at(g, w, ly.N, *ix)),
                          ("dw", dwh[tuple(iw)], oracle.conv_backward_filter_at(x, g, ly.n, *iw))):
        scale = float(np.max(np.abs(ref)))
        diff = float(np.max(np.abs(got - ref)))
        errs[key] = diff / scale if scale > 0 else diff
    err = max(errs.values())

    out = {
        "metric": "OaA conv fwd+bwd ms & direct-equiv TFLOP/s; % of HBM BW / MFMA peak",
        "value": value,
        "unit": "TFLOP/s (direct-conv equivalent)",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded numpy draws, resident in HBM)",
        "config": {"workload": f"{ly.name}: x[{ly.B},{ly.C},{ly.N},{ly.N}] w[{ly.K},{ly.C},{ly.n},{ly.n}] "
                               f"valid stride 1, forward + backward_data + backward_filter",
                   "B": ly.B, "C": ly.C, "K": ly.K, "N": ly.N, "n": ly.n,
                   "L": geo["L"], "block": geo["b"], "T": geo["T"], "split": geo["split"], "tiling": args.tiling,
                   "method": args.method,
                   "contraction": args.contraction},
        "roofline": roof,
        "graph_ms_per_step": ms_graph,
        "stages": per_stage,
        "sampled_rel_err": err,
        "sampled_rel_err_by_output": errs,
    }
    if args.stages_out:
        with open(args.stages_out, "w") as f:
            json.dump(per_stage, f, indent=1)
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle sample", file=sys.stderr, flush=True)
        out["cpu_baseline"] = cpu_baseline(ly, x, w, g, args.cpu_budget)
    else:
        out["cpu_baseline"] = None
    print(json.dumps(out), flush=True)
    if not err <= PARITY_TOL:
        print(f"[bench] sampled outputs differ from the oracle: {errs} > {PARITY_TOL}", file=sys.stderr, flush=True)
        sys.exit(1)


if __name__ == "__main__":
    main()
