"""Benchmark of the FAVOR hot path on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]

One step is one pass of the whole path over the protein-shaped workload
(B4 H8 L8192, d 64, M 256, bf16): draw the orthogonal random features for the
8 heads (favor_orf_draw, a fresh seed per step), then bidirectional FAVOR and
unidirectional FAVOR over the same Q, K, V (favor_attn_both: one pass over the
keys serves both directions). Inputs are synthetic and already resident in HBM;
nothing is skipped inside the timed region. Untimed warmup runs at least
--warmup steps and at least --min-warmup-seconds (the clocks settle over a few
hundred milliseconds; a short warmup reads about 7% slow).

value = B*H*L / (seconds per step): token-heads per second through the whole
step (each token-head goes through the draw, both directions), from a timed
region without per-launch instrumentation, the draw in line before the
attention pass on one stream. ms_per_step_pipelined times the same steps with
the features of step i + 1 drawn on a second stream while step i attends with
its own (two feature buffers, ordered by events); every attention kernel fills
the chip, so there the draw delays them instead of hiding. A third region,
serial, with every launch bracketed by HIP events on its stream, gives the
per-kernel durations and the roofline entry for the dominant
kernel. The line also carries the fp64 CPU oracle timed on this host
(cpu_baseline), and under "variants" the same step with generalized attention
(ReLU features) and with the renormalisation off, the draw alone for every kind
of random features, one GPU's share of a causal pass sharded eight ways along
the sequence (the last L/8 tokens from a carried state), the step captured once
as a HIP graph and replayed (and the launch-bound B1 H1 L1024 configuration
eager against replayed), the backward pass of the step's attention, and the
training step (forward saving the row scales, then the backward reading them),
timed the same way.

Beside the headline, the line carries "feature_map" (favor_feature_map on the
workload's Q: the materialised feature-map phase) and "workloads": every
other workload of the configuration list at its full size, each with its step
time, per-kernel durations and the roofline of its dominant kernel
(bidir_b8h8 and causal_b8h8 with the draw timed on its own beside the step,
causal_b8h8 also over three causal segment lengths; causal_long with the
redraw inside the timed step); the causal workloads also over both chunk
lengths of the scan (64 and 32 tokens).

python bench.py --summarize-counters DIR turns rocprofv3 FETCH_SIZE /
WRITE_SIZE runs (see summarize_counters) into profiles/traffic.json.
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import workloads as wl  # noqa: E402

# MI355X published peaks
PEAK_HBM_GBS = 8000.0
PEAK_MFMA_TFLOPS = {"bf16": 2500.0, "f32": 157.3}
# v_cos_f32 issues at half the fp32 rate on CDNA4: 256 CUs x 4 SIMD x 16 lanes x
# 2.4 GHz / 2 = 19.66e12 cosines per second (the rate this GPU reaches is in the
# line's measured_peaks, from the library's cosine probe).
PEAK_COS_PER_S = 256 * 4 * 16 * 2.4e9 / 2
# Measured HBM traffic per launch (rocprofv3 FETCH_SIZE / WRITE_SIZE, scaled by a
# plain copy of known size), valid only for the kernel sources it was taken on.
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")
KERNEL_SOURCES = os.path.join(ROOT, "paper_2006_03555_amd", "csrc")


# Sources of the kernels the bench step launches and of their launch planning, and
# the build script (its per-source compiler flags change the kernels too).
STEP_SOURCES = ("bidir.hip", "causal.hip", "feature_map.hip", "orf_draw.hip", "favor_api.cpp",
                "favor_common.hpp", "kernels.hpp", "tile_common.hpp", "../build.py")


def kernel_source_hash():
    import hashlib
    h = hashlib.sha256()
    for fn in STEP_SOURCES:
        with open(os.path.join(KERNEL_SOURCES, fn), "rb") as f:
            h.update(fn.encode() + b"\0" + f.read())
    return h.hexdigest()


def measured_traffic(kernel, workload):
    """HBM bytes per launch of `kernel` on `workload` from the committed counter
    summary, or None if there is none or the kernel sources changed since."""
    try:
        with open(TRAFFIC_FILE) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("source_sha256") != kernel_source_hash():
        return None
    k = t.get("workloads", {}).get(workload, {}).get("kernels", {}).get(kernel)
    return None if k is None else k["bytes_per_launch"]


def per_token_head(kernel, d, M, elt, out_elt=None):
    """Algorithmic (flops, bytes, cosines) per token-head of one launch of `kernel`.

    flops: the feature projections (2 d M each side computed) and the
    contractions of Algorithm 1 / Eq. cumsum (2 M (d+1) each); bytes: the
    minimal HBM traffic of the kernel's inputs and outputs; cosines: M per
    feature row computed."""
    proj = 2 * d * M
    contr = 2 * M * (d + 1)
    row = d * elt
    out_elt = elt if out_elt is None else out_elt
    if kernel == "k_causal":      # Q and K features, Q S + intra, S update; reads Q K V, writes out
        return 2 * proj + 2 * contr, 4 * row, 2 * M
    if kernel == "k_qside":       # Q features, Q' Buf1; reads Q, writes out
        return proj + contr, 2 * row, M
    if kernel == "k_kside":       # K features, K'^T [V 1]; reads K, V
        return proj + contr, 2 * row, M
    if kernel == "k_feature_map":  # X features; reads X, writes X' (M values per row)
        return proj, row + M * out_elt, M
    return None


def cpu_baseline(w, Q, K, V):
    """The fp64 oracle on this host's cores over the whole workload (or a head
    subset), timed like one GPU step: ORF draw + bidirectional + causal."""
    from oracle import favor
    try:
        from threadpoolctl import threadpool_info
        blas = [p for p in threadpool_info() if p.get("user_api") == "blas"]
        cores = max((p["num_threads"] for p in blas), default=1)
        vendor = ", ".join(sorted({f"{p.get('internal_api')} {p.get('version')}" for p in blas}))
    except Exception:
        cores, vendor = 1, "unknown"
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    heads = w.B * w.H
    t0 = time.perf_counter()
    Wr, br = favor.orf_draw(12345, w.H, w.M, w.d)
    Qp = favor.feature_map(Q, Wr, br, w.input_scale)
    Kp = favor.feature_map(K, Wr, br, w.input_scale)
    favor.attn_bidir_features(Qp, Kp, V)
    favor.attn_causal_features(Qp, Kp, V)
    t = time.perf_counter() - t0
    return {"value": heads * w.L / t, "unit": "token-heads/s", "cores": int(cores),
            "kind": "oracle", "cpu_model": model, "blas": vendor,
            "host_cpus_available": len(os.sched_getaffinity(0)),
            "sample": f"whole workload ({w.B}x{w.H} heads x L={w.L}): ORF draw + bidirectional "
                      f"+ causal in fp64 NumPy, {t:.2f} s wall"}


def roofline(kernels, w, token_heads, out_elt=None):
    """Roofline entry of the kernel with the largest share of the step: its
    algorithmic FLOP, bytes and cosines per launch over its average launch
    duration against the MI355X peaks; the reported bound is the resource with
    the largest fraction."""
    dom = max(kernels, key=lambda k: kernels[k]["ms_per_launch"] * kernels[k]["launches_per_step"])
    elt = 2 if w.dtype == "bf16" else 4
    costs = per_token_head(dom, w.d, w.M, elt, out_elt)
    if costs is None:
        return {"kernel": dom, "bound": None}
    fl, by, cs = costs
    t = kernels[dom]["ms_per_launch"] / 1e3
    cand = {
        "mfma": (fl * token_heads / t / 1e12, PEAK_MFMA_TFLOPS[w.dtype], "TFLOP/s"),
        "hbm": (by * token_heads / t / 1e9, PEAK_HBM_GBS, "GB/s"),
        "alu": (cs * token_heads / t / 1e12, PEAK_COS_PER_S / 1e12, "Tcos/s"),
    }
    bound = max(cand, key=lambda k: cand[k][0] / cand[k][1])
    a, p, u = cand[bound]
    return {"kernel": dom, "bound": bound, "achieved": a, "peak": p, "unit": u, "frac": a / p,
            "traffic": measured_traffic(dom, w.name),
            "algorithmic_bytes_per_launch": by * token_heads,
            "algorithmic_flop_per_launch": fl * token_heads,
            "others": {k: {"achieved": v[0], "peak": v[1], "unit": v[2], "frac": v[0] / v[1]}
                       for k, v in cand.items() if k != bound}}


def time_steps(torch, fv, stream, step, first, steps, instrumented=False):
    """Milliseconds per step over `steps` calls of step(first + i), timed with
    HIP events on `stream` (the library launches on the stream it is given);
    instrumented also returns the library's per-kernel event times."""
    torch.cuda.synchronize()
    if instrumented:
        fv.timing_reset()
        fv.timing_enable(True)
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for i in range(steps):
        step(first + i)
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    if not instrumented:
        return ms
    fv.timing_enable(False)
    kt = fv.timing_read()
    return ms, {k: {"ms_per_launch": v[0] / v[1], "launches_per_step": v[1] / steps}
                for k, v in kt.items() if v[1] > 0}


def measured_peaks(torch, fv):
    """Rates this GPU reaches on the resources the roofline uses, beside the
    published peaks: bf16 matrix-core FLOP/s and cosines/s from the library's
    probes (favor_probe), HBM bytes/s from a 1 GiB device copy (read + write).
    Best of five launches each."""
    st = torch.cuda.current_stream()
    sink = torch.zeros(512, dtype=torch.float32, device="cuda")
    out = {}

    def best(fn, n=5):
        ts = []
        for _ in range(n + 1):
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record(st)
            fn()
            e1.record(st)
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1) / 1e3)
        return min(ts[1:])

    for kind, iters, key, scale in ((0, 400, "mfma_bf16_tflops", 1e12),
                                    (1, 20000, "cos_per_s", 1.0),
                                    (2, 40, "hadamard_apply_tokens_per_s", 1.0)):
        import ctypes
        run = lambda: fv.lib().favor_probe(kind, iters, ctypes.c_void_p(sink.data_ptr()),
                                           ctypes.c_void_p(st.cuda_stream))
        t = best(run)
        out[key] = fv.lib().favor_probe_work(kind, iters) / t / scale
    # the dense projection of one token onto M = 256 rows is 2 d M = 32768 FLOP on the
    # matrix cores; the structured H-ORF apply does it in O(M log d) vector additions
    out["dense_projection_tokens_per_s"] = out["mfma_bf16_tflops"] * 1e12 / (2 * 64 * 256)
    n = (1 << 30) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    t = best(lambda: dst.copy_(src))
    out["hbm_copy_gbs"] = 2 * n * 4 / t / 1e9
    out["published"] = {"mfma_bf16_tflops": PEAK_MFMA_TFLOPS["bf16"], "cos_per_s": PEAK_COS_PER_S,
                        "hbm_gbs": PEAK_HBM_GBS}
    del src, dst
    return out


def default_chunk(w):
    """The chunk length the library picks for chunk = 0 (favor_desc.chunk)."""
    return 32 if w.dtype == "bf16" and w.M <= 128 else 64


def bench_workload(name, args, torch, fv, segment_rows=(0,), chunks=(0,)):
    """One workload of the configuration list at its full size: the step is its
    attention call(s) over inputs resident in HBM, with the random-feature draw
    inside the step when the workload redraws on every call, else timed on its
    own beside it. Returns its entry for the bench line."""
    w = wl.WORKLOADS[name]
    dev = torch.device("cuda", 0)
    Q, K, V = wl.make_qkv(w)
    tdt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    up = lambda x: torch.from_numpy(x).to(device=dev, dtype=tdt).contiguous()
    Qd, Kd, Vd = up(Q), up(K), up(V)
    del Q, K, V
    s, H, M = w.input_scale, w.H, w.M
    code = fv.BF16 if w.dtype == "bf16" else fv.F32
    Wd = torch.empty((H, M, w.d), dtype=torch.float32, device=dev)
    bd = torch.empty((H, M), dtype=torch.float32, device=dev)
    out = torch.empty_like(Qd)
    out2 = torch.empty_like(Qd)
    st = torch.cuda.current_stream()
    op = {"bidir": 0, "causal": 1, "both": 2}[w.direction]
    th = w.B * w.H * w.L
    first = 0
    entry = {"config": {"B": w.B, "H": H, "L": w.L, "d": w.d, "M": M, "dtype": w.dtype,
                        "direction": w.direction,
                        "orf_draw": "inside the timed step (redrawn every call)" if w.redraw
                        else "outside the timed step (timed on its own)"}}
    fv.orf_draw(77, H, M, w.d, W=Wd, b=bd, stream=st)
    sweep = {}
    # (segment rows, chunk tokens): the first is the entry's own figure
    configs = [(rows, chunks[0]) for rows in segment_rows] + [(segment_rows[0], c)
                                                              for c in chunks[1:]]
    for rows, chunk in configs:
        g = fv.make_desc(w.B, H, w.L, w.d, M, code, code, s, segment=rows, chunk=chunk)
        ws = torch.empty(fv.workspace_size(g, op), dtype=torch.uint8, device=dev)

        def step(i):
            if w.redraw:
                fv.orf_draw(1000 + i, H, M, w.d, W=Wd, b=bd, stream=st)
            if op == 0:
                fv.attn_bidir(Qd, Kd, Vd, Wd, bd, s, out=out, workspace=ws, stream=st)
            elif op == 1:
                fv.attn_causal(Qd, Kd, Vd, Wd, bd, s, out=out, workspace=ws, stream=st,
                               segment=rows, chunk=chunk)
            else:
                fv.attn_both(Qd, Kd, Vd, Wd, bd, s, out_bidir=out, out_causal=out2,
                             workspace=ws, stream=st, segment=rows, chunk=chunk)

        t0 = time.perf_counter()
        n = 0
        while n < args.warmup or time.perf_counter() - t0 < args.min_warmup_seconds:
            step(first + n)
            n += 1
            if n % 16 == 0:
                torch.cuda.synchronize()
        first += n
        ms = time_steps(torch, fv, st, step, first, args.steps)
        first += args.steps
        ms_i, kernels = time_steps(torch, fv, st, step, first, args.steps, instrumented=True)
        first += args.steps
        sweep[(rows, chunk)] = {"ms_per_step": ms, "value": th / (ms / 1e3),
                                "ms_per_step_instrumented": ms_i, "kernels": kernels,
                                "roofline": roofline(kernels, w, th)}
    entry.update(sweep[configs[0]])
    brief = lambda v: {"ms_per_step": v["ms_per_step"], "value": v["value"],
                       "kernels": {k: x["ms_per_launch"] for k, x in v["kernels"].items()}}
    if len(segment_rows) > 1:
        entry["causal_segment_rows_sweep"] = {
            ("library default" if r == 0 else str(r)): brief(sweep[(r, chunks[0])])
            for r in segment_rows}
    if len(chunks) > 1:
        entry["causal_chunk_tokens_sweep"] = {
            str(c or default_chunk(w)): brief(sweep[(segment_rows[0], c)]) for c in chunks}
    if not w.redraw:
        draw = lambda i: fv.orf_draw(1000 + i, H, M, w.d, W=Wd, b=bd, stream=st)
        for i in range(args.warmup):
            draw(first + i)
        first += args.warmup
        entry["ms_orf_draw"] = time_steps(torch, fv, st, draw, first, args.steps)
    return entry


def bench_feature_map(w, Qd, Wd, bd, args, torch, fv):
    """favor_feature_map on the workload's Q with bf16 (or the input dtype's) X'
    of all M features: the materialised feature-map phase (Sec. 2.3)."""
    st = torch.cuda.current_stream()
    Xp = torch.empty((w.B, w.H, w.L, w.M), dtype=Qd.dtype, device=Qd.device)
    step = lambda i: fv.feature_map(Qd, Wd, bd, w.input_scale, out=Xp, stream=st)
    # warm up like the other entries: at least the warmup steps and the minimum time
    t0 = time.perf_counter()
    n = 0
    while n < max(args.warmup, 20) or time.perf_counter() - t0 < args.min_warmup_seconds:
        step(n)
        n += 1
        if n % 64 == 0:
            torch.cuda.synchronize()
    ms = time_steps(torch, fv, st, step, 0, args.steps)
    ms_i, kernels = time_steps(torch, fv, st, step, 0, args.steps, instrumented=True)
    th = w.B * w.H * w.L
    elt = Qd.element_size()
    # every launch of the uninstrumented region is k_feature_map, so its time per
    # call is the kernel's average duration; the events bracketing each launch in
    # the instrumented region add a few microseconds to a kernel this short
    kernels_region = {k: dict(v, ms_per_launch=ms / v["launches_per_step"])
                      for k, v in kernels.items()}
    roof = roofline(kernels_region, w, th, out_elt=elt)
    del Xp
    return {"what": f"X' = phi(Q) of the {w.name} workload ({w.B}x{w.H} heads x L={w.L}, "
                    f"M={w.M}), {w.dtype} in and out",
            "ms_per_call": ms, "value": th / (ms / 1e3), "ms_per_call_instrumented": ms_i,
            "kernels": kernels, "roofline": roof}


def copy_reference(nbytes, steps, warmup):
    """Time dst.copy_(src) on the device: nbytes read + nbytes written per launch."""
    import torch
    torch.cuda.set_device(0)
    n = nbytes // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(warmup):
        dst.copy_(src)
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    print(json.dumps({"copy_bytes": n * 4, "ms_per_copy": ms,
                      "GB_per_s_read_plus_write": 2 * n * 4 / (ms / 1e3) / 1e9}), flush=True)


COUNTERS = ("FETCH_SIZE", "WRITE_SIZE")
COPY_KIB = 262144.0      # the calibration copy: 256 MiB read and 256 MiB written


def _short_kernel(name):
    for k in ("k_causal", "k_orf_draw", "k_kside", "k_qside", "k_seg_scan", "k_finalize",
              "k_feature_map"):
        if k in name:
            return k
    if "copyBuffer" in name:   # the runtime's device-to-device copy of the calibration run
        return "copy"
    return name[:40]


def _pmc_means(path):
    import collections
    import csv
    agg = collections.defaultdict(list)
    with open(path) as f:
        for r in csv.DictReader(f):
            agg[_short_kernel(r["Kernel_Name"])].append(float(r["Counter_Value"]))
    return {k: sum(v) / len(v) for k, v in agg.items()}


def summarize_counters(root):
    """profiles/traffic.json from rocprofv3 --pmc runs, one counter per run:
    <root>/pmc_<COUNTER>_<workload>/run_counter_collection.csv for each workload
    and <root>/pmccopy_<COUNTER>/... for the calibration copy (bench.py
    --copy-bytes 268435456). Each counter's KiB per dispatch is scaled by what it
    reads for the copy, whose true traffic is 256 MiB each way."""
    import glob
    scale = {}
    for c in COUNTERS:
        copy = _pmc_means(os.path.join(root, f"pmccopy_{c}", "run_counter_collection.csv"))
        scale[c] = COPY_KIB / copy["copy"]
    out = {"source_sha256": kernel_source_hash(),
           "fetch_scale": scale["FETCH_SIZE"], "write_scale": scale["WRITE_SIZE"],
           "commands": {
               "counter": "rocprofv3 --pmc <COUNTER> -f csv -d "
                          "gpurun_out/pmc/pmc_<COUNTER>_<workload> -o run -- python3 bench.py "
                          "--workload <workload> --steps 3 --warmup 1 --min-warmup-seconds 0 "
                          "--no-cpu-baseline --no-variants --no-peaks --workloads ''",
               "copy": "rocprofv3 --pmc <COUNTER> -f csv -d "
                       "gpurun_out/pmc/pmccopy_<COUNTER> -o run -- python3 bench.py "
                       "--copy-bytes 268435456 --steps 3 --warmup 1",
               "summary": "python3 bench.py --summarize-counters gpurun_out/pmc"},
           "workloads": {}}
    for d in sorted(glob.glob(os.path.join(root, "pmc_FETCH_SIZE_*"))):
        if not os.path.isdir(d):
            continue
        name = os.path.basename(d)[len("pmc_FETCH_SIZE_"):]
        fetch = _pmc_means(os.path.join(d, "run_counter_collection.csv"))
        write = _pmc_means(os.path.join(root, f"pmc_WRITE_SIZE_{name}",
                                        "run_counter_collection.csv"))
        out["workloads"][name] = {"kernels": {
            k: {"fetch_kib_raw": v, "write_kib_raw": write.get(k, 0.0),
                "bytes_per_launch": (v * scale["FETCH_SIZE"]
                                     + write.get(k, 0.0) * scale["WRITE_SIZE"]) * 1024}
            for k, v in fetch.items()}}
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(out, f, indent=1)
    print(json.dumps(out, indent=1))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--min-warmup-seconds", type=float, default=0.3,
                    help="keep running untimed warmup steps until this long has passed "
                         "(the GPU clocks settle over a few hundred milliseconds)")
    ap.add_argument("--workload", default="protein_b4h8", choices=sorted(wl.WORKLOADS))
    ap.add_argument("--segment", type=int, default=0,
                    help="rows per segment of the causal scan (a multiple of 64; 0 = the "
                         "library's choice, one workgroup per CU with 64-token chunks, two "
                         "with 32) for the forward steps")
    ap.add_argument("--chunk", type=int, default=0, choices=(0, 32, 64),
                    help="tokens per step of the causal scan for the forward steps (0 = the "
                         "library's choice: 32 for bf16 inputs with M <= 128, else 64); the "
                         "causal workloads also time the other")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-variants", action="store_true",
                    help="skip the ReLU, unnormalised and backward variants (profiler runs "
                         "that average counters over every launch of a kernel)")
    ap.add_argument("--variants",
                    default="relu,softmax_no_renormalize,draws,causal_shard,graph,backward,"
                            "train_step",
                    help="comma-separated variants to time after the headline step")
    ap.add_argument("--workloads", default="bidir_b8h8,causal_b8h8,causal_long",
                    help="comma-separated further workloads of the configuration list, each "
                         "timed at full size into the line's 'workloads' object ('' = none)")
    ap.add_argument("--no-peaks", action="store_true",
                    help="skip the measured-peak probes (matrix cores, cosines, device copy)")
    ap.add_argument("--no-feature-map", action="store_true",
                    help="skip the materialised feature-map phase (favor_feature_map)")
    ap.add_argument("--summarize-counters", default="",
                    help="instead of running, read the rocprofv3 FETCH_SIZE / WRITE_SIZE CSVs "
                         "under this directory (pmc_<COUNTER>_<workload>/ and "
                         "pmccopy_<COUNTER>/) and write profiles/traffic.json")
    ap.add_argument("--copy-bytes", type=int, default=0,
                    help="instead of the workload, time a plain device-to-device copy of this "
                         "many bytes (reference for HBM bandwidth and for scaling the "
                         "FETCH_SIZE / WRITE_SIZE counters)")
    args = ap.parse_args()
    if args.summarize_counters:
        summarize_counters(args.summarize_counters)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the FAVOR path "
              "shards over heads with no communication between GPUs", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2006_03555_amd as fv

    if args.copy_bytes:
        copy_reference(args.copy_bytes, args.steps, args.warmup)
        return

    w = wl.WORKLOADS[args.workload]
    torch.cuda.set_device(0)
    dev = torch.device("cuda", 0)
    Q, K, V = wl.make_qkv(w)
    tdt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    up = lambda x: torch.from_numpy(x).to(device=dev, dtype=tdt).contiguous()
    Qd, Kd, Vd = up(Q), up(K), up(V)
    s = w.input_scale
    H, M = w.H, w.M
    # two random-feature buffers: a step reads slot i % 2 while the next step's
    # features are drawn into the other one
    Wd = [torch.empty((H, M, w.d), dtype=torch.float32, device=dev) for _ in range(2)]
    bd = [torch.empty((H, M), dtype=torch.float32, device=dev) for _ in range(2)]
    out_b = torch.empty_like(Qd)
    out_c = torch.empty_like(Qd)
    g = fv.make_desc(w.B, H, w.L, w.d, M, fv.BF16 if w.dtype == "bf16" else fv.F32,
                     fv.BF16 if w.dtype == "bf16" else fv.F32, s, segment=args.segment,
                     chunk=args.chunk)
    op = {"bidir": 0, "causal": 1, "both": 2}[w.direction]
    ws = torch.empty(fv.workspace_size(g, op), dtype=torch.uint8, device=dev)
    s_main = torch.cuda.current_stream()
    s_draw = torch.cuda.Stream()   # default priority, like every stream here
    ev_draw = [torch.cuda.Event(), torch.cuda.Event()]   # slot k drawn
    ev_attn = [torch.cuda.Event(), torch.cuda.Event()]   # attention done reading slot k

    def attention(slot, opts=None, stream=s_main):
        opts = dict(opts or {})
        if op != 0:
            opts["segment"] = args.segment
            opts["chunk"] = args.chunk
        if op == 2:     # one key pass serves both directions
            fv.attn_both(Qd, Kd, Vd, Wd[slot], bd[slot], s, out_bidir=out_b, out_causal=out_c,
                         workspace=ws, stream=stream, **opts)
        elif op == 0:
            fv.attn_bidir(Qd, Kd, Vd, Wd[slot], bd[slot], s, out=out_b, workspace=ws,
                          stream=stream, **opts)
        else:
            fv.attn_causal(Qd, Kd, Vd, Wd[slot], bd[slot], s, out=out_c, workspace=ws,
                           stream=stream, **opts)

    def step_serial(i, opts=None):
        """Draw this step's features, then attend with them (one stream)."""
        fv.orf_draw(1000 + i, H, M, w.d, W=Wd[0], b=bd[0], stream=s_main)
        attention(0, opts)

    def prime(i):
        """Draw the features of step i ahead of the pipelined steps."""
        for e in ev_attn:
            e.record(s_main)
        s_draw.wait_stream(s_main)
        fv.orf_draw(1000 + i, H, M, w.d, W=Wd[i & 1], b=bd[i & 1], stream=s_draw)
        ev_draw[i & 1].record(s_draw)

    def step_pipelined(i):
        """Attend with the features drawn during step i - 1 while the second stream
        draws those of step i + 1 into the other slot."""
        slot, nxt = i & 1, (i & 1) ^ 1
        s_draw.wait_event(ev_attn[nxt])       # step i - 1 no longer reads slot nxt
        fv.orf_draw(1000 + i + 1, H, M, w.d, W=Wd[nxt], b=bd[nxt], stream=s_draw)
        ev_draw[nxt].record(s_draw)
        s_main.wait_event(ev_draw[slot])      # this step's features are ready
        attention(slot)
        ev_attn[slot].record(s_main)

    def timed_region(step, first, instrumented=False, last_draw=None):
        """Time args.steps steps with events on the main stream (the library launches
        on the stream it is given). A pipelined region also waits for the draw it
        issued in its last step, so it holds exactly args.steps draws."""
        torch.cuda.synchronize()
        if instrumented:
            fv.timing_reset()
            fv.timing_enable(True)
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(s_main)
        for i in range(args.steps):
            step(first + i)
        if last_draw is not None:
            s_main.wait_event(last_draw((first + args.steps) & 1))
        e1.record(s_main)
        torch.cuda.synchronize()
        if instrumented:
            fv.timing_enable(False)
        return e0.elapsed_time(e1) / args.steps

    t_warm = time.perf_counter()
    n_warm = 0
    while n_warm < args.warmup or time.perf_counter() - t_warm < args.min_warmup_seconds:
        step_serial(n_warm)
        n_warm += 1
        if n_warm % 16 == 0:
            torch.cuda.synchronize()
    torch.cuda.synchronize()
    first = n_warm
    # headline: the draw in line on one stream, no per-launch instrumentation (each
    # event record adds a gap of a few microseconds between launches)
    ms_step = timed_region(step_serial, first)
    first += args.steps
    # the same steps with the next step's draw on a second stream (every attention
    # kernel fills the chip, so the draw's workgroups delay them rather than hide)
    prime(first)
    for i in range(args.warmup):
        step_pipelined(first + i)
    first += args.warmup
    torch.cuda.synchronize()
    prime(first)
    ms_step_pipelined = timed_region(step_pipelined, first, last_draw=lambda k: ev_draw[k])
    first += args.steps
    # per-kernel durations: serial steps with every launch bracketed by events
    ms_step_instrumented = timed_region(step_serial, first, instrumented=True)
    kt = fv.timing_read()
    kernels = {k: {"ms_per_launch": v[0] / v[1], "launches_per_step": v[1] / args.steps}
               for k, v in kt.items() if v[1] > 0}
    first += args.steps

    # the same step with generalized attention (ReLU features) and without the
    # renormalisation: same draw, same launches, other feature epilogue / finalisation
    variants = {}
    chosen = set() if args.no_variants else set(args.variants.split(","))
    if args.segment:   # the backward calls take the library's segments
        chosen -= {"backward", "train_step"}
    for name, opts in (("relu", dict(kernel=fv.KERNEL_RELU)),
                       ("softmax_no_renormalize", dict(renormalize=False))):
        if name not in chosen:
            continue
        step_v = lambda i, o=opts: step_serial(i, o)
        for i in range(args.warmup):
            step_v(first + i)
        first += args.warmup
        ms_v = timed_region(step_v, first)
        first += args.steps
        ms_vi = timed_region(step_v, first, instrumented=True)
        first += args.steps
        kv = fv.timing_read()
        variants[name] = {
            "ms_per_step": ms_v, "value": w.B * w.H * w.L / (ms_v / 1e3),
            "ms_per_step_instrumented": ms_vi,
            "kernels": {k: {"ms_per_launch": v[0] / v[1]} for k, v in kv.items() if v[1] > 0}}

    # one GPU's share of a causal pass sharded over 8 GPUs along the sequence: the
    # last L/8 tokens, entered with the state the seven shards before it hand over
    # (state_in non-zero; state_out is the hand-off to a next shard). The state is
    # computed before the timed region; the step is the draw + the shard's pass.
    if "causal_shard" in chosen and w.L % 8 == 0:
        ls = w.L // 8
        sl = slice(w.L - ls, w.L)
        Qs, Ks, Vs = (x[:, :, sl].contiguous() for x in (Qd, Kd, Vd))
        fv.orf_draw(999, H, M, w.d, W=Wd[1], b=bd[1], stream=s_main)
        before = [x[:, :, :w.L - ls].contiguous() for x in (Qd, Kd, Vd)]
        _, st_in = fv.attn_causal(*before, Wd[1], bd[1], s, return_state=True, stream=s_main)
        del before
        st_out = torch.empty_like(st_in)
        out_s = torch.empty_like(Qs)
        code = fv.BF16 if w.dtype == "bf16" else fv.F32
        gs = fv.make_desc(w.B, H, ls, w.d, M, code, code, s)
        ws_s = torch.empty(max(fv.workspace_size(gs, 1), 1), dtype=torch.uint8, device=dev)

        def step_shard(i):
            fv.orf_draw(1000 + i, H, M, w.d, W=Wd[0], b=bd[0], stream=s_main)
            fv.attn_causal(Qs, Ks, Vs, Wd[0], bd[0], s, state_in=st_in, state_out=st_out,
                           out=out_s, workspace=ws_s, stream=s_main)

        for i in range(args.warmup):
            step_shard(first + i)
        first += args.warmup
        ms_sh = timed_region(step_shard, first)
        first += args.steps
        ms_shi = timed_region(step_shard, first, instrumented=True)
        first += args.steps
        ks = fv.timing_read()
        variants["causal_shard"] = {
            "ms_per_step": ms_sh, "value": w.B * w.H * ls / (ms_sh / 1e3),
            "ms_per_step_instrumented": ms_shi,
            "what": f"ORF draw + causal pass over tokens {w.L - ls}..{w.L - 1} (one GPU's share "
                    "of 8 along the sequence) from the state of the tokens before them",
            "kernels": {k: {"ms_per_launch": v[0] / v[1]} for k, v in ks.items() if v[1] > 0}}

    # the random-feature draw of the step (8 heads x M rows) for every kind of features
    if "draws" in chosen:
        kinds = {"ortho_chi": fv.RF_ORTHO_CHI, "ortho_fixed": fv.RF_ORTHO_FIXED,
                 "iid": fv.RF_IID, "hadamard": fv.RF_HADAMARD, "givens": fv.RF_GIVENS}
        draws = {}
        for name, kind in kinds.items():
            step_d = lambda i, k=kind: fv.orf_draw(1000 + i, H, M, w.d, kind=k, W=Wd[0], b=bd[0],
                                                   stream=s_main)
            for i in range(args.warmup):
                step_d(first + i)
            first += args.warmup
            # wall time per call (a short draw is bound by the host's launch rate)
            # and the draw kernel's own duration from the events around its launch
            draws[name] = {"ms_per_draw": timed_region(step_d, first)}
            first += args.steps
            timed_region(step_d, first, instrumented=True)
            kd = fv.timing_read()
            first += args.steps
            tot, cnt = (sum(v[0] for v in kd.values()), sum(v[1] for v in kd.values()))
            draws[name]["ms_per_launch"] = tot / cnt if cnt else None
            draws[name]["kernel"] = ",".join(sorted(k for k, v in kd.items() if v[1] > 0))
        variants["draws"] = draws

    # the step captured once as a HIP graph and replayed (the library launches only
    # kernels, so a whole step is capturable); each replay redoes the draw, with the
    # seed captured. The launch-bound smallest configuration (B1 H1 L1024, fp32)
    # shows what the capture saves in host launch time.
    if "graph" in chosen:
        def capture(step):
            side = torch.cuda.Stream()   # default priority
            side.wait_stream(s_main)
            with torch.cuda.stream(side):
                step()
            s_main.wait_stream(side)
            gr = torch.cuda.CUDAGraph()
            with torch.cuda.graph(gr):
                step()
            torch.cuda.synchronize()
            return gr

        def replays(gr):
            for _ in range(args.warmup):
                gr.replay()
            return time_steps(torch, fv, s_main, lambda i: gr.replay(), 0, args.steps)

        def captured_step():
            fv.orf_draw(1000 + first, H, M, w.d, W=Wd[0], b=bd[0])
            attention(0, stream=torch.cuda.current_stream())

        gr = capture(captured_step)
        ms_g = replays(gr)
        del gr
        w_small = wl.WORKLOADS["bidir_small"]
        q1, k1, v1 = (torch.from_numpy(x).to(dev) for x in wl.make_qkv(w_small))
        W1 = torch.empty((w_small.H, w_small.M, w_small.d), dtype=torch.float32, device=dev)
        b1 = torch.empty((w_small.H, w_small.M), dtype=torch.float32, device=dev)
        o1 = torch.empty_like(q1)
        g1 = fv.make_desc(w_small.B, w_small.H, w_small.L, w_small.d, w_small.M, fv.F32,
                          fv.F32, w_small.input_scale)
        wk1 = torch.empty(fv.workspace_size(g1, 0), dtype=torch.uint8, device=dev)

        def small_step(i=0):
            fv.orf_draw(77, w_small.H, w_small.M, w_small.d, W=W1, b=b1)
            fv.attn_bidir(q1, k1, v1, W1, b1, w_small.input_scale, out=o1, workspace=wk1)

        for i in range(args.warmup):
            small_step()
        ms_small = time_steps(torch, fv, s_main, small_step, 0, args.steps)
        gr = capture(small_step)
        ms_small_g = replays(gr)
        del gr
        variants["graph"] = {
            "ms_per_step": ms_g, "value": w.B * w.H * w.L / (ms_g / 1e3),
            "what": "the step (ORF draw + " + w.direction + " attention) captured once as a "
                    "HIP graph and replayed; each replay redoes the draw with the seed captured",
            "small": {"workload": "bidir_small (B1 H1 L1024 M128 fp32, draw + bidirectional)",
                      "ms_per_step_eager": ms_small, "ms_per_step_graph": ms_small_g}}

    # the backward pass of the step's attention: gradients with respect to Q, K, V of
    # each direction the step computes, for a fixed synthetic upstream gradient; the
    # draw stays in the step. "backward": the gradient calls alone, each recomputing
    # its forward quantities. "train_step": the forward pass saving each row's
    # 1 / (D-hat + eps), then the gradient calls reading the saved outputs and scales.
    # Both directions take one favor_attn_both_backward call, with an upstream
    # gradient of its own for each output.
    directions = {0: "bidirectional", 1: "causal", 2: "bidirectional and causal"}[op]
    if chosen & {"backward", "train_step"}:
        rng = np.random.default_rng(7)
        dO = torch.from_numpy(rng.standard_normal(Q.shape, dtype=np.float32)).to(
            device=dev, dtype=tdt).contiguous()
        dO2 = torch.from_numpy(rng.standard_normal(Q.shape, dtype=np.float32)).to(
            device=dev, dtype=tdt).contiguous()   # the causal output's gradient (both)
        grads = [torch.empty_like(Qd) for _ in range(3)]
        nbw = fv.backward_workspace_size(g, {0: False, 1: True, 2: 2}[op])
        wsb = torch.empty(nbw, dtype=torch.uint8, device=dev)
        rs_b = torch.empty((w.B, H, w.L), dtype=torch.float32, device=dev)
        rs_c = torch.empty_like(rs_b)

        fwd_call = {0: "bidir", 1: "causal", 2: "both"}[op]

        def gradients(saved):
            # saved: the forward call just ran with row scales; its outputs, row
            # scales and workspace (Buf1, segment prefixes, W'') are read back
            gq, gk, gv = grads
            fwd = dict(forward_workspace=ws, forward_call=fwd_call) if saved else {}
            if op == 2:
                # one call for both directions: a single dK, dV pass over the
                # bidirectional dBuf1 plus the causal suffix states
                sv = dict(out_bidir=out_b, row_scale_bidir=rs_b, out_causal=out_c,
                          row_scale_causal=rs_c) if saved else {}
                fv.attn_both_backward(Qd, Kd, Vd, Wd[0], bd[0], s, dO, dO2, dQ=gq, dK=gk,
                                      dV=gv, workspace=wsb, stream=s_main, **sv, **fwd)
                return
            if op != 1:
                fv.attn_bidir_backward(Qd, Kd, Vd, Wd[0], bd[0], s, dO, dQ=gq, dK=gk, dV=gv,
                                       workspace=wsb, stream=s_main,
                                       out=out_b if saved else None,
                                       row_scale=rs_b if saved else None, **fwd)
            if op != 0:
                fv.attn_causal_backward(Qd, Kd, Vd, Wd[0], bd[0], s, dO, dQ=gq, dK=gk, dV=gv,
                                        workspace=wsb, stream=s_main,
                                        out=out_c if saved else None,
                                        row_scale=rs_c if saved else None, **fwd)

        def step_bwd(i):
            fv.orf_draw(1000 + i, H, M, w.d, W=Wd[0], b=bd[0], stream=s_main)
            gradients(False)

        def step_train(i):
            fv.orf_draw(1000 + i, H, M, w.d, W=Wd[0], b=bd[0], stream=s_main)
            if op == 2:
                fv.attn_both(Qd, Kd, Vd, Wd[0], bd[0], s, out_bidir=out_b, out_causal=out_c,
                             workspace=ws, stream=s_main, row_scale_bidir=rs_b,
                             row_scale_causal=rs_c)
            elif op == 0:
                fv.attn_bidir(Qd, Kd, Vd, Wd[0], bd[0], s, out=out_b, workspace=ws,
                              stream=s_main, row_scale=rs_b)
            else:
                fv.attn_causal(Qd, Kd, Vd, Wd[0], bd[0], s, out=out_c, workspace=ws,
                               stream=s_main, row_scale=rs_c)
            gradients(True)

        for name, step_v, what in (
                ("backward", step_bwd, "ORF draw + gradients of " + directions
                 + " attention with respect to Q, K, V (forward recomputed inside)"),
                ("train_step", step_train, "ORF draw + " + directions + " attention saving "
                 "the row scales + gradients with respect to Q, K, V from the saved outputs, "
                 "row scales and forward workspace")):
            if name not in chosen:
                continue
            for i in range(args.warmup):
                step_v(first + i)
            first += args.warmup
            ms_b = timed_region(step_v, first)
            first += args.steps
            ms_bi = timed_region(step_v, first, instrumented=True)
            first += args.steps
            kb = fv.timing_read()
            variants[name] = {
                "ms_per_step": ms_b, "value": w.B * w.H * w.L / (ms_b / 1e3),
                "ms_per_step_instrumented": ms_bi, "what": what,
                "kernels": {k: {"ms_per_launch": v[0] / v[1],
                                "launches_per_step": v[1] / args.steps}
                            for k, v in kb.items() if v[1] > 0}}

    token_heads = w.B * w.H * w.L
    value = token_heads / (ms_step / 1e3)
    roof = roofline(kernels, w, token_heads)

    peaks = None if args.no_peaks else measured_peaks(torch, fv)
    feature_map = None
    if not args.no_feature_map:
        feature_map = bench_feature_map(w, Qd, Wd[0], bd[0], args, torch, fv)
    # the other workloads of the configuration list, each at its full size
    others = {}
    names = [n for n in args.workloads.split(",") if n and n != w.name]
    if names:
        del Wd, bd, out_b, out_c, ws, Qd, Kd, Vd
        for name in names:
            causal = wl.WORKLOADS[name].direction != "bidir"
            rows = (0, 1024, 4096) if name == "causal_b8h8" else (0,)
            first = args.chunk or default_chunk(wl.WORKLOADS[name])
            chunks = (args.chunk, 64 if first == 32 else 32) if causal else (0,)
            others[name] = bench_workload(name, args, torch, fv, segment_rows=rows,
                                          chunks=chunks)

    res = {
        "metric": "FAVOR attention tokens/sec (B*H*L/s) + % of MFMA/HBM peak at L=8192, M=256",
        "value": value,
        "unit": "token-heads/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "H": w.H, "L": w.L, "d": w.d, "M": M,
                   "direction": w.direction, "orf_draw_per_step": True,
                   "causal_segment_rows": args.segment or "library default",
                   "causal_chunk_tokens": args.chunk or default_chunk(w),
                   "orf_draw": "drawn in line before the attention pass, same stream",
                   "parallelism": "single GPU"},
        "kernels": kernels,
        "warmup_steps_run": n_warm,
        "ms_per_step_pipelined": ms_step_pipelined,
        "ms_per_step_instrumented": ms_step_instrumented,
        "roofline": roof,
        "measured_peaks": peaks,
        "feature_map": feature_map,
        "workloads": others,
        "variants": variants,
    }
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(w, Q, K, V)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
