#!/usr/bin/env python3
"""Throughput of the masked second-order HLA hot path on one MI355X.

One step = one hla2_forward over the whole batch of the workload (per-chunk
summaries, the semidirect-product scan and the readout), inputs resident in
HBM.  Prints ONE JSON line with tokens/s, a roofline entry for the kernel that
takes the most time, and the CPU oracle timed on the host cores.

  python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--algo auto|chunked|fused]
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
BF16_MFMA_PEAK_TFLOPS = 2500.0  # dense bf16 MFMA
FP32_VALU_PEAK_TFLOPS = 157.3   # fp32 vector

DEFAULT_WORKLOAD = "hla2-masked-normalized-bf16-B2H32-n16384-d128-C128"
SUB_WORKLOAD = "hla2-masked-bf16-B4H16-n4096-d64-C64"
FLUSH_BYTES = 512 << 20          # written between cold iterations: twice the 256 MB last-level cache


def kernel_costs(w, P=None, tile=None, first=None, per=None, two_pass=False):
    """Algorithmic cost of one launch of each kernel of the forward path:
    {name: (bound, bytes, flops)}.  bytes = HBM bytes the kernel must move
    (inputs read once, outputs written once); flops = useful arithmetic of
    the kernel's formulation (a dense C x C product counts C^2 per output
    element; triangles are not halved).  P = segments per head, tile = the
    token tile, first / per = the tiles of segment 0 / of each later segment
    of the fused path's plan (from the library); two_pass: the plan that walks
    segment 0 beside the summary walks and then the other segments' output."""
    B, H, n, d, dv, C = w["B"], w["H"], w["n"], w["d"], w["dv"], w["chunk"]
    BH = B * H
    M = -(-n // C)
    es = 2 if w["dist"] == "unit" else 4
    F = d * d + 2 * d * dv + 2 * d
    tok = BH * n
    qkv_tok = (2 * d + dv) * es
    costs = {
        # general path
        "chunk_summary": ("alu", tok * qkv_tok + BH * M * F * 4, tok * 2 * (C * d / 2 + C * dv / 2 + d * d + 2 * d * dv)),
        "readout": ("alu", tok * (qkv_tok + 4 * dv) + BH * M * F * 4,
                    tok * 2 * (d * d + 1.5 * C * d + 2 * d * dv + C * dv / 2)),
        "scan": ("hbm", 2 * BH * M * F * 4, BH * M * 2 * (d * d * dv + d * d)),
    }
    if P:
        Ct = tile
        cps = per or -(-(-(-n // Ct)) // P)
        sum_tok = BH * min(n, (P - 1) * cps * Ct)
        costs.update({
            # fused path: the output walk reads q/k/v once and writes out once
            # (the carry records it also reads are this design's own traffic).
            # flops: the dense count of the chunk form at the tile the walk runs
            "walk": ("hbm", tok * (qkv_tok + 4 * dv), tok * reference_flops_per_token(Ct, d, dv)),
            "walk_summary": ("hbm", sum_tok * qkv_tok + BH * (P - 1) * F * 4,
                             sum_tok * 2 * (2 * Ct * d + 2 * d * d + 2 * d * dv + d * dv)),
            # segment moments: k read once, S = K^T K per segment written
            "moments": ("hbm", tok * d * es + BH * P * d * d * 4, tok * 2 * d * d),
            # carry fix-up: q read, out read and written (den read when normalised)
            "fix": ("hbm", tok * (d * es + 8 * dv + (4 if w["normalized"] else 0)), tok * 2 * d * dv),
            # carry: the segments' Phi/eta brackets read, their running sums written
            "carry": ("hbm", BH * (2 * P + 1) * (d * dv + d) * 4, BH * P * (d * dv + d)),
            # running sums of the per-segment records (S, or the Phi/eta brackets): read once, written once
            "seg_prefix": ("hbm", BH * 2 * P * (d * d + d * dv + d) * 4, BH * P * (d * d + d * dv + d)),
            "init_convert": ("hbm", BH * 2 * F * 4, BH * 2 * (d * d * dv + d * d)),
            "total": ("hbm", BH * (P + 2) * F * 4, BH * 2 * (d * d * dv + d * d)),
        })
        if two_pass and P > 1:
            # launch 1: segment 0's output walk and the summary walks of
            # segments 1 .. P-2 (which also form C = Q^T V); launch 2: the
            # output walks of segments 1 .. P-1
            seg0 = BH * min(n, first * Ct)
            summ = BH * min(n, (first + (P - 2) * cps) * Ct) - seg0
            out_tok = tok - seg0
            ref = reference_flops_per_token(Ct, d, dv)
            costs.update({
                "walk": ("hbm", out_tok * (qkv_tok + 4 * dv), out_tok * ref),
                "walk_first": ("hbm", seg0 * (qkv_tok + 4 * dv) + summ * qkv_tok + BH * (P - 1) * F * 4,
                               seg0 * ref + summ * 2 * (2 * Ct * d + 2 * d * d + 2 * d * dv)),
                # the S prefixes of segments 1 .. P-1 (the S of records 0 .. P-2 read,
                # the prefixes written) and the brackets: C, m and (Phi, eta) read,
                # (Phi, eta) written
                "bracket": ("hbm", BH * (2 * (P - 1) * d * d + (P - 2) * (d * dv + d + 2 * (d * dv + d))) * 4,
                            BH * (P - 2) * 2 * (d * d * dv + d * d)),
                # one prefix launch: the running sums of the (Phi, eta) brackets
                "seg_prefix": ("hbm", BH * 2 * P * (d * dv + d) * 4, BH * P * (d * dv + d)),
            })
    return costs


def reference_flops_per_token(C, d, dv):
    """Dense flop count per token of the chunk form with chunk C (no triangle
    discount): 2 (C^2 + 2 C d + 2 C dv + 2 d^2 + 4 d dv)."""
    return 2 * (C * C + 2 * C * d + 2 * C * dv + 2 * d * d + 4 * d * dv)


def peak_for(bound):
    if bound == "hbm":
        return HBM_PEAK_GBS, "GB/s"
    if bound == "mfma":
        return BF16_MFMA_PEAK_TFLOPS, "TFLOP/s"
    return FP32_VALU_PEAK_TFLOPS, "TFLOP/s"


def traffic_for(kernel, workload):
    """HBM traffic per launch from the committed counter summary, if it was
    taken on the current kernel source; else None."""
    path = os.path.join(ROOT, "profiles", "hbm_traffic.json")
    if not os.path.exists(path):
        return None
    try:
        rec = json.load(open(path))
    except Exception:
        return None
    e = rec.get(workload, {}).get(kernel)
    if not e:
        return None
    if e.get("source_sha") != source_sha():
        return None
    return e.get("bytes_per_launch")


def kernel_key(name):
    """Bench name of a library kernel from its (demangled) dispatch name."""
    if "k_ahla_walk" in name:
        return "ahla_walk"
    if "k_la<" in name or "k_laI" in name:
        return "bwd_pass"
    if "k_walk_ws_first" in name:
        return "walk_first"
    if "k_ws_bracket" in name:
        return "bracket"
    if "k_walk" in name:
        return "walk_summary" if ("true" in name or "Lb1E" in name) else "walk"
    for key in ("k_init_convert", "k_total", "k_moments", "k_carry", "k_fix", "k_scan", "k_chunk_summary", "k_readout",
                "k_step", "k_seg_prefix"):
        if key in name:
            return key[2:]
    return None


def ingest_counters(workload, fetch_csv, write_csv, copy_fetch_csv, copy_write_csv, copy_bytes):
    """Per-launch HBM bytes of each kernel from two rocprofv3 --pmc runs
    (FETCH_SIZE, WRITE_SIZE; KiB per dispatch), each scaled by what the same
    counter reads for a plain copy of copy_bytes bytes.  Updates
    profiles/hbm_traffic.json under the workload, keyed by the source hash."""
    import csv
    import collections

    def per_kernel(path):
        acc = collections.defaultdict(list)
        for r in csv.DictReader(open(path)):
            acc[r["Kernel_Name"]].append(float(r["Counter_Value"]))
        return acc

    def copy_kib(path):
        vals = [v for name, vs in per_kernel(path).items() if kernel_key(name) is None for v in vs]
        return max(vals)

    f_scale = copy_bytes / (copy_kib(copy_fetch_csv) * 1024)
    w_scale = copy_bytes / (copy_kib(copy_write_csv) * 1024)
    fetch, write = per_kernel(fetch_csv), per_kernel(write_csv)
    out = {}
    for name, vals in fetch.items():
        key = kernel_key(name)
        if key is None or name not in write:
            continue
        fb = sum(vals) / len(vals) * 1024 * f_scale
        wb = sum(write[name]) / len(write[name]) * 1024 * w_scale
        out[key] = {"bytes_per_launch": fb + wb, "fetch_bytes": fb, "write_bytes": wb,
                    "dispatches": len(vals), "source_sha": source_sha(),
                    "fetch_scale": f_scale, "write_scale": w_scale}
    path = os.path.join(ROOT, "profiles", "hbm_traffic.json")
    rec = json.load(open(path)) if os.path.exists(path) else {}
    rec[workload] = out
    with open(path, "w") as fh:
        json.dump(rec, fh, indent=1, sort_keys=True)
    print(json.dumps({workload: out}, indent=1))


# Sources the fused forward's kernels (moments, walk, carry, fix-up) are built
# from: the HBM counter summary is used only while these hash as recorded.
FORWARD_SOURCES = ("fused.hip", "fused_ws.h", "fused_tiles.h", "fused.h", "common.h", "profile.h")


def source_sha():
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2510_27258_amd", "csrc")
    for f in FORWARD_SOURCES:
        h.update(open(os.path.join(csrc, f), "rb").read())
    return h.hexdigest()[:16]


def cpu_model():
    """The host CPU's model name (lscpu, else /proc/cpuinfo)."""
    import subprocess
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in out.splitlines():
            if line.startswith("Model name:"):
                return line.split(":", 1)[1].strip()
    except Exception:
        pass
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except Exception:
        pass
    return "unknown"


def cpu_baseline(w, q, k, v, budget_s=20.0, min_s=10.0, one_thread_s=4.0):
    """The C oracle (serial fp64 recurrence, heads over OpenMP threads) on the
    host cores, on as many whole heads of the workload as fit the budget; the
    sample is repeated until it has run for at least min_s seconds, so short
    samples are timed over several passes.  Also one thread on one head, for
    the per-core rate.  Inputs are converted to fp64 before the clock starts."""
    from oracle import native
    B, H, n = w["B"], w["H"], w["n"]
    threads = os.cpu_count() or 1
    qs = q.reshape(B * H, n, -1)
    ks = k.reshape(B * H, n, -1)
    vs = v.reshape(B * H, n, -1)
    # one thread, one head (repeated to one_thread_s); also sizes the sample
    import numpy as np
    q1, k1, v1 = (np.ascontiguousarray(x[:1], dtype=np.float64) for x in (qs, ks, vs))
    passes1 = 0
    t0 = time.perf_counter()
    while True:
        native.hla2_serial_c(q1, k1, v1, masked=bool(w["masked"]), threads=1, return_state=False)
        passes1 += 1
        dt1 = time.perf_counter() - t0
        if dt1 >= one_thread_s or passes1 >= 1000:
            break
    per_head = max(dt1 / passes1, 1e-6)
    heads = int(min(B * H, max(1, budget_s * threads / per_head / 2)))
    heads = max(min(heads, B * H), min(threads, B * H))
    import numpy as np
    qh, kh, vh = (np.ascontiguousarray(x[:heads], dtype=np.float64) for x in (qs, ks, vs))
    passes, used = 0, 1
    t0 = time.perf_counter()
    while True:
        _, _, _, used = native.hla2_serial_c(qh, kh, vh, masked=bool(w["masked"]),
                                             threads=threads, return_state=False)
        passes += 1
        dt = time.perf_counter() - t0
        if dt >= min_s or passes >= 1000:
            break
    return {"value": passes * heads * n / dt, "unit": "tokens/s", "cores": int(used), "kind": "oracle",
            "cpu_model": cpu_model(), "nproc": threads,
            "one_thread": {"value": passes1 * n / dt1, "unit": "tokens/s", "sample": f"1 head x {n} tokens, "
                           f"{passes1} passes in {dt1:.2f} s"},
            "sample": f"{heads} of {B * H} heads x {n} tokens, C fp64 serial recurrence, {passes} passes "
                      f"in {dt:.2f} s on {int(used)} threads"}


def stats_ms(xs):
    """median, p10, p90 and mean of a list of per-iteration times (ms)."""
    import numpy as np
    a = np.asarray(xs, dtype=np.float64)
    return {"median_ms": float(np.median(a)), "p10_ms": float(np.percentile(a, 10)),
            "p90_ms": float(np.percentile(a, 90)), "mean_ms": float(a.mean()), "iters": int(a.size)}


def time_iters(fn, iters, cold=False, clean=False):
    """Per-iteration HIP-event times of fn() on the current stream.  cold:
    a FLUSH_BYTES buffer is written before each iteration (outside its
    events), so the 256 MB last-level cache holds none of fn's inputs but is
    full of dirty lines, whose write-back fn's own traffic then pays for (the
    pessimistic case).  clean (with cold): the buffer is read instead, which
    leaves the cache holding clean lines of no use to fn, so fn's writes may
    stay in it past the timed region (the optimistic case)."""
    import torch
    flush = torch.ones(FLUSH_BYTES // 4, dtype=torch.float32, device="cuda") if cold else None
    sink = torch.empty((), dtype=torch.float32, device="cuda") if cold else None
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(iters)]
    torch.cuda.synchronize()
    for a, b in ev:
        if cold and clean:
            torch.sum(flush, dim=0, out=sink)
        elif cold:
            flush.fill_(1.0)
        a.record()
        fn()
        b.record()
    torch.cuda.synchronize()
    return [a.elapsed_time(b) for a, b in ev]


def measure_scan(name, iters=50):
    """The semidirect-product scan kernel alone over the per-chunk summaries of
    a workload (chunk states from hla2_chunk_summaries): reads every chunk
    state and writes its exclusive prefix and the total.  Warm (repeated on one
    input) and cold (last-level cache flushed before each launch)."""
    import torch
    import paper_2510_27258_amd as hla
    from paper_2510_27258_amd import inputs as I
    w = I.WORKLOADS[name]
    q, k, v, code = I.draw_qkv(w["B"], w["H"], w["n"], w["d"], w["dv"], w["dist"], w["seed"])
    qd, kd, vd = (I.to_torch(x, code, "cuda") for x in (q, k, v))
    del q, k, v
    d, dv = w["d"], w["dv"]
    states = hla.chunk_summaries(qd, kd, vd, w["chunk"])
    del qd, kd, vd
    hla.scan(states, d, dv)
    torch.cuda.synchronize()
    B, H, M, F = states.shape
    nbytes = 2 * states.numel() * 4 + B * H * F * 4
    rec = {"kernel": "scan", "workload": name, "states": B * H * M, "algorithmic_bytes": nbytes, "unit": "GB/s",
           "peak": HBM_PEAK_GBS}
    for mode in ("warm", "cold", "cold_clean"):
        st = stats_ms(time_iters(lambda: hla.scan(states, d, dv), iters, cold=(mode != "warm"),
                                 clean=(mode == "cold_clean")))
        gbs = nbytes / st["median_ms"] / 1e6
        rec[mode] = dict(st, achieved=gbs, frac=gbs / HBM_PEAK_GBS)
    del states
    torch.cuda.empty_cache()
    return rec


def measure_hla3(reps=20, masked=True):
    """hla3_forward on the third-order workload (B1 H8 n2048 d=dv=16, fp32,
    chunk 32), masked or unmasked: tokens/s by HIP events, and per-kernel
    times."""
    import torch
    import paper_2510_27258_amd as hla
    from paper_2510_27258_amd import capi
    from paper_2510_27258_amd import inputs as I
    name = "hla3-masked-fp32-B1H8-n2048-d16-C32"
    w = I.WORKLOADS[name]
    q, k, v, code = I.draw_qkv(w["B"], w["H"], w["n"], w["d"], w["dv"], w["dist"], w["seed"])
    dev = torch.device("cuda:0")
    qd, kd, vd = (I.to_torch(x, code, dev) for x in (q, k, v))
    out = torch.empty(w["B"], w["H"], w["n"], w["dv"], dtype=torch.float32, device=dev)
    wsb = capi.hla3_workspace_bytes(w["B"], w["H"], w["n"], w["d"], w["dv"], w["chunk"], code)
    ws = torch.empty(max(wsb, 1), dtype=torch.uint8, device=dev)
    run = lambda: hla.hla3_forward(qd, kd, vd, w["chunk"], masked=masked, out=out, workspace=ws)
    for _ in range(3):
        run()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        run()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    capi.hla_profile_begin(8 * reps + 8)
    for _ in range(reps):
        run()
    torch.cuda.synchronize()
    prof = capi.hla_profile_summary()
    capi.hla_profile_end()
    tokens = w["B"] * w["H"] * w["n"]
    if not masked:
        name = name.replace("masked", "unmasked")
    return {"workload": name, "value": tokens / (ms / 1e3), "unit": "tokens/s", "ms": ms, "dtype": "f32",
            "kernels_ms": {k_: v_[1] / v_[0] for k_, v_ in prof.items()}}


def measure_decay(reps=10):
    """hla2_forward_decay on the decayed workload (B4 H16 n4096 d=dv=64, bf16,
    chunk 64, gamma 0.99): tokens/s by HIP events, per-kernel times, and the
    fused walk against HBM (q, k, v read once, out written once) and against
    the bf16 MFMA peak with the undecayed dense reference flop count."""
    import torch
    import paper_2510_27258_amd as hla
    from paper_2510_27258_amd import capi
    from paper_2510_27258_amd import inputs as I
    name = "hla2-decay-bf16-B4H16-n4096-d64-C64"
    w = I.WORKLOADS[name]
    q, k, v, code = I.draw_qkv(w["B"], w["H"], w["n"], w["d"], w["dv"], w["dist"], w["seed"])
    dev = torch.device("cuda:0")
    qd, kd, vd = (I.to_torch(x, code, dev) for x in (q, k, v))
    out = torch.empty(w["B"], w["H"], w["n"], w["dv"], dtype=torch.float32, device=dev)
    wsb = capi.hla2_forward_decay_workspace_bytes(w["B"], w["H"], w["n"], w["d"], w["dv"], w["chunk"], code)
    ws = torch.empty(max(wsb, 1), dtype=torch.uint8, device=dev)
    run = lambda: hla.forward_decay(qd, kd, vd, w["chunk"], w["gamma"], out=out, workspace=ws)
    for _ in range(3):
        run()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        run()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    capi.hla_profile_begin(8 * reps + 8)
    for _ in range(reps):
        run()
    torch.cuda.synchronize()
    prof = capi.hla_profile_summary()
    capi.hla_profile_end()
    kms = {k_: v_[1] / v_[0] for k_, v_ in prof.items()}
    B, H, n, d, dv, C = w["B"], w["H"], w["n"], w["d"], w["dv"], w["chunk"]
    tokens = B * H * n
    nbytes = tokens * (2 * (2 * d + dv) + 4 * dv)
    flops = tokens * reference_flops_per_token(C, d, dv)
    s = kms["walk"] / 1e3
    return {"workload": name, "value": tokens / (ms / 1e3), "unit": "tokens/s", "ms": ms, "dtype": "bf16",
            "gamma": w["gamma"], "kernels_ms": kms,
            "roofline": {"kernel": "walk", "bound": "hbm", "achieved": nbytes / s / 1e9, "peak": HBM_PEAK_GBS,
                         "unit": "GB/s", "frac": nbytes / s / 1e9 / HBM_PEAK_GBS, "algorithmic_bytes": nbytes,
                         "algorithmic_flops": flops, "mfma_tflops": flops / s / 1e12,
                         "mfma_frac": flops / s / 1e12 / BF16_MFMA_PEAK_TFLOPS}}


def ahla_flops_per_token(C, d, dv):
    """Dense flop count per token of the AHLA chunk form with tile C (no
    triangle discount): A = Q K^T (C d), R = A V + Q P0 (C dv + d dv),
    O = A R + Q E0 (C dv + d dv), P0 += K^T V and E0 += K^T R (2 d dv)."""
    return 2 * (C * d + 2 * C * dv + 4 * d * dv)


def measure_ahla(reps=10):
    """ahla_forward on the AHLA workload (B4 H16 n4096 d=dv=64, bf16, chunk
    64): tokens/s by HIP events, per-kernel times, and the walk against HBM
    (q, k, v read once, out written once) and against the bf16 MFMA peak with
    the dense chunk-form flop count."""
    import torch
    import paper_2510_27258_amd as hla
    from paper_2510_27258_amd import capi
    from paper_2510_27258_amd import inputs as I
    name = "ahla-bf16-B4H16-n4096-d64-C64"
    w = I.WORKLOADS[name]
    q, k, v, code = I.draw_qkv(w["B"], w["H"], w["n"], w["d"], w["dv"], w["dist"], w["seed"])
    dev = torch.device("cuda:0")
    qd, kd, vd = (I.to_torch(x, code, dev) for x in (q, k, v))
    out = torch.empty(w["B"], w["H"], w["n"], w["dv"], dtype=torch.float32, device=dev)
    wsb = capi.ahla_workspace_bytes(w["B"], w["H"], w["n"], w["d"], w["dv"], w["chunk"], code)
    ws = torch.empty(max(wsb, 1), dtype=torch.uint8, device=dev)
    run = lambda: hla.ahla_forward(qd, kd, vd, w["chunk"], out=out, workspace=ws)
    for _ in range(3):
        run()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        run()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    capi.hla_profile_begin(8 * reps + 8)
    for _ in range(reps):
        run()
    torch.cuda.synchronize()
    prof = capi.hla_profile_summary()
    capi.hla_profile_end()
    kms = {k_: v_[1] / v_[0] for k_, v_ in prof.items()}
    B, H, n, d, dv = w["B"], w["H"], w["n"], w["d"], w["dv"]
    tokens = B * H * n
    nbytes = tokens * (2 * 2 * d + 2 * dv + 4 * dv)
    flops = tokens * ahla_flops_per_token(64, d, dv)
    s = kms["ahla_walk"] / 1e3
    return {"workload": name, "value": tokens / (ms / 1e3), "unit": "tokens/s", "ms": ms, "dtype": "bf16",
            "kernels_ms": kms,
            "roofline": {"kernel": "ahla_walk", "bound": "hbm", "achieved": nbytes / s / 1e9, "peak": HBM_PEAK_GBS,
                         "unit": "GB/s", "frac": nbytes / s / 1e9 / HBM_PEAK_GBS, "algorithmic_bytes": nbytes,
                         "algorithmic_flops": flops, "mfma_tflops": flops / s / 1e12,
                         "mfma_frac": flops / s / 1e12 / BF16_MFMA_PEAK_TFLOPS}}


# Per-token HBM bytes / d of each launch of the backward: x, y, z read (bf16
# 2 B or fp32 4 B per element; the r pass also reads v, for the v^T r moments
# of its output), the output written (4 B), and read back (4 B) when the pass
# adds to it; a launch of several passes side by side counts them all.
BWD_PASS_BYTES = {"bwd_ru": [(2 + 2 + 2 + 2 + 4) + (2 + 4 + 2 + 4)],
                  "bwd_dq_dv_dk": [(4 + 2 + 4 + 4) + (4 + 2 + 4 + 4) + (2 + 2 + 4 + 4)],
                  "bwd_dq": [4 + 2 + 2 + 8]}


def measure_backward(reps=10):
    """hla2_backward on the B4 H16 n4096 d=dv=64 bf16 shape (upstream gradient
    fp32): gradient tokens/s by HIP events, per-pass times, and the slowest pass
    against HBM (its operands read once, its output written once) and against
    the bf16 MFMA peak with the dense first-order chunk-form count
    2 (2 C d + 2 d^2) per token."""
    import torch
    import paper_2510_27258_amd as hla
    from paper_2510_27258_amd import capi
    from paper_2510_27258_amd import inputs as I
    name = "hla2-masked-bf16-B4H16-n4096-d64-C64"
    w = I.WORKLOADS[name]
    B, H, n, d = w["B"], w["H"], w["n"], w["d"]
    q, k, v, code = I.draw_qkv(B, H, n, d, w["dv"], w["dist"], w["seed"])
    dev = torch.device("cuda:0")
    qd, kd, vd = (I.to_torch(x, code, dev) for x in (q, k, v))
    g = torch.from_numpy(I.draw_grad(B, H, n, w["dv"], 1)).to(dev)
    wsb = capi.hla2_backward_workspace_bytes(B, H, n, d, w["dv"], w["chunk"], code)
    ws = torch.empty(max(wsb, 1), dtype=torch.uint8, device=dev)
    run = lambda: hla.backward(qd, kd, vd, g, w["chunk"], workspace=ws)
    for _ in range(3):
        run()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        run()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    capi.hla_profile_begin(32 * reps + 8)
    for _ in range(reps):
        run()
    torch.cuda.synchronize()
    prof = capi.hla_profile_summary()
    capi.hla_profile_end()
    kms = {k_: v_[1] / v_[0] for k_, v_ in prof.items()}
    tokens = B * H * n
    dom = max((k_ for k_ in kms if k_ in BWD_PASS_BYTES), key=lambda k_: kms[k_])
    nbytes = tokens * d * sum(BWD_PASS_BYTES[dom]) / len(BWD_PASS_BYTES[dom])
    flops = tokens * 2 * (2 * 64 * d + 2 * d * d)
    s = kms[dom] / 1e3
    return {"workload": name + " backward", "value": tokens / (ms / 1e3), "unit": "tokens/s", "ms": ms,
            "dtype": "bf16", "kernels_ms": kms,
            "roofline": {"kernel": dom, "bound": "hbm", "achieved": nbytes / s / 1e9, "peak": HBM_PEAK_GBS,
                         "unit": "GB/s", "frac": nbytes / s / 1e9 / HBM_PEAK_GBS, "algorithmic_bytes": nbytes,
                         "algorithmic_flops": flops, "mfma_tflops": flops / s / 1e12,
                         "mfma_frac": flops / s / 1e12 / BF16_MFMA_PEAK_TFLOPS}}


def measure_decode(steps=None):
    """hla2_step on the decode workload: state from a prefill of the seeded
    2048-token prefix, then the seeded step tokens, one launch per step."""
    import numpy as np
    import torch
    import paper_2510_27258_amd as hla
    from paper_2510_27258_amd import capi
    from paper_2510_27258_amd import inputs as I
    w = I.WORKLOADS["hla2-decode-bf16-B64H32-d128-prefix2048-steps1024"]
    B, H, d, dv, n = w["B"], w["H"], w["d"], w["dv"], w["n"]
    steps = steps or w["steps"]
    dev = torch.device("cuda:0")
    state = hla.State(B, H, d, dv, dtype=torch.bfloat16, device=dev)
    # prefix in batch slices to bound host memory; draws follow the seeded recipe per slice
    q, k, v, code = I.draw_qkv(B, H, n, d, dv, w["dist"], w["seed"])
    qd, kd, vd = (I.to_torch(x, code, dev) for x in (q, k, v))
    del q, k, v
    hla.prefill(state, qd, kd, vd, w["chunk"], want_out=False)
    del qd, kd, vd
    qs, ks, vs, _ = I.draw_qkv(B, H, steps, d, dv, w["dist"], w["step_seed"])
    qsd, ksd, vsd = (I.to_torch(x, code, dev).permute(2, 0, 1, 3).contiguous() for x in (qs, ks, vs))
    del qs, ks, vs
    outs = torch.empty(steps, B, H, dv, dtype=torch.float32, device=dev)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for t in range(steps):
        hla.step(state, qsd[t], ksd[t], vsd[t], out=outs[t])
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    # the state is read and written once (S packed symmetric), tokens read, output written
    per_head = 2 * capi.hla2_state_bytes(1, 1, d, dv) + (2 * d + dv) * 2 + dv * 4
    nbytes = B * H * per_head
    return {"workload": "hla2-decode-bf16-B64H32-d128-prefix2048-steps1024", "steps": steps, "ms_per_step": ms,
            "achieved": nbytes / ms / 1e6, "unit": "GB/s", "peak": HBM_PEAK_GBS,
            "frac": nbytes / ms / 1e6 / HBM_PEAK_GBS, "bytes_per_step": nbytes}


def measure_forward(name, steps, warmup, algo_name="auto", cold_iters=0):
    """Forward throughput on a named workload: `steps` back-to-back forwards
    bracketed by synchronisations (tokens/s), per-iteration HIP-event times
    (median, p10, p90), optionally cold iterations (last-level cache flushed
    before each), per-kernel durations from the library's dispatch
    timestamps, and the roofline entry of the kernel that takes the most
    time."""
    import torch
    import paper_2510_27258_amd as hla
    from paper_2510_27258_amd import capi
    from paper_2510_27258_amd import inputs as I

    w = dict(I.WORKLOADS[name])
    if w["kind"] != "forward":
        raise SystemExit("bench.py times the forward workloads")
    B, H, n, d, dv, C = w["B"], w["H"], w["n"], w["d"], w["dv"], w["chunk"]
    q, k, v, code = I.draw_qkv(B, H, n, d, dv, w["dist"], w["seed"])
    dev = torch.device("cuda:0")
    qd, kd, vd = (I.to_torch(x, code, dev) for x in (q, k, v))
    algo = {"auto": capi.HLA_ALGO_AUTO, "chunked": capi.HLA_ALGO_CHUNKED, "fused": capi.HLA_ALGO_FUSED}[algo_name]
    wsb = capi.hla2_workspace_query(B, H, n, d, dv, C, code, algo)
    ws = torch.empty(wsb, dtype=torch.uint8, device=dev)
    out = torch.empty(B, H, n, dv, dtype=torch.float32, device=dev)

    def step():
        hla.forward(qd, kd, vd, C, masked=bool(w["masked"]), normalized=bool(w["normalized"]), eps=w["eps"],
                    algo=algo, out=out, workspace=ws)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(steps):
        step()
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    warm = stats_ms(time_iters(step, max(steps, 50)))
    cold = stats_ms(time_iters(step, cold_iters, cold=True)) if cold_iters else None
    cold_clean = stats_ms(time_iters(step, cold_iters, cold=True, clean=True)) if cold_iters else None

    # per-kernel durations: a second pass with the library's event bracketing
    capi.hla_profile_begin(8 * steps + 8)
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    prof = capi.hla_profile_summary()
    capi.hla_profile_end()
    used_algo = "fused" if "walk" in prof else "chunked"
    P = tile = first = per = None
    if used_algo == "fused":
        P, tile, first, per = capi.hla2_fused_plan(B, H, n, d, dv, C, tiles=True)
    costs = kernel_costs(w, P, tile, first, per, two_pass="walk_first" in prof)
    dom = max(prof, key=lambda kname: prof[kname][1])
    cnt, tot_ms = prof[dom]
    avg_s = tot_ms / cnt / 1e3
    bound, nbytes, nflops = costs[dom]
    peak, unit = peak_for(bound)
    achieved = (nbytes / avg_s / 1e9) if bound == "hbm" else (nflops / avg_s / 1e12)
    tokens = B * H * n
    roof = {"bound": bound, "achieved": achieved, "peak": peak, "unit": unit, "frac": achieved / peak,
            "traffic": traffic_for(dom, name), "kernel": dom, "avg_launch_ms": avg_s * 1e3,
            "algorithmic_bytes": nbytes, "algorithmic_flops": nflops,
            "mfma_tflops": nflops / avg_s / 1e12, "mfma_frac": nflops / avg_s / 1e12 / BF16_MFMA_PEAK_TFLOPS}
    if dom == "walk" and tile != C:
        # the same launch counted densely at the workload's chunk instead of the tile it walks
        f_chunk = nflops * reference_flops_per_token(C, d, dv) / reference_flops_per_token(tile, d, dv)
        roof["mfma_frac_at_chunk"] = f_chunk / avg_s / 1e12 / BF16_MFMA_PEAK_TFLOPS
    rec = {
        "value": tokens / (ms / 1e3),
        "ms_per_step": ms,
        "warm": warm,
        "dtype": "bf16" if used_algo == "fused" else "f32",
        "config": {"workload": name, "B": B, "H": H, "n": n, "d": d, "dv": dv, "chunk": C,
                   "masked": w["masked"], "normalized": w["normalized"], "input_dtype": "bf16" if code else "fp32",
                   "algo": used_algo, "segments_per_head": P, "tile": tile, "segment_tiles": [first, per],
                   "global_batch": B * H, "seq_len": n,
                   "parallelism": "none"},
        "roofline": roof,
        "kernels_ms": {kname: v_[1] / v_[0] for kname, v_ in prof.items()},
        "forward_mfma_frac": (tokens * reference_flops_per_token(tile or C, d, dv)) / (ms / 1e3) / 1e12
                             / BF16_MFMA_PEAK_TFLOPS,
    }
    if cold is not None:
        rec["cold"] = dict(cold, value=tokens / (cold["median_ms"] / 1e3))
        rec["cold_clean"] = dict(cold_clean, value=tokens / (cold_clean["median_ms"] / 1e3))
    return rec, (w, q, k, v)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--algo", default="auto", choices=["auto", "chunked", "fused"])
    ap.add_argument("--cold-iters", type=int, default=50, help="cold (flushed) iterations of the forwards")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-sub", action="store_true", help="skip the second (d = 64) forward workload")
    ap.add_argument("--no-decode", action="store_true", help="skip the decode-step measurement")
    ap.add_argument("--no-scan", action="store_true", help="skip the standalone scan measurement")
    ap.add_argument("--no-hla3", action="store_true", help="skip the third-order measurement")
    ap.add_argument("--no-decay", action="store_true", help="skip the decayed-forward measurement")
    ap.add_argument("--no-ahla", action="store_true", help="skip the AHLA measurement")
    ap.add_argument("--no-backward", action="store_true", help="skip the backward measurement")
    ap.add_argument("--only", choices=["ahla", "decay", "hla3", "hla3u", "backward", "decode", "scan"],
                    help="run only that measurement and print its record (for profiling one path)")
    ap.add_argument("--copy-bytes", type=int, default=0,
                    help="only run --steps device-to-device copies of this many bytes (counter calibration)")
    ap.add_argument("--ingest-counters", nargs=4, metavar=("FETCH_CSV", "WRITE_CSV", "COPY_FETCH_CSV", "COPY_WRITE_CSV"),
                    help="write profiles/hbm_traffic.json for --workload from counter CSVs (with --copy-bytes)")
    args = ap.parse_args()
    if args.ingest_counters:
        ingest_counters(args.workload, *args.ingest_counters, args.copy_bytes)
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path (heads, or sequence segments with "
              "their carries exchanged, would shard across GPUs). Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch

    if args.copy_bytes:
        src = torch.ones(args.copy_bytes // 4, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(args.steps):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": args.copy_bytes, "steps": args.steps}))
        return

    if args.only:
        rec = {"ahla": measure_ahla, "decay": measure_decay, "hla3": measure_hla3,
               "hla3u": lambda: measure_hla3(masked=False), "backward": measure_backward,
               "decode": measure_decode, "scan": lambda: measure_scan(args.workload)}[args.only]()
        print(json.dumps(rec), flush=True)
        return

    head, (w, q, k, v) = measure_forward(args.workload, args.steps, args.warmup, args.algo, args.cold_iters)
    print(f"forward {args.workload}: {head['ms_per_step']:.4f} ms per step", file=sys.stderr, flush=True)
    rec = {
        "metric": "masked HLA-2 forward tokens/s (B*H*n) + % bf16 MFMA peak; decode step GB/s",
        "value": head["value"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": head["dtype"],
        "data": "synthetic",
        "config": head["config"],
        "roofline": head["roofline"],
        "kernels_ms": head["kernels_ms"],
        "warm": head["warm"],
        "cold": head.get("cold"),
        "cold_clean": head.get("cold_clean"),
        "forward_mfma_frac": head["forward_mfma_frac"],
    }
    if not args.no_sub and args.workload != SUB_WORKLOAD:
        sub, _ = measure_forward(SUB_WORKLOAD, args.steps, args.warmup, args.algo, args.cold_iters)
        rec["sub_forward"] = sub
        print(f"forward {SUB_WORKLOAD}: {sub['ms_per_step']:.4f} ms per step", file=sys.stderr, flush=True)
    if not args.no_cpu_baseline:
        rec["cpu_baseline"] = cpu_baseline(w, q, k, v)
        print("cpu baseline done", file=sys.stderr, flush=True)
    del q, k, v
    torch.cuda.empty_cache()
    if not args.no_scan:
        rec["scan"] = {"d64": measure_scan(SUB_WORKLOAD), "d128": measure_scan(DEFAULT_WORKLOAD)}
        print("scan done", file=sys.stderr, flush=True)
    if not args.no_hla3:
        rec["hla3"] = measure_hla3()
        rec["hla3_unmasked"] = measure_hla3(masked=False)
    if not args.no_decay:
        rec["decay"] = measure_decay()
    if not args.no_ahla:
        rec["ahla"] = measure_ahla()
    if not args.no_backward:
        rec["backward"] = measure_backward()
    print("next rows done", file=sys.stderr, flush=True)
    if not args.no_decode:
        torch.cuda.empty_cache()
        rec["decode"] = measure_decode()
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
