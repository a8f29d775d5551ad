"""Benchmark of the LUNA attention forward hot path on one MI355X.

One step = one pass of the whole hot path over one batch of synthetic input:
  * non-causal LUNA attention on the long-sequence encoder problem
    B=32, H=8, n=4096, d=64, M=16 projections x L=8 channels (D=128), bf16;
  * causal LUNA attention (chunked prefix scan, chunk 64) on the long causal problem
    B=8, H=16, n=16384, d=128, M=32 x L=8 (D=256), bf16.
Both read their inputs from HBM (2.7 GB in total, far beyond the 256 MB
Infinity Cache) and each processes 131072 tokens (a token is one sequence
position across all heads).  value = tokens of both problems / step time.

Before the W warm-up steps the step's own calls run untimed for --ramp-ms milliseconds
(default 200): the GPU's power management settles on this workload only after some tens
of its calls, longer than a few warm-up steps last.

The JSON line also carries
  roofline      for the call that takes most of the step: algorithmic HBM bytes per
                call (read Q, K, V once, write out once) divided by its average
                duration from HIP events on the launch stream (the causal call is
                the table build and two scan launches of one kernel);
                traffic is the HBM bytes per call measured by rocprofv3 counters
                (see profiles/), or null when the kernel source changed since they
                were taken;
  cpu_baseline  the float64 oracle timed on the host cores on a bounded sample,
                scaled to the same unit;
  parity        the last timed step's outputs against the oracle's outputs for the
                heads of that sample (largest per-row normwise error).
Only one GPU is supported: --gpus above 1 exits with a message.
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

METRIC = "LUNA attn fwd tokens/sec + % HBM/MFMA roofline at n=4096, causal+non"
HBM_PEAK_GBS = 8000.0          # MI355X HBM3E
MFMA_BF16_PEAK_TFLOPS = 2500.0  # dense bf16 matrix cores
KERNEL_SOURCES = {
    "causal_kernel": ["luna_causal.hip", "luna_device.hpp", "luna_kernels.hpp"],
    "nc_fused_kernel": ["luna_noncausal.hip", "luna_device.hpp", "luna_kernels.hpp"],
    "featuremap_kernel": ["luna_featuremap.hip", "luna_device.hpp", "luna_kernels.hpp"],
}
KERNEL_WORKLOAD = {"causal_kernel": "long_causal", "nc_fused_kernel": "long_noncausal",
                   "featuremap_kernel": "featuremap_long_noncausal"}
# launches of the kernel per ABI call on these workloads: the causal call (128 heads)
# runs two scan launches (the first beside a state-only part, the second from its states)
LAUNCHES_PER_CALL = {"causal_kernel": 2, "nc_fused_kernel": 1, "featuremap_kernel": 1}
COPY_BYTES = 1 << 30  # the --copy-calibration copy


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def source_hash(kernel: str) -> str:
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[kernel]:
        with open(os.path.join(ROOT, "paper_2512_08061_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per call from the committed rocprofv3 counter summary, if current."""
    path = os.path.join(ROOT, "profiles", f"hbm_traffic_{kernel}_{workload}.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    if rec.get("source_hash") != source_hash(kernel):
        return None
    return rec.get("bytes_per_call")


def measured_figure(tag: str, workload: str, kernel: str, figure: str):
    """A figure of the committed rocprofv3 counter summary of `tag` on `workload`, if
    the summary was taken on the kernel's current sources."""
    import re

    path = os.path.join(ROOT, "profiles", f"counters_{tag}_{workload}.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m = re.search(r"Source hash of its files[^`]*`([0-9a-f]+)`", text)
    if not m or m.group(1) != source_hash(kernel):
        return None
    m = re.search(r"^\| " + re.escape(figure) + r"[^|]*\| ([0-9.e+-]+) \|", text, re.M)
    return float(m.group(1)) if m else None


def traffic_from(fetch_csv: str, write_csv: str, command: str) -> int:
    """Turn two rocprofv3 --pmc csv runs (FETCH_SIZE, then WRITE_SIZE, both of
    `bench.py --copy-calibration`) into profiles/hbm_traffic_<kernel>_<workload>.json.

    Each counter is scaled by (1 GiB) / (what it reads for the 1 GiB device copy),
    so that a counter that sees only part of the memory traffic is corrected."""
    import collections
    import csv

    def per_dispatch(path, counter):
        vals = collections.defaultdict(float)
        names = {}
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] != counter:
                continue
            d = int(r["Dispatch_Id"])
            vals[d] += float(r["Counter_Value"]) * 1024.0  # KiB -> bytes
            names[d] = r["Kernel_Name"]
        return vals, names

    out = {}
    for counter, path in (("FETCH_SIZE", fetch_csv), ("WRITE_SIZE", write_csv)):
        vals, names = per_dispatch(path, counter)
        copies = [v for d, v in vals.items() if "copyBuffer" in names[d] and v > 0.25 * COPY_BYTES]
        if not copies:
            log(f"{path}: no 1 GiB copy dispatch found (run bench.py with --copy-calibration)")
            return 1
        if not any(f"{len(k)}{k}" in nm for k in KERNEL_SOURCES for nm in names.values()):
            log(f"{path}: none of the measured kernels")
            return 1
        factor = COPY_BYTES / (sum(copies) / len(copies))
        for kern in KERNEL_SOURCES:
            ds = [d for d in vals if f"{len(kern)}{kern}" in names[d]]
            if ds:
                rec = out.setdefault(kern, {})
                calls = len(ds) / LAUNCHES_PER_CALL[kern]
                rec[counter] = {"counter_bytes_per_call": sum(vals[d] for d in ds) / calls, "dispatches": len(ds),
                                "launches_per_call": LAUNCHES_PER_CALL[kern], "copy_factor": factor}
    for kern, rec in out.items():
        if "FETCH_SIZE" not in rec or "WRITE_SIZE" not in rec:
            continue
        rd = rec["FETCH_SIZE"]["counter_bytes_per_call"] * rec["FETCH_SIZE"]["copy_factor"]
        wr = rec["WRITE_SIZE"]["counter_bytes_per_call"] * rec["WRITE_SIZE"]["copy_factor"]
        wl_name = KERNEL_WORKLOAD[kern]
        doc = {
            "kernel": kern,
            "workload": wl_name,
            "source_hash": source_hash(kern),
            "bytes_per_call": int(rd + wr),
            "read_bytes_per_call": int(rd),
            "write_bytes_per_call": int(wr),
            "counters": rec,
            "copy_calibration": f"{COPY_BYTES} B device-to-device copy in the same process",
            "command": command,
        }
        path = os.path.join(ROOT, "profiles", f"hbm_traffic_{kern}_{wl_name}.json")
        with open(path, "w") as fh:
            json.dump(doc, fh, indent=1)
            fh.write("\n")
        log(f"wrote {path}: read {rd / 2**20:.1f} MiB, write {wr / 2**20:.1f} MiB per call")
    return 0


def copy_calibration(dev) -> None:
    """Three 1 GiB device-to-device copies: the known traffic that rocprofv3's
    FETCH_SIZE / WRITE_SIZE readings are scaled by."""
    import torch

    src = torch.empty(COPY_BYTES, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst


def flops_per_token_head(w, causal: bool) -> int:
    """Matrix-core flops per (b, h, token): projections of q and k (4dM), S and the
    readout (4Dd), z and the denominator (4D), plus the causal intra-chunk blocks
    P, PV and P1 over full 64x64 blocks (2C(D + d + 1))."""
    D = w.M * w.L
    f = 4 * w.d * w.M + 4 * D * w.d + 4 * D
    if causal:
        f += 2 * w.chunk * (D + w.d + 1)
    return f


def bytes_per_token_head(w) -> int:
    """Read q, k, v and write out once, in the storage dtype."""
    return 4 * w.d * (2 if w.dtype == "bf16" else 4)


def clock_ramp(step, ms: float) -> None:
    """Runs the step's own calls, untimed, for `ms` milliseconds before the warm-up steps.
    The GPU's power management settles on this workload only after some tens of its
    calls (with the driver's 5 warm-up steps the timed steps measured 0.970 ms, after 30
    0.879 ms, after 100 0.874 ms; tens of milliseconds of plain matrix products or HBM
    reads beforehand brought only 0.940-0.960 ms), so that the timed steps would measure
    the GPU's ramp rather than the kernels."""
    import torch

    t0 = time.perf_counter()
    calls = 0
    while time.perf_counter() - t0 < ms / 1e3:
        for _ in range(10):
            step()
        calls += 10
        torch.cuda.synchronize()
    log(f"clock ramp: {calls} untimed steps in {1e3 * (time.perf_counter() - t0):.0f} ms before the warm-up steps")


def cpu_baseline(w4, arrs4, p4, w5, arrs5, p5, refs=None):
    """The float64 oracle on a bounded sample of the same step, scaled to tokens/s.
    The oracle's outputs for the sampled heads go into `refs` (name -> list of
    ((b, h), out)) for the parity check of the GPU's outputs."""
    import numpy as np
    from threadpoolctl import threadpool_limits

    import oracle

    threads = len(os.sched_getaffinity(0))
    budget = 8.0  # seconds per part: whole heads are added until a part has run this long
    with threadpool_limits(threads):
        nc_heads, t_nc = 0, 0.0
        while nc_heads < w4.B * w4.H and t_nc < budget:
            b, h = divmod(nc_heads, w4.H)
            Q, K, V = (a[b, h:h + 1].astype(np.float64) for a in arrs4)
            t0 = time.perf_counter()
            o = oracle.attn_noncausal(Q, K, V, p4, eps=w4.eps)
            t_nc += time.perf_counter() - t0
            nc_heads += 1
            if refs is not None:
                refs.setdefault("long_noncausal", []).append(((b, h), o[0]))
        cs_heads, t_cs = 0, 0.0
        while cs_heads < w5.B * w5.H and t_cs < budget:
            b, h = divmod(cs_heads, w5.H)
            Q, K, V = (a[b, h:h + 1].astype(np.float64) for a in arrs5)
            t0 = time.perf_counter()
            o = oracle.attn_causal(Q, K, V, p5, eps=w5.eps)
            t_cs += time.perf_counter() - t0
            cs_heads += 1
            if refs is not None:
                refs.setdefault("long_causal", []).append(((b, h), o[0]))
    step = t_nc * (w4.B * w4.H) / nc_heads + t_cs * (w5.B * w5.H) / cs_heads
    tokens = w4.B * w4.n + w5.B * w5.n
    return {
        "value": tokens / step,
        "unit": "tokens/s",
        "cores": threads,
        "kind": "oracle",
        "sample": (f"float64 oracle on whole heads: non-causal {nc_heads} of {w4.B * w4.H} heads ({t_nc:.1f} s), "
                   f"causal token recurrence {cs_heads} of {w5.B * w5.H} heads ({t_cs:.1f} s), "
                   f"scaled by heads to one full step"),
    }


def parity_check(refs, outs) -> dict:
    """The GPU's outputs of the last timed step against the oracle's outputs for the
    heads the CPU baseline ran: the largest per-row normwise error
    max|gpu - ref| / max|ref| (the tests' metric for bf16, tolerance 2e-2)."""
    import numpy as np

    res = {"tol": 2e-2, "metric": "max over rows of max|gpu - oracle| / max|oracle| per row"}
    ok = True
    for name, lst in refs.items():
        worst = 0.0
        for (b, h), ref in lst:
            got = outs[name][b, h].float().cpu().numpy().astype(np.float64)
            err = np.abs(got - ref).max(axis=1) / np.maximum(np.abs(ref).max(axis=1), 1e-30)
            worst = max(worst, float(err.max()))
        res[name] = {"heads_checked": len(lst), "max_row_err": worst}
        ok = ok and worst <= res["tol"]
    res["pass"] = ok
    return res


def featuremap_bench(args) -> int:
    """luna_featuremap on the long encoder problem's queries (B=32, H=8, n=4096, d=64,
    M=16 x L=8, bf16 in and out): HIP events around each call (table build included),
    algorithmic bytes = rows x (d + D) x 2 (read x, write phi)."""
    import ctypes

    import torch

    from paper_2512_08061_amd import luna
    from paper_2512_08061_amd import workloads as wl

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    lib = luna.load_library()
    w = wl.WORKLOADS["long_noncausal"]
    Q, _, _ = wl.make_inputs(w, args.seed)
    p = wl.make_params(w, args.seed)
    x = torch.from_numpy(Q).to(dev).to(torch.bfloat16).contiguous()
    del Q
    pt = luna.PhiParams.from_arrays(p, dev, torch.bfloat16)
    pc = pt.c()
    D = w.M * w.L
    out = torch.empty((w.B, w.H, w.n, D), dtype=torch.bfloat16, device=dev)
    nb = luna.workspace_bytes(luna.OP_FEATUREMAP, luna.LUNA_BF16, w.B, w.H, w.n, w.d, pt)
    ws = torch.empty(nb + 256, dtype=torch.uint8, device=dev)
    wsp = ws.data_ptr() + (-ws.data_ptr()) % 256
    stream = torch.cuda.current_stream(dev)
    if args.copy_calibration:
        copy_calibration(dev)

    def call():
        st = lib.luna_featuremap(x.data_ptr(), luna.LUNA_BF16, w.B, w.H, w.n, w.d, ctypes.byref(pc), out.data_ptr(),
                                 luna.LUNA_BF16, wsp, nb, stream.cuda_stream)
        assert st == luna.LUNA_OK, lib.luna_last_error()

    for _ in range(args.warmup):
        call()
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    for e0, e1 in ev:
        e0.record(stream)
        call()
        e1.record(stream)
    torch.cuda.synchronize()
    ms = sum(e0.elapsed_time(e1) for e0, e1 in ev) / args.steps
    rows = w.B * w.H * w.n
    nbytes = rows * (w.d + D) * 2
    gbs = nbytes / (ms * 1e-3) / 1e9
    line = {
        "metric": "LUNA feature map rows/sec (luna_featuremap)",
        "value": rows / (ms * 1e-3), "unit": "rows/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms, 5), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16", "data": "synthetic (seeded)",
        "config": {"workload": "phi of the long encoder problem's queries, B=32 H=8 n=4096 d=64, M=16 x L=8 "
                               "(D=128), bf16 in and out"},
        "roofline": {"bound": "hbm", "achieved": round(gbs, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": None, "kernel": "featuremap_kernel",
                     "bytes_per_call": nbytes,
                     "timing": "HIP events around each ABI call (table build and feature-map kernel)"},
    }
    print(json.dumps(line), flush=True)
    return 0


def backward_bench(args) -> int:
    """luna_attn_bwd (input and parameter gradients) on the long encoder problem and on
    the long causal problem: HIP events around each call.  The algorithmic bytes are
    reading Q, K, V, dO and writing dQ, dK, dV once (7 d elements per token and head)."""
    import numpy as np
    import torch

    from paper_2512_08061_amd import luna
    from paper_2512_08061_amd import workloads as wl

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    luna.load_library()
    stream = torch.cuda.current_stream(dev)
    for name in ("long_noncausal", "long_causal"):
        w = wl.WORKLOADS[name]
        arrs = wl.make_inputs(w, args.seed)
        p = wl.make_params(w, args.seed)
        q, k, v = (torch.from_numpy(a).to(dev).to(torch.bfloat16) for a in arrs)
        del arrs
        do = torch.from_numpy(np.random.default_rng(args.seed + 7).standard_normal(q.shape).astype(np.float32))
        do = do.to(dev).to(torch.bfloat16)
        pt = luna.PhiParams.from_arrays(p, dev, torch.bfloat16)
        for _ in range(args.warmup):
            luna.attn_bwd(q, k, v, do, pt, causal=w.causal, eps=w.eps)
        torch.cuda.synchronize()
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
        for e0, e1 in ev:
            e0.record(stream)
            luna.attn_bwd(q, k, v, do, pt, causal=w.causal, eps=w.eps)
            e1.record(stream)
        torch.cuda.synchronize()
        ms = sorted(e0.elapsed_time(e1) for e0, e1 in ev)[len(ev) // 2]
        th = w.B * w.H * w.n
        nbytes = 7 * w.d * 2 * th
        gbs = nbytes / (ms * 1e-3) / 1e9
        line = {
            "metric": "LUNA attention backward tokens/sec (luna_attn_bwd, input and parameter gradients)",
            "value": w.B * w.n / (ms * 1e-3), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True, "scaling": "weak",
            "vs_baseline": None, "dtype": "bf16", "data": "synthetic (seeded)",
            "config": {"workload": f"{name} {w.B}x{w.H}x{w.n}x{w.d} D={w.M * w.L} "
                                   f"{'causal chunk=64' if w.causal else 'non-causal'}, bf16 in, fp32 arithmetic"},
            "roofline": {"bound": "hbm", "achieved": round(gbs, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                         "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": None, "bytes_per_call": nbytes,
                         "timing": "HIP events around each ABI call (median); workspace allocated per call by the "
                                   "binding"},
        }
        print(json.dumps(line), flush=True)
        del q, k, v, do, pt
        torch.cuda.synchronize()
    return 0


# Counters that `--counters-from` summarises, with what each derived figure means.
COUNTER_RATIOS = [
    ("VALU instructions per wave", "SQ_INSTS_VALU", "SQ_WAVES", 1.0),
    ("MFMA instructions per wave", "SQ_INSTS_MFMA", "SQ_WAVES", 1.0),
    ("LDS instructions per wave", "SQ_INSTS_LDS", "SQ_WAVES", 1.0),
    ("SALU instructions per wave", "SQ_INSTS_SALU", "SQ_WAVES", 1.0),
    ("vector memory reads per wave", "SQ_INSTS_VMEM_RD", "SQ_WAVES", 1.0),
    ("vector memory writes per wave", "SQ_INSTS_VMEM_WR", "SQ_WAVES", 1.0),
    ("wave lifetime, cycles per wave (SQ_WAVE_CYCLES counts 4-cycle units)", "SQ_WAVE_CYCLES", "SQ_WAVES", 4.0),
    ("share of wave lifetime issuing VALU", "SQ_ACTIVE_INST_VALU", "SQ_WAVE_CYCLES", 1.0),
    ("share of wave lifetime issuing LDS", "SQ_ACTIVE_INST_LDS", "SQ_WAVE_CYCLES", 1.0),
    ("share of wave lifetime issuing anything", "SQ_ACTIVE_INST_ANY", "SQ_WAVE_CYCLES", 1.0),
    ("share of wave lifetime waiting on dependencies (s_waitcnt)", "SQ_WAIT_INST_ANY", "SQ_WAVE_CYCLES", 1.0),
    ("share of wave lifetime waiting on LDS", "SQ_WAIT_INST_LDS", "SQ_WAVE_CYCLES", 1.0),
    ("LDS bank-conflict cycles per LDS-active cycle", "SQ_LDS_BANK_CONFLICT", "SQ_LDS_IDX_ACTIVE", 1.0),
]
# (figure, counter, units): counter / (cycles of the dispatch x units), the dispatch's
# cycles being GRBM_GUI_ACTIVE / 8: rocprofv3 sums that counter over the 8 XCDs (it
# reads 8x the kernel's duration in GPU clocks)
XCDS = 8
COUNTER_UTIL = [
    ("MFMA busy, share of all SIMD cycles (1024 SIMDs)", "SQ_VALU_MFMA_BUSY_CYCLES", 1024),
    ("LDS active, share of all CU cycles (256 CUs)", "SQ_LDS_IDX_ACTIVE", 256),
    ("SQ busy, share of all CU cycles (256 CUs)", "SQ_BUSY_CU_CYCLES", 256),
]
COUNTER_KERNELS = {  # kernel-name pattern (mangled or not) -> (file tag, workload, kernel whose sources are hashed)
    r"nc_fused_kernel(<|I)": ("nc_fused_kernel", "long_noncausal", "nc_fused_kernel"),
    r"(13causal_kernelI.*Lb1ELb0EE|\bcausal_kernel<.*true, false>)": ("causal_kernel_state_launch", "long_causal",
                                                                         "causal_kernel"),
    r"(13causal_kernelI.*Lb0ELb0EE|\bcausal_kernel<.*false, false>)": ("causal_kernel_scan_launch", "long_causal",
                                                                          "causal_kernel"),
    r"pwl_prepare_kernel": ("pwl_prepare_kernel", "bench_step", None),
    r"featuremap_kernel(<|I)": ("featuremap_kernel", "featuremap_long_noncausal", None),
}


def counters_from(csvs, command: str) -> int:
    """Average every counter per dispatch, per kernel, over rocprofv3 --pmc csv files
    (one file per pass), and write profiles/counters_<kernel>_<workload>.md."""
    import collections
    import csv
    import re

    per = collections.defaultdict(dict)  # (kernel, counter) -> {(file, dispatch): value}
    names = set()
    for path in csvs:
        for r in csv.DictReader(open(path)):
            key = (r["Kernel_Name"], r["Counter_Name"])
            d = (path, int(r["Dispatch_Id"]))
            per[key][d] = per[key].get(d, 0.0) + float(r["Counter_Value"])
            names.add(r["Kernel_Name"])
    written = 0
    for pat, (tag, wl_name, src) in COUNTER_KERNELS.items():
        kern = sorted(k for k in names if re.search(pat, k))
        if not kern:
            continue
        vals = {}
        for (k, c), d in per.items():
            if k in kern:
                vals[c] = sum(d.values()) / len(d)
        rows = []
        for label, a, b, mul in COUNTER_RATIOS:
            if a in vals and b in vals and vals[b] > 0:
                rows.append((label, mul * vals[a] / vals[b], (f"{mul:g} x " if mul != 1 else "") + f"{a} / {b}"))
        if vals.get("GRBM_GUI_ACTIVE", 0) > 0:
            rows.append(("dispatch duration, GPU cycles", vals["GRBM_GUI_ACTIVE"] / XCDS,
                         f"GRBM_GUI_ACTIVE / {XCDS} (summed over the XCDs)"))
        for label, a, units in COUNTER_UTIL:
            if a in vals and vals.get("GRBM_GUI_ACTIVE", 0) > 0:
                rows.append((label, vals[a] * XCDS / (vals["GRBM_GUI_ACTIVE"] * units),
                             f"{a} / (GRBM_GUI_ACTIVE / {XCDS} x {units})"))
        path = os.path.join(ROOT, "profiles", f"counters_{tag}_{wl_name}.md")
        lines = [f"# rocprofv3 counters: {tag} ({wl_name})", "", f"Kernel: `{kern[0]}`", ""]
        if src:
            lines += [f"Source hash of its files (as bench.py's traffic records): `{source_hash(src)}`", ""]
        lines += ["Commands (one counter pass each; every counter averaged per dispatch of the kernel):", "",
                  "```", command, "```", "", "| figure | value | from |", "|---|---|---|"]
        lines += [f"| {label} | {v:.4g} | `{how}` |" for label, v, how in rows]
        lines += ["", "| counter | mean per dispatch |", "|---|---|"]
        lines += [f"| {c} | {vals[c]:.6g} |" for c in sorted(vals)]
        with open(path, "w") as fh:
            fh.write("\n".join(lines) + "\n")
        log(f"wrote {path}")
        written += 1
    return 0 if written else 1


def decode_bench(args) -> int:
    """Streaming steps of m tokens per head from the state of a 16384-token prefix on
    the long causal problem's shape (B=8, H=16, d=128, M=32 x L=8, bf16).  Each step
    reads and writes the fp32 state S [128 heads][256][128] and z once."""
    import torch

    from paper_2512_08061_amd import luna
    from paper_2512_08061_amd import workloads as wl

    if args.gpus != 1:
        print("bench.py runs on one GPU only; use --gpus 1.", file=sys.stderr)
        return 2
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    luna.load_library()
    w = wl.WORKLOADS["long_causal"]
    m = int(args.decode)
    Q, K, V = wl.make_inputs(w, args.seed)
    p = wl.make_params(w, args.seed)
    up = lambda a: torch.from_numpy(a).to(dev).to(torch.bfloat16).contiguous()  # noqa: E731
    kt, vt = up(K), up(V)
    pt = luna.PhiParams.from_arrays(p, dev, torch.bfloat16)
    S, z = luna.attn_state(kt, vt, pt)  # the prefix
    del kt, vt
    rng = __import__("numpy").random.default_rng(args.seed + 1)
    new = [up(rng.standard_normal((w.B, w.H, m, w.d)).astype("float32")) for _ in range(3)]
    # one persistent workspace: the first step builds the channel tables, the others reuse them
    plan = luna.StepPlan(pt, w.B, w.H, m, w.d, torch.bfloat16, dev, eps=w.eps)
    out = torch.empty_like(new[0])
    stream = torch.cuda.current_stream(dev)

    def step():
        plan.run(new[0], new[1], new[2], S, z, out, stream.cuda_stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    run = step
    if args.graph:  # one call captured (the tables are built by then), replayed
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            plan.run(new[0], new[1], new[2], S, z, out)
        torch.cuda.synchronize()
        run = g.replay
        stream = torch.cuda.current_stream(dev)
        for _ in range(args.warmup):
            run()
        torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(args.steps):
        run()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / args.steps
    heads, D = w.B * w.H, w.M * w.L
    state_bytes = 2 * heads * D * (w.d + 1) * 4  # S and z, read and written once
    io_bytes = 4 * heads * m * w.d * 2            # q, k, v read, out written
    gbs = (state_bytes + io_bytes) / (ms * 1e-3) / 1e9
    line = {
        "metric": "LUNA causal streaming step tokens/sec (decode)",
        "value": heads * m / (ms * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded)",
        "config": {"workload": f"streaming step of {m} token(s) per head after a 16384-token prefix, "
                               "B=8 H=16 d=128 M=32 L=8 (D=256), bf16, fp32 state", "m": m,
                   "graph": bool(args.graph)},
        "roofline": {"bound": "hbm", "achieved": round(gbs, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": None, "kernel": "causal_step_kernel",
                     "bytes_per_call": state_bytes + io_bytes,
                     "timing": ("replays of a HIP graph holding one call" if args.graph else
                                "HIP events around the ABI calls (tables built by the first, reused after)") +
                               ": one feature-map launch for the new queries and keys, then the step kernel"},
    }
    print(json.dumps(line), flush=True)
    return 0


MFMA_F32_PEAK_TFLOPS = 157.3  # dense fp32 matrix cores


def config_cases():
    """(label, workload) pairs of the per-configuration report: the five synthetic
    problems, the sequence-length sweep n = 1024 .. 16384 at the long encoder
    problem's other sizes (B=32, H=8, d=64, M=16 x L=8), non-causal and causal, and
    the one-channel variants (L=1, M = D) of the two long problems."""
    from paper_2512_08061_amd import workloads as wl

    W = wl.WORKLOADS
    cases = [(name, W[name]) for name in ("tiny_f32", "text_encoder", "vision_encoder", "long_noncausal",
                                          "long_causal")]
    for causal in (False, True):
        for n in (1024, 2048, 4096, 8192, 16384):
            tag = "causal" if causal else "noncausal"
            cases.append((f"sweep_{tag}_n{n}", W["long_noncausal"].with_(n=n, causal=causal, name=f"sweep_{n}")))
    cases.append(("long_noncausal_L1", W["long_noncausal"].with_(M=128, L=1)))
    cases.append(("long_causal_L1", W["long_causal"].with_(M=256, L=1)))
    return cases


def config_oracle(w, arrs, p, out, budget: float) -> dict:
    """The float64 oracle on whole heads of one configuration's inputs (the linear form
    non-causal, the token recurrence causal), heads added until `budget` seconds have
    run (at least one), scaled by heads to tokens/s of the whole configuration; and the
    largest per-row error of the GPU output `out` on those heads."""
    import numpy as np
    from threadpoolctl import threadpool_limits

    import oracle

    threads = len(os.sched_getaffinity(0))
    f = oracle.attn_causal if w.causal else oracle.attn_noncausal
    tol = 2e-2 if w.dtype == "bf16" else 1e-4
    heads, spent, worst = 0, 0.0, 0.0
    with threadpool_limits(threads):
        while heads < w.B * w.H and (heads == 0 or spent < budget):
            b, h = divmod(heads, w.H)
            Q, K, V = (a[b, h:h + 1].astype(np.float64) for a in arrs)
            t0 = time.perf_counter()
            ref = f(Q, K, V, p, eps=w.eps)[0]
            spent += time.perf_counter() - t0
            got = out[b, h].float().cpu().numpy().astype(np.float64)
            err = np.abs(got - ref).max(axis=1) / np.maximum(np.abs(ref).max(axis=1), 1e-30)
            worst = max(worst, float(err.max()))
            heads += 1
    secs = spent * (w.B * w.H) / heads
    return {"tokens_per_s": w.B * w.n / secs, "cores": threads, "heads": heads, "seconds": round(spent, 3),
            "max_row_err": worst, "tol": tol, "pass": worst <= tol}


def configs_bench(args) -> int:
    """One timed ABI call per configuration, each on its own seeded inputs, with the
    caches flushed before every timed call (a 1 GiB buffer is read, which evicts the
    256 MB Infinity Cache and the L2s without leaving dirty lines whose write-back
    would fall into the timed call), so that the small problems, whose inputs would
    otherwise stay cached between calls, read them from HBM.  Prints one
    JSON line per configuration (median and 10th / 90th percentile call time from HIP
    events on the launch stream; the table build is part of every call)."""
    import torch

    from paper_2512_08061_amd import luna
    from paper_2512_08061_amd import workloads as wl

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    luna.load_library()
    stream = torch.cuda.current_stream(dev)
    flush = torch.ones(1 << 28, dtype=torch.float32, device=dev)
    sink = torch.empty((), dtype=torch.float32, device=dev)
    rows = []
    only = set(filter(None, args.configs_only.split(",")))
    for label, w in config_cases():
        if only and label not in only:
            continue
        tdt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
        arrs = wl.make_inputs(w, args.seed)
        p = wl.make_params(w, args.seed)
        q, k, v = (torch.from_numpy(a).to(dev).to(tdt) for a in arrs)
        rec = {"config": label, "shape": {"B": w.B, "H": w.H, "n": w.n, "d": w.d, "M": w.M, "L": w.L,
                                          "D": w.M * w.L, "causal": w.causal, "dtype": w.dtype, "dist": w.dist}}
        try:
            pt = luna.PhiParams.from_arrays(p, dev, tdt)
            plan = luna.Plan(luna.OP_ATTN_CAUSAL if w.causal else luna.OP_ATTN, q, k, v, pt, eps=w.eps,
                             chunk=w.chunk)
            plan.run()  # an unsupported (d, M, L) is reported here, before anything is launched
        except luna.LunaError as e:
            rec["status"] = f"not run: {e}"
            log(f"{label}: {rec['status']}")
            rows.append(rec)
            print(json.dumps(rec), flush=True)
            continue
        # flushes, calls and events are queued back to back with one synchronisation at
        # the end, so that the GPU never idles (it keeps its clock) and the host's launch
        # time is hidden behind the flush that precedes each call
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(args.steps)]
        for i in range(args.warmup):
            torch.amax(flush, dim=0, out=sink)
            plan.run()
        for i, (e0, e1) in enumerate(ev):
            torch.amax(flush, dim=0, out=sink)
            e0.record(stream)
            plan.run()
            e1.record(stream)
        torch.cuda.synchronize()
        times = sorted(e0.elapsed_time(e1) for e0, e1 in ev)
        pick = lambda f: times[min(len(times) - 1, int(f * len(times)))]  # noqa: E731
        ms = pick(0.5)
        th = w.B * w.H * w.n
        gb = bytes_per_token_head(w) * th / 1e9
        tf = flops_per_token_head(w, w.causal) * th / 1e12
        mfma_peak = MFMA_BF16_PEAK_TFLOPS if w.dtype == "bf16" else MFMA_F32_PEAK_TFLOPS
        t_hbm, t_mfma = gb / HBM_PEAK_GBS, tf / mfma_peak
        # the path, from the workspace beyond the tables (a feature-map call's workspace):
        # the fp32 GEMM path holds fp32 features of the queries and keys (8 M L bytes per
        # token and head), the causal kernel with the features given bf16 ones (4 M L),
        # the attention kernels at most small partial statistics
        ws_tables = luna.workspace_bytes(luna.OP_FEATUREMAP, luna.LUNA_BF16 if w.dtype == "bf16" else luna.LUNA_F32,
                                         w.B, w.H, w.n, w.d, pt)
        fb = (plan.ws_bytes - ws_tables) / (w.M * w.L * th)
        path = "fp32 GEMM" if fb >= 8 else "features mapped, then scan" if fb >= 4 else "attention kernels"
        rec.update({
            "status": "ok",
            "path": path,
            "ms_median": round(ms, 5), "ms_p10": round(pick(0.1), 5), "ms_p90": round(pick(0.9), 5),
            "tokens_per_s": w.B * w.n / (ms / 1e3),
            "head_tokens_per_s": th / (ms / 1e3),
            "attn_tflops": tf / (ms / 1e3),
            "hbm_gbs": gb / (ms / 1e3),
            "bound": "hbm" if t_hbm >= t_mfma else "mfma",
            "roofline_frac": max(t_hbm, t_mfma) / (ms / 1e3),
            "floor_us": 1e6 * max(t_hbm, t_mfma),
        })
        oc = config_oracle(w, arrs, p, plan.out, args.oracle_budget)
        rec["oracle"] = oc
        rec["speedup_vs_oracle"] = oc["tokens_per_s"] and rec["tokens_per_s"] / oc["tokens_per_s"]
        log(f"{label}: {ms * 1e3:.1f} us, {rec['roofline_frac']:.1%} of the {rec['bound']} roofline; oracle "
            f"{oc['tokens_per_s']:.3g} tokens/s on {oc['cores']} cores ({oc['heads']} heads), parity "
            f"{oc['max_row_err']:.2e}")
        rows.append(rec)
        print(json.dumps(rec), flush=True)
        del plan, q, k, v, arrs
        torch.cuda.synchronize()
    bad = [r["config"] for r in rows if r["status"] == "ok" and not r["oracle"]["pass"]]
    if bad:
        log(f"parity against the oracle FAILED for {bad}")
    if args.configs_table:
        with open(args.configs_table, "w") as fh:
            fh.write("# LUNA attention forward per configuration on one MI355X\n\n")
            fh.write(f"Command: `python bench.py --configs --steps {args.steps} --warmup {args.warmup} "
                     f"--oracle-budget {args.oracle_budget:g} --configs-table {args.configs_table}`\n\n")
            fh.write("One ABI call per row (table build included), median of the timed calls with the 10th and "
                     "90th percentiles, HIP events on the launch stream, caches flushed by a 1 GiB read before "
                     "every timed call. tokens/s counts B*n (a token is one position across all heads); "
                     "TFLOP/s counts the matrix-core work (projections, S, readout, z, denominators, and for "
                     "causal the full 64x64 intra-chunk blocks); the floor is the larger of the HBM time of the "
                     "algorithmic bytes (read Q, K, V, write out) at 8 TB/s and the MFMA time at the dtype's "
                     "dense peak. path: the attention kernels (fused, or the split state / reduce / readout kernels "
                     "below 192 heads), the features mapped first and then the causal scan kernel, or the fp32 "
                     "GEMM path of the shapes that have neither (features in the workspace, all arithmetic "
                     "fp32).\n\n")
            cores = next((r["oracle"]["cores"] for r in rows if r["status"] == "ok"), 0)
            fh.write(f"oracle: the float64 CPU oracle (the linear form non-causal, the token recurrence causal) "
                     f"timed in the same run on {cores} host cores over whole heads of the same inputs, added "
                     f"until about {args.oracle_budget:g} s had run (at least one head), scaled by heads to the "
                     f"whole configuration; parity: the largest per-row error max|gpu - oracle| / max|oracle| "
                     f"of the timed call's output on those heads (bar 2e-2 bf16, 1e-4 fp32).\n\n")
            fh.write("| config | B,H,n,d | M x L | dtype | causal | path | median us (p10-p90) | tokens/s "
                     "| head-tokens/s | TFLOP/s | GB/s | floor us | roofline | oracle tokens/s (heads) "
                     "| GPU / oracle | parity |\n"
                     "|---|---|---|---|---|---|---|---|---|---|---|---|---|---|---|---|\n")
            for r in rows:
                s = r["shape"]
                head = (f"| {r['config']} | {s['B']},{s['H']},{s['n']},{s['d']} | {s['M']} x {s['L']} | "
                        f"{s['dtype']} | {'yes' if s['causal'] else 'no'} |")
                if r["status"] != "ok":
                    fh.write(head + f" | {r['status']} | | | | | | | | | |\n")
                    continue
                oc = r["oracle"]
                fh.write(head + f" {r['path']} | {1e3 * r['ms_median']:.1f} ({1e3 * r['ms_p10']:.1f}-{1e3 * r['ms_p90']:.1f}) | "
                         f"{r['tokens_per_s']:.3g} | {r['head_tokens_per_s']:.3g} | {r['attn_tflops']:.1f} | "
                         f"{r['hbm_gbs']:.0f} | {r['floor_us']:.1f} | {r['roofline_frac']:.1%} {r['bound']} | "
                         f"{oc['tokens_per_s']:.3g} ({oc['heads']}) | {r['speedup_vs_oracle']:.3g}x | "
                         f"{oc['max_row_err']:.1e} {'ok' if oc['pass'] else 'FAIL'} |\n")
        log(f"wrote {args.configs_table}")
    return 1 if bad else 0


VALU_LANE_OPS = 78.6e12  # fp32 vector FMA lane-operations per second (157.3 TFLOP/s / 2)
# VALU issue slots of a channel-MLP hidden unit beyond its two multiply-adds and a relu,
# as the kernels evaluate the activations, a transcendental (exp2, rcp) counted as four
# slots (quarter rate): silu z rcp(1 + 2^(-z log2 e)) and tanh 1 - 2 rcp(2^(2z log2 e) + 1)
# take 3 + 2 x 4 more; gelu (erf by Abramowitz and Stegun 7.1.26) 12 + 2 x 4 more.
ACT_EXTRA_SLOTS = {"relu": 0, "silu": 10, "tanh": 10, "gelu": 20}


def mlp_slots_per_unit(act: str, shared: bool, L: int) -> float:
    """VALU issue slots per (projection, channel, hidden unit) of a channel MLP: the
    first layer's multiply-add, the activation and the second layer's multiply-add; with
    a shared first layer the first two are paid once for the L channels."""
    if shared:
        return (2 + ACT_EXTRA_SLOTS[act] + L) / L
    return 3 + ACT_EXTRA_SLOTS[act]
# (label, kind, act, M, L, options) of the variant report, on the long encoder problem's
# queries; every map has D = 128 features per row except Bank+Coef (D = M = 16)
VARIANT_CASES = [
    ("rff_cos", "rff_cos", "relu", 128, 1, {}),
    ("rff_sincos", "rff_sincos", "relu", 64, 1, {}),
    ("performer", "performer", "relu", 128, 1, {}),
    ("mlp_relu", "mlp", "relu", 16, 8, {}),
    ("mlp_gelu", "mlp", "gelu", 16, 8, {}),
    ("mlp_silu_shared", "mlp", "silu", 16, 8, {"shared": True}),
    ("mlp_tanh_envelope", "mlp", "tanh", 16, 8, {"env": True}),
    ("mlp_gelu_ch_rms", "mlp", "gelu", 16, 8, {"ch_rms": True}),
    ("mlp_gelu_bank", "mlp", "gelu", 16, 8, {"bank": True}),
]


def _timed_calls(fn, steps, warmup, stream, flush, sink):
    """Median, 10th and 90th percentile of HIP-event call times (ms), with a 1 GiB read
    before every call so that the inputs come from HBM."""
    import torch

    for _ in range(warmup):
        torch.amax(flush, dim=0, out=sink)
        fn()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    for e0, e1 in ev:
        torch.amax(flush, dim=0, out=sink)
        e0.record(stream)
        fn()
        e1.record(stream)
    torch.cuda.synchronize()
    times = sorted(e0.elapsed_time(e1) for e0, e1 in ev)
    pick = lambda f: times[min(len(times) - 1, int(f * len(times)))]  # noqa: E731
    return pick(0.5), pick(0.1), pick(0.9)


def variants_bench(args) -> int:
    """The feature-map variants (luna_featuremap_variant) on the long encoder problem's
    queries (B=32, H=8, n=4096, d=64, bf16 in and out), and attention from given
    features (luna_attn_fwd_features) at the two long problems' shapes.  One JSON line
    per case: median call time (HIP events, caches flushed before every call), the HBM
    floor of the algorithmic bytes (read x, write phi; channel RMS also writes and reads
    y in fp32 between its passes) and, for the channel MLPs, the VALU floor of their
    hidden units (mlp_slots_per_unit issue slots each at 78.6e12 lane slots/s)."""
    import torch

    from paper_2512_08061_amd import luna
    from paper_2512_08061_amd import workloads as wl

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    luna.load_library()
    stream = torch.cuda.current_stream(dev)
    flush = torch.ones(1 << 28, dtype=torch.float32, device=dev)
    sink = torch.empty((), dtype=torch.float32, device=dev)
    w = wl.WORKLOADS["long_noncausal"]
    Q, _, _ = wl.make_inputs(w, args.seed)
    x = torch.from_numpy(Q).to(dev).to(torch.bfloat16).contiguous()
    del Q
    rows = w.B * w.H * w.n
    rows_out = []
    only = set(filter(None, args.variants_only.split(",")))
    for label, kind, act, M, L, opts in VARIANT_CASES:
        if only and label not in only:
            continue
        p = wl.make_variant_params(kind, M, w.d, L=L, act=act, seed=args.seed, **opts)
        v = luna.PhiVariant.from_arrays(p, dev, torch.bfloat16)
        D = v.features()
        out = torch.empty((w.B, w.H, w.n, D), dtype=torch.bfloat16, device=dev)
        fn = lambda: luna.featuremap_variant(x, v, out=out)  # noqa: E731
        ms, p10, p90 = _timed_calls(fn, args.steps, args.warmup, stream, flush, sink)
        nbytes = rows * (w.d + D) * 2 + (rows * M * L * 4 * 2 if opts.get("ch_rms") else 0)
        t_hbm = nbytes / (HBM_PEAK_GBS * 1e9)
        units = rows * M * L * p.get("hidden", 0) if kind == "mlp" else 0
        t_alu = units * mlp_slots_per_unit(act, bool(opts.get("shared")), L) / VALU_LANE_OPS if units else 0.0
        bound, floor = ("alu", t_alu) if t_alu > t_hbm else ("hbm", t_hbm)
        rec = {"case": label, "kind": kind, "act": act, "M": M, "L": L, "D": D, "options": opts,
               "workload": "long encoder queries B=32 H=8 n=4096 d=64, bf16 in and out",
               "ms_median": round(ms, 5), "ms_p10": round(p10, 5), "ms_p90": round(p90, 5),
               "rows_per_s": rows / (ms * 1e-3), "hbm_gbs": nbytes / (ms * 1e-3) / 1e9,
               "hidden_units_per_s": units / (ms * 1e-3) if units else None,
               "bound": bound, "floor_us": 1e6 * floor, "roofline_frac": floor / (ms * 1e-3)}
        log(f"{label}: {1e3 * ms:.1f} us, {rec['roofline_frac']:.1%} of the {bound} floor")
        print(json.dumps(rec), flush=True)
        rows_out.append(rec)
        del out
    del x
    # attention from given features: positive features exp(N(0, 1/4)) / sqrt(D), drawn
    # on the device from a seeded generator
    gen = torch.Generator(device=dev)
    gen.manual_seed(args.seed)
    for label, (B, H, n, d, D, fdt, causal) in (
            ("features_causal_bf16", (8, 16, 16384, 128, 256, torch.bfloat16, True)),
            ("features_noncausal_f32", (32, 8, 4096, 64, 128, torch.float32, False))):
        if only and label not in only:
            continue
        feats = []
        for _ in range(2):
            t = torch.empty((B, H, n, D), dtype=fdt, device=dev)
            for b in range(B):  # a batch entry at a time: fp32 temporaries stay small
                t[b] = (torch.randn((H, n, D), generator=gen, device=dev) * 0.5).exp_().div_(D ** 0.5).to(fdt)
            feats.append(t)
        V = torch.randn((B, H, n, d), generator=gen, device=dev).to(torch.bfloat16)
        out = torch.empty_like(V)
        fn = lambda: luna.attn_fwd_features(feats[0], feats[1], V, causal=causal, out=out)  # noqa: E731
        ms, p10, p90 = _timed_calls(fn, args.steps, args.warmup, stream, flush, sink)
        th = B * H * n
        fb = 2 if fdt == torch.bfloat16 else 4
        nbytes = th * (2 * D * fb + 2 * d * 2)
        t_hbm = nbytes / (HBM_PEAK_GBS * 1e9)
        rec = {"case": label, "shape": {"B": B, "H": H, "n": n, "d": d, "D": D, "causal": causal,
                                        "features": "bf16" if fb == 2 else "f32", "values": "bf16"},
               "path": "causal scan kernel" if (causal and fb == 2) else "fp32 GEMM",
               "ms_median": round(ms, 5), "ms_p10": round(p10, 5), "ms_p90": round(p90, 5),
               "tokens_per_s": B * n / (ms * 1e-3), "hbm_gbs": nbytes / (ms * 1e-3) / 1e9,
               "bound": "hbm", "floor_us": 1e6 * t_hbm, "roofline_frac": t_hbm / (ms * 1e-3)}
        log(f"{label}: {1e3 * ms:.1f} us, {rec['roofline_frac']:.1%} of the hbm floor")
        print(json.dumps(rec), flush=True)
        rows_out.append(rec)
        del feats, V, out
        torch.cuda.synchronize()
    if args.variants_table:
        with open(args.variants_table, "w") as fh:
            fh.write("# Feature-map variants and attention from given features on one MI355X\n\n")
            fh.write(f"Command: `python bench.py --variants --steps {args.steps} --warmup {args.warmup} "
                     f"--variants-table {args.variants_table}`\n\n")
            fh.write("One ABI call per timing, median of the timed calls with the 10th and 90th percentiles, HIP "
                     "events on the launch stream, caches flushed by a 1 GiB read before every call. Maps: the long "
                     "encoder problem's queries (1,048,576 rows, d = 64), bf16 in and out; the HBM floor is reading x "
                     "and writing phi at 8 TB/s (channel RMS: also y in fp32 written and read back); the ALU floor of "
                     "a channel MLP is its hidden units at 78.6e12 VALU lane slots/s, a unit costing its two "
                     "multiply-adds and its activation (relu 1 slot; silu and tanh 3 + two transcendentals, gelu 12 + "
                     "two, a transcendental counted as 4 slots; with a shared first layer the first multiply-add and "
                     "the activation are paid once for the L channels). Attention from features: read both feature "
                     "matrices and V, write out.\n\n")
            fh.write("| case | D | median us (p10-p90) | rows/s or tokens/s | GB/s | hidden units/s | floor us | "
                     "roofline |\n|---|---|---|---|---|---|---|---|\n")
            for r in rows_out:
                D = r.get("D", r.get("shape", {}).get("D"))
                rate = r.get("rows_per_s", r.get("tokens_per_s"))
                hu = r.get("hidden_units_per_s")
                fh.write(f"| {r['case']} | {D} | {1e3 * r['ms_median']:.1f} ({1e3 * r['ms_p10']:.1f}-"
                         f"{1e3 * r['ms_p90']:.1f}) | {rate:.3g} | {r['hbm_gbs']:.0f} | "
                         f"{'' if hu is None else f'{hu:.3g}'} | {r['floor_us']:.1f} | "
                         f"{r['roofline_frac']:.1%} {r['bound']} |\n")
        log(f"wrote {args.variants_table}")
    return 0


def distill_bench(args) -> int:
    """luna_distill (attention-distillation loss, with and without the feature-map
    parameter gradients) on the long encoder problem (non-causal) and the long causal
    problem: HIP events around each call.  The algorithmic work is the matrix-core
    products the loss needs once, S = Q K^T and P = phi(Q) phi(K)^T (2 (d + D) flops per
    visible (query, key) pair), plus the two gradient products G phi(K) and G^T phi(Q)
    (4 D per pair) with the gradients; the kernels compute S and P twice or three times
    (the softmax statistics first) and split G into two bf16 parts."""
    import torch

    from paper_2512_08061_amd import luna
    from paper_2512_08061_amd import workloads as wl

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    luna.load_library()
    stream = torch.cuda.current_stream(dev)
    for name, causal in (("long_noncausal", False), ("long_causal", True)):
        w = wl.WORKLOADS[name]
        Q, K, _ = wl.make_inputs(w, args.seed)
        p = wl.make_params(w, args.seed)
        q = torch.from_numpy(Q).to(dev).to(torch.bfloat16).contiguous()
        k = torch.from_numpy(K).to(dev).to(torch.bfloat16).contiguous()
        del Q, K
        pt = luna.PhiParams.from_arrays(p, dev, torch.bfloat16)
        D = w.M * w.L
        pairs = w.B * w.H * (w.n * (w.n + 1) // 2 if causal else w.n * w.n)
        for grads in (False, True):
            fn = lambda: luna.distill(q, k, pt, causal=causal, param_grads=grads)  # noqa: E731
            for _ in range(max(1, args.warmup // 10)):
                fn()
            torch.cuda.synchronize()
            steps = max(1, args.steps // 10)
            ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
            for e0, e1 in ev:
                e0.record(stream)
                fn()
                e1.record(stream)
            torch.cuda.synchronize()
            ms = sorted(e0.elapsed_time(e1) for e0, e1 in ev)[steps // 2]
            flops = pairs * (2 * (w.d + D) + (4 * D if grads else 0))
            tf = flops / (ms * 1e-3) / 1e12
            line = {
                "metric": "LUNA attention-distillation rows/sec (luna_distill)", "value": w.B * w.H * w.n / (ms * 1e-3),
                "unit": "rows/s", "n_gpus": 1, "steps": steps, "ms_per_step": round(ms, 4), "higher_is_better": True,
                "dtype": "bf16", "data": "synthetic (seeded)",
                "config": {"workload": f"{name} B={w.B} H={w.H} n={w.n} d={w.d} M={w.M} x L={w.L} (D={D})",
                           "causal": causal, "param_grads": grads},
                "roofline": {"bound": "mfma", "achieved": round(tf, 2), "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                             "frac": round(tf / MFMA_BF16_PEAK_TFLOPS, 4), "algorithmic_tflop": round(flops / 1e12, 3)},
            }
            log(f"{name} grads={grads}: {ms:.3f} ms, {tf:.1f} TFLOP/s")
            print(json.dumps(line), flush=True)
        del q, k
        torch.cuda.synchronize()
    return 0


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    # The GPU takes some tens of milliseconds under load to reach its full clock: the
    # default warm-up (about 0.1 s of steps) covers that, so that the timed steps see
    # the steady state.  Explicit values are used as given.
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=100)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--ramp-ms", type=float, default=200.0,
                    help="milliseconds of untimed steps before the warm-up steps (the GPU settling on the "
                         "workload); 0: none")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a plain 1 GiB device copy (for scaling HBM counters)")
    ap.add_argument("--traffic-from", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="summarise two rocprofv3 --pmc csv runs into profiles/hbm_traffic_*.json and exit")
    ap.add_argument("--traffic-command", default="",
                    help="the rocprofv3 commands that produced --traffic-from, recorded in the summary")
    ap.add_argument("--backward", action="store_true",
                    help="instead of the hot-path step: time luna_attn_bwd on the two long problems")
    ap.add_argument("--featuremap", action="store_true",
                    help="instead of the hot-path step: time luna_featuremap on the long encoder problem's queries")
    ap.add_argument("--counters-from", nargs="+", metavar="CSV",
                    help="summarise rocprofv3 --pmc csv runs (one per counter pass) into "
                         "profiles/counters_<kernel>_<workload>.md and exit")
    ap.add_argument("--counters-command", default="",
                    help="the rocprofv3 commands that produced --counters-from, recorded in the summaries")
    ap.add_argument("--graph", action="store_true",
                    help="with --decode: capture one streaming call in a HIP graph and time its replays")
    ap.add_argument("--decode", type=int, default=0, metavar="M",
                    help="instead of the hot-path step: time streaming steps of M new tokens per head "
                         "(luna_attn_causal_step) on the long causal problem's shape, after the state of "
                         "its 16384-token prefix, and print their JSON line")
    ap.add_argument("--configs", action="store_true",
                    help="instead of the hot-path step: time one call per synthetic configuration, a "
                         "sequence-length sweep and the one-channel variants, each with the caches flushed "
                         "before every timed call, and print one JSON line per configuration")
    ap.add_argument("--oracle-budget", type=float, default=1.5, metavar="SECONDS",
                    help="with --configs: seconds of oracle time per configuration (whole heads, at least one)")
    ap.add_argument("--configs-table", default="", metavar="PATH",
                    help="with --configs: also write the results as a markdown table to PATH")
    ap.add_argument("--configs-only", default="", metavar="NAMES",
                    help="with --configs: comma-separated configuration labels to run (default: all)")
    ap.add_argument("--variants", action="store_true",
                    help="instead of the hot-path step: time the feature-map variants on the long encoder "
                         "problem's queries and attention from given features, one JSON line per case")
    ap.add_argument("--variants-table", default="", metavar="PATH",
                    help="with --variants: also write the results as a markdown table to PATH")
    ap.add_argument("--distill", action="store_true",
                    help="instead of the hot-path step: time luna_distill (loss, and loss with parameter gradients) "
                         "on the two long problems")
    ap.add_argument("--variants-only", default="", metavar="NAMES",
                    help="with --variants: comma-separated case labels to run (default: all)")
    args = ap.parse_args()
    if args.traffic_from:
        return traffic_from(*args.traffic_from, args.traffic_command)
    if args.counters_from:
        return counters_from(args.counters_from, args.counters_command)
    if args.gpus != 1 and (args.decode or args.configs or args.featuremap or args.backward or args.variants
                           or args.distill):
        print("bench.py runs on one GPU only; use --gpus 1.", file=sys.stderr)
        return 2
    if args.decode:
        return decode_bench(args)
    if args.featuremap:
        return featuremap_bench(args)
    if args.backward:
        return backward_bench(args)
    if args.configs:
        return configs_bench(args)
    if args.variants:
        return variants_bench(args)
    if args.distill:
        return distill_bench(args)

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py runs on one GPU only: LUNA attention shards over (batch, head) with no "
              "communication, and this build measures the single-GPU kernel; use --gpus 1.", file=sys.stderr)
        return 2

    import torch

    from paper_2512_08061_amd import luna
    from paper_2512_08061_amd import workloads as wl

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    luna.load_library()

    w4, w5 = wl.WORKLOADS["long_noncausal"], wl.WORKLOADS["long_causal"]
    t0 = time.perf_counter()
    arrs4, arrs5 = wl.make_inputs(w4, args.seed), wl.make_inputs(w5, args.seed)
    p4, p5 = wl.make_params(w4, args.seed), wl.make_params(w5, args.seed)
    log(f"inputs generated in {time.perf_counter() - t0:.1f} s")
    up = lambda a: torch.from_numpy(a).to(dev).to(torch.bfloat16)  # noqa: E731
    q4, k4, v4 = (up(a) for a in arrs4)
    q5, k5, v5 = (up(a) for a in arrs5)
    pt4 = luna.PhiParams.from_arrays(p4, dev, torch.bfloat16)
    pt5 = luna.PhiParams.from_arrays(p5, dev, torch.bfloat16)
    nc = luna.Plan(luna.OP_ATTN, q4, k4, v4, pt4, eps=w4.eps)
    cs = luna.Plan(luna.OP_ATTN_CAUSAL, q5, k5, v5, pt5, eps=w5.eps, chunk=w5.chunk)
    torch.cuda.synchronize()

    if args.copy_calibration:
        copy_calibration(dev)

    if args.ramp_ms > 0:
        clock_ramp(lambda: (nc.run(), cs.run()), args.ramp_ms)
    for _ in range(args.warmup):
        nc.run()
        cs.run()
    torch.cuda.synchronize()
    log(f"warmup done ({args.warmup} steps)")

    stream = torch.cuda.current_stream(dev)
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    for i in range(args.steps):
        ev[i][0].record(stream)
        nc.run()
        ev[i][1].record(stream)
        cs.run()
        ev[i][2].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    ms_step = 1e3 * wall / args.steps
    ms_nc = sum(e[0].elapsed_time(e[1]) for e in ev) / args.steps
    ms_cs = sum(e[1].elapsed_time(e[2]) for e in ev) / args.steps
    log(f"timed {args.steps} steps: {ms_step:.3f} ms/step (non-causal call {ms_nc:.3f} ms, causal call {ms_cs:.3f} ms)")

    tokens = w4.B * w4.n + w5.B * w5.n
    # 256 heads fill the device, so the library runs its one-pass kernel (one workgroup per head)
    nc_kernel = "nc_fused_kernel"
    parts = {}
    for name, w, ms, causal, kern in (("long_noncausal", w4, ms_nc, False, nc_kernel),
                                      ("long_causal", w5, ms_cs, True, "causal_kernel")):
        th = w.B * w.H * w.n
        gb = bytes_per_token_head(w) * th / 1e9
        tf = flops_per_token_head(w, causal) * th / 1e12
        t_hbm, t_mfma = gb / HBM_PEAK_GBS, tf / MFMA_BF16_PEAK_TFLOPS
        parts[name] = {
            "shape": {"B": w.B, "H": w.H, "n": w.n, "d": w.d, "M": w.M, "L": w.L, "D": w.M * w.L,
                      "causal": causal, **({"chunk": w.chunk} if causal else {})},
            "kernels": kern,
            "ms_per_call": round(ms, 4),
            "tokens_per_s": w.B * w.n / (ms / 1e3),
            "head_tokens_per_s": th / (ms / 1e3),
            "attn_tflops": tf / (ms / 1e3),
            "hbm_gbs": gb / (ms / 1e3),
            "hbm_frac": (gb / (ms / 1e3)) / HBM_PEAK_GBS,
            "mfma_frac": (tf / (ms / 1e3)) / MFMA_BF16_PEAK_TFLOPS,
            "bound": "hbm" if t_hbm >= t_mfma else "mfma",
            "roofline_frac": max(t_hbm, t_mfma) / (ms / 1e3),
            "algorithmic_bytes": int(gb * 1e9),
            "algorithmic_flops": int(tf * 1e12),
        }

    dom = max(parts, key=lambda k: parts[k]["ms_per_call"])
    P = parts[dom]
    kname = "causal_kernel" if dom == "long_causal" else P["kernels"]
    roofline = {
        "bound": P["bound"],
        "achieved": round(P["hbm_gbs"] if P["bound"] == "hbm" else P["attn_tflops"], 2),
        "peak": HBM_PEAK_GBS if P["bound"] == "hbm" else MFMA_BF16_PEAK_TFLOPS,
        "unit": "GB/s" if P["bound"] == "hbm" else "TFLOP/s",
        "frac": round(P["roofline_frac"], 4),
        "traffic": measured_traffic(kname, dom) if kname in KERNEL_SOURCES else None,
        # matrix-core busy share of the kernel's (scan launch's) SIMD cycles, from the
        # committed counter summary (null once the kernel has changed since)
        "mfma_busy": measured_figure("causal_kernel_scan_launch" if kname == "causal_kernel" else kname, dom,
                                     kname, "MFMA busy") if kname in KERNEL_SOURCES else None,
        # the LDS's active share of the CU cycles and the bank-conflict share of those
        # cycles, from the same summary: the LDS, not HBM, is what these kernels are
        # bound by (their tables, phi tiles and operand reads)
        "lds_busy": measured_figure("causal_kernel_scan_launch" if kname == "causal_kernel" else kname, dom,
                                    kname, "LDS active") if kname in KERNEL_SOURCES else None,
        "lds_conflict_share": measured_figure("causal_kernel_scan_launch" if kname == "causal_kernel" else kname,
                                              dom, kname, "LDS bank-conflict cycles per LDS-active cycle")
        if kname in KERNEL_SOURCES else None,
        "kernel": kname,
        "workload": dom,
        "timing": "HIP events on the launch stream around each ABI call (includes the table-build kernel; the "
                  "causal call is two scan launches of causal_kernel)",
    }

    out = {
        "metric": METRIC,
        "value": round(tokens / (ms_step / 1e3), 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "clock_ramp_ms": args.ramp_ms,
        "clock_ramp": "the step's own calls, untimed, before the warm-up steps",
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded; shapes and distributions of the paper's encoder and long-context settings)",
        "config": {
            "workload": "long_noncausal 32x8x4096x64 D=128 + long_causal 8x16x16384x128 D=256 chunk=64, bf16",
            "tokens_per_step": tokens,
            "parts": parts,
        },
        "roofline": roofline,
        "cpu_baseline": None,
        "parity": None,
    }
    if not args.no_cpu_baseline:
        t0 = time.perf_counter()
        refs = {}
        out["cpu_baseline"] = cpu_baseline(w4, arrs4, p4, w5, arrs5, p5, refs)
        log(f"cpu baseline in {time.perf_counter() - t0:.1f} s")
        out["parity"] = parity_check(refs, {"long_noncausal": nc.out, "long_causal": cs.out})
        log(f"parity of the timed outputs against the oracle: {out['parity']}")
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
