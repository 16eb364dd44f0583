#!/usr/bin/env python3
"""Throughput of the ACP-SGD compressor + decompressor on one MI355X.

One step = every bucket of the workload compressed (acp_compress), its factor buffer passed
on unchanged (the all-reduce of one worker) and decompressed (acp_decompress) into a separate
output buffer; steps alternate P-steps and Q-steps.  Inputs are two resident gradient sets
used in turn (2.7 GB for BERT-large, more than the 256 MB last-level cache).

value = algorithmic bytes per step / measured step time, where the algorithmic bytes are
16 B per gradient element (read M, read E, write E, write M_hat; pack + unpack for raw
vectors) plus the factor traffic 10 r (n + m) B per matrix (average of a P-step and a Q-step).

Also reported: the roofline entry of the dominant kernel (its own bytes per launch over its
event-timed average launch duration) and the CPU oracle's throughput on a bounded sample of
the same workload.
"""

from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

HBM_PEAK_GBS = 8000.0
MFMA_F32_PEAK_TFLOPS = 157.3  # dense fp32 matrix-core peak of MI355X


def algorithmic_bytes(wl, rank):
    """(bytes per average step, bytes of P-step compress, of Q-step compress, of decompress)."""
    nc = n1 = fac = 0
    fac_p = fac_q = 0
    for p in wl.params:
        s = p.shape
        if len(s) >= 2:
            n, m = s[0], p.numel // s[0]
            if rank < min(n, m):
                nc += p.numel
                fac += 10 * rank * (n + m)
                fac_p += 4 * rank * (m + n)       # read Q, write P
                fac_q += 4 * rank * (n + m)       # read P, write Q
                continue
        n1 += p.numel
    step = 16 * nc + 16 * n1 + fac
    comp = 12 * nc + 8 * n1
    return step, comp + fac_p, comp + fac_q, 4 * nc + 8 * n1, nc, n1


def cpu_baseline(wl, seconds: float = 12.0):
    """The fp64 oracle on a bounded sample of the same workload: every bucket, steps 1, 2, ...
    (P-steps and Q-steps in turn) until about ``seconds`` of oracle work (input generation is
    not timed)."""
    from threadpoolctl import threadpool_info
    import synthgrad as sg
    from oracle.acp import AcpOracle
    from oracle.layout import plan

    shapes = [p.shape for p in wl.params]
    lay = plan(shapes, wl.rank, wl.cap_bytes)
    orc = AcpOracle(shapes, wl.rank, seed=wl.seed, cap_bytes=wl.cap_bytes)
    step_bytes = algorithmic_bytes(wl, wl.rank)[0]
    elapsed, steps = 0.0, 0
    while elapsed < seconds and steps < 20:
        t = steps + 1
        grads = sg.gradient_set(wl, t)
        tb = time.perf_counter()
        for b in range(len(lay.buckets)):
            buf = orc.compress_bucket(t, b, grads)
            orc.decompress_bucket(t, b, buf)
        elapsed += time.perf_counter() - tb
        steps += 1
        del grads
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    return {"value": round(steps * step_bytes / elapsed / 1e9, 4), "unit": "GB/s", "cores": int(threads),
            "kind": "oracle",
            "sample": f"{wl.name}: all {len(lay.buckets)} buckets, steps 1-{steps}, fp64 NumPy "
                      f"(OpenBLAS), {elapsed:.1f} s of oracle work"}


def kernel_families(rank: int):
    """(label, ACP_KERNEL_* family, kernel symbol prefix) of the timed kernel families: the rank-4
    register-resident kernels; the one-wave MFMA kernels of ranks 8 to 32; from rank 64 the
    rank-split MFMA compress kernels, with the one-wave decompress up to rank 128 and the
    rank-split one at 256; and the separate orthogonalisation kernels."""
    from paper_2306_08881_amd import _lib as L
    if rank >= 64:
        p, q, d = "k_spstep", "k_sqstep", "k_srecon" if rank >= 256 else "k_wrecon"
    elif rank >= 8:
        p, q, d = "k_wpstep", "k_wqstep", "k_wrecon"
    else:
        p, q, d = "k_pfused", "k_qstep", "k_recon4"
    orth = ("k_apply, k_wfact, k_gsum, k_chol" if rank >= 128 else "k_apply, k_wfact, k_chol") if rank >= 8 else "k_chol"
    return [(f"P-step compress ({p})", L.ACP_KERNEL_P_STEP, p),
            (f"Q-step compress ({q})", L.ACP_KERNEL_Q_STEP, q),
            ("Q-step finish (k_qfin)", L.ACP_KERNEL_Q_FINISH, "k_qfin"),
            (f"decompress ({d})", L.ACP_KERNEL_RECONSTRUCT, d),
            (f"orthogonalisation ({orth})", L.ACP_KERNEL_ORTH, orth)]


WORKLOAD_KIND = {"conv": "one 256x64x3x3 convolution gradient", "resnet50": "ResNet-50-shaped gradients",
                 "resnet152": "ResNet-152-shaped gradients", "bert_base": "BERT-base-shaped gradients",
                 "bert_large": "BERT-large-shaped gradients"}
TRAFFIC_FILE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "profiles", "traffic.txt")


def kernel_source_hash() -> str:
    """Fingerprint of the kernel sources and of the planner that sets their tiles and launches."""
    import hashlib
    csrc = os.path.join(os.path.dirname(os.path.abspath(__file__)), "paper_2306_08881_amd", "csrc")
    h = hashlib.sha256()
    for f in ("kernels.hip", "wide.hip", "device.hpp", "acp_internal.hpp", "plan.cpp"):
        h.update(open(os.path.join(csrc, f), "rb").read())
    return h.hexdigest()[:16]


def pmc_summary(fetch_csv: str, write_csv: str, workload: str):
    """Per-kernel HBM bytes per dispatch from FETCH_SIZE / WRITE_SIZE runs, each scaled by what
    the counter reads for the copy probe (a device-to-device copy of 1 GiB), written to
    profiles/traffic.txt with the kernel source hash they were taken on."""
    import csv
    from collections import defaultdict

    def load(path):
        d = defaultdict(list)
        for r in csv.DictReader(open(path)):
            d[r["Kernel_Name"]].append(float(r["Counter_Value"]))
        return d

    f, w = load(fetch_csv), load(write_csv)
    gib_kib = float(1 << 20)
    copy_f = [v for k, vs in f.items() if "copyBuffer" in k for v in vs if v > 0.25 * gib_kib]
    copy_w = [v for k, vs in w.items() if "copyBuffer" in k for v in vs if v > 0.5 * gib_kib]
    sf = gib_kib / (sum(copy_f) / len(copy_f))
    sw = gib_kib / (sum(copy_w) / len(copy_w))
    out = {"source_hash": kernel_source_hash(), "workload": workload, "fetch_scale": round(sf, 4),
           "write_scale": round(sw, 4), "kernels": {}}
    print(f"| kernel | dispatches | FETCH_SIZE KiB/dispatch | WRITE_SIZE KiB/dispatch | HBM bytes/dispatch (scaled) |")
    print("|---|---|---|---|---|")
    for name in sorted(f):
        if "acp::" not in name and "copyBuffer" not in name:
            continue
        fv, wv = f[name], w.get(name, [0.0])
        fa, wa = sum(fv) / len(fv), sum(wv) / len(wv)
        hbm = (fa * sf + wa * sw) * 1024
        short = name[name.find("k_"):name.find("(", name.find("k_"))] if "k_" in name else name
        out["kernels"][short] = {"dispatches": len(fv), "fetch_kib": round(fa, 1), "write_kib": round(wa, 1),
                                 "hbm_bytes": round(hbm, 1)}
        print(f"| {short} | {len(fv)} | {fa:.0f} | {wa:.0f} | {hbm:.4g} |")
    print(f"\ncopy probe scale factors: FETCH_SIZE x{sf:.4f}, WRITE_SIZE x{sw:.4f}")
    os.makedirs(os.path.dirname(TRAFFIC_FILE), exist_ok=True)
    json.dump(out, open(TRAFFIC_FILE, "w"), indent=1)


def measured_traffic(workload: str, family: str, launches: int):
    """HBM bytes per launch of the dominant kernel family from profiles/traffic.txt, or None
    when the counters were taken on other kernel sources or for another workload."""
    try:
        t = json.load(open(TRAFFIC_FILE))
    except (OSError, ValueError):
        return None
    if t.get("source_hash") != kernel_source_hash() or t.get("workload") not in (None, workload):
        return None
    sym = next((k[2] for k in kernel_families(4) + kernel_families(8) + kernel_families(64) + kernel_families(256) if k[0] == family), None)
    ks = [v for k, v in t["kernels"].items() if sym and k.startswith(sym)]
    if not ks:
        return None
    # dispatch-weighted bytes per launch of the family (its launches of every class)
    tot = sum(v["hbm_bytes"] * v["dispatches"] for v in ks)
    n = sum(v["dispatches"] for v in ks)
    return round(tot / n, 1) if n else None


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="bert_large_r4")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--streams", type=int, default=4,
                    help="per-bucket mode: HIP streams the buckets are spread over (bucket b on "
                         "stream b %% streams)")
    ap.add_argument("--mode", choices=["all", "bucket"], default="all",
                    help="all: acp_compress_all / acp_decompress_all (every bucket in one launch per "
                         "kernel kind); bucket: acp_compress / acp_decompress per bucket")
    ap.add_argument("--compare", action="store_true",
                    help="also time the other mode and report it in config")
    ap.add_argument("--pmc-summary", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="summarise two rocprofv3 --pmc runs of this benchmark (FETCH_SIZE, then "
                         "WRITE_SIZE counter_collection.csv) and exit")
    args = ap.parse_args()
    if args.pmc_summary:
        pmc_summary(*args.pmc_summary, workload=args.workload)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported by this build "
              "(the compressor is data-parallel: each rank runs this same step on its own GPU).",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    import synthgrad as sg
    from paper_2306_08881_amd import _lib as L
    from paper_2306_08881_amd.acp import Acp

    wl = sg.WORKLOADS[args.workload]
    shapes = [p.shape for p in wl.params]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    t_setup = time.time()
    acp = Acp(shapes, wl.rank, seed=wl.seed, cap_bytes=wl.cap_bytes, device=dev)
    nb = acp.num_buckets()
    info = [acp.bucket_info(b) for b in range(nb)]
    lay = [acp.layout(b) for b in range(nb)]
    gsets = []
    for key in (1, 2):
        grads = sg.gradient_set(wl, key, threads=16)
        bufs = []
        for b in range(nb):
            host = np.empty(info[b][1], np.float32)
            tids, go = lay[b][0], lay[b][1]
            for k, tid in enumerate(tids):
                g = grads[int(tid)].reshape(-1)
                host[go[k]:go[k] + g.size] = g
            bufs.append(torch.from_numpy(host).to(dev))
        gsets.append(bufs)
        del grads
    fbuf = [torch.zeros(max(i[2], i[3], 4), dtype=torch.float32, device=dev) for i in info]
    out = [torch.zeros(i[1], dtype=torch.float32, device=dev) for i in info]
    main = torch.cuda.current_stream()
    nstreams = max(1, args.streams)
    streams = [main] if nstreams == 1 else [torch.cuda.Stream(device=dev) for _ in range(nstreams)]
    torch.cuda.synchronize()
    print(f"# setup {time.time() - t_setup:.1f}s: {wl.name}, {nb} buckets, {wl.numel} parameters, "
          f"{nstreams} stream(s)", file=sys.stderr, flush=True)

    step_no = [0]

    def one_step(mode):
        step_no[0] += 1
        t = step_no[0]
        g = gsets[t % 2]
        if mode == "all":
            acp.compress_all(t, g, fbuf, stream=main)
            acp.decompress_all(t, fbuf, out, stream=main)
            return
        if nstreams > 1:
            fork = torch.cuda.Event()
            fork.record(main)
            for s in streams:
                s.wait_event(fork)
        for b in range(nb):
            s = streams[b % nstreams]
            acp.compress(t, b, g[b], fbuf[b], stream=s)
            acp.decompress(t, b, fbuf[b], out[b], stream=s)
        if nstreams > 1:
            for s in streams:
                join = torch.cuda.Event()
                join.record(s)
                main.wait_event(join)

    def timed(steps, mode):
        torch.cuda.synchronize()
        start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        start.record(main)
        for _ in range(steps):
            one_step(mode)
        end.record(main)
        torch.cuda.synchronize()
        return start.elapsed_time(end) / steps

    def per_step(steps, mode, flush=None):
        """Per-step times (ms): HIP events around each step on the caller's stream; `flush`, when
        given, runs between steps outside the events."""
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(steps)]
        torch.cuda.synchronize()
        for e0, e1 in ev:
            if flush is not None:
                flush()
            e0.record(main)
            one_step(mode)
            e1.record(main)
        torch.cuda.synchronize()
        return np.array([e0.elapsed_time(e1) for e0, e1 in ev])

    other = "bucket" if args.mode == "all" else "all"
    for _ in range(args.warmup):
        one_step(args.mode)
    if step_no[0] % 2:  # start every timed region on a P-step
        one_step(args.mode)
    steps = args.steps + (args.steps % 2)
    ms = timed(steps, args.mode)
    ms_other = timed(steps, other) if args.compare else None

    # per-step statistics (a pass of its own, so the timed region above holds no extra events):
    # every step, P-steps (odd t) and Q-steps apart; then the same with the 256 MB last-level
    # (MALL) cache flushed before each step by an untimed 512 MB fill
    t_step = per_step(steps, args.mode)
    scratch = torch.empty(1 << 27, dtype=torch.float32, device=dev)
    t_flush = per_step(steps, args.mode, flush=lambda: scratch.fill_(1.0))
    del scratch

    # per-kernel pass: the same steps again with every launch of one kernel family bracketed by
    # HIP events on its own stream (acp_profile_*), once per family
    fams = kernel_families(wl.rank)
    kern = {}
    for name, fam, _ in fams:
        acp.profile_start(fam, 64 * nb * steps)
        timed(steps, args.mode)
        n, sec, by = acp.profile_stop()
        if n:
            kern[name] = {"launches": n, "avg_launch_us": sec / n * 1e6, "bytes_per_launch": by / n,
                          "gbs": by / sec / 1e9, "ms_per_step": sec / steps * 1e3}
    # the dominant kernel: the Q-step kernel, the longest-running single kernel of the step (one
    # launch per Q-step); at rank 4 the P-step time is split over one k_pfused launch per column
    # class
    dom = fams[1][0] if fams[1][0] in kern else max(kern, key=lambda k: kern[k]["ms_per_step"])
    dk = kern[dom]
    step_bytes, bp, bq, bd, nc, n1 = algorithmic_bytes(wl, wl.rank)
    gbs = step_bytes / (ms * 1e-3) / 1e9
    roof = {"bound": "hbm", "achieved": round(dk["gbs"], 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(dk["gbs"] / HBM_PEAK_GBS, 4),
            "traffic": measured_traffic(wl.name, dom, dk["launches"]),
            "kernel": dom, "avg_launch_us": round(dk["avg_launch_us"], 3),
            "bytes_per_launch": round(dk["bytes_per_launch"], 1)}
    if wl.rank >= 8 and dom == fams[1][0]:
        # the MFMA Q-step does one rank-r correction and one rank-r product per compressed element
        # (4 r flop); past the machine balance its bound is the fp32 matrix-core peak
        flops = 4 * wl.rank * nc / (dk["launches"] / (steps / 2))
        t_hbm = dk["bytes_per_launch"] / (HBM_PEAK_GBS * 1e9)
        t_mfma = flops / (MFMA_F32_PEAK_TFLOPS * 1e12)
        tflops = flops / (dk["avg_launch_us"] * 1e-6) / 1e12
        roof["flops_per_launch"] = flops
        if t_mfma > t_hbm:
            roof.update({"bound": "mfma", "achieved": round(tflops, 2), "peak": MFMA_F32_PEAK_TFLOPS,
                         "unit": "TFLOP/s", "frac": round(tflops / MFMA_F32_PEAK_TFLOPS, 4),
                         "hbm_gbs": round(dk["gbs"], 2)})
    res = {
        "metric": "ACP-SGD compress+decompress gradient GB/s and % HBM peak, BERT-large r=4",
        "value": round(gbs, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded N(0, 0.02^2) gradients of the workload's shapes)",
        "config": {"workload": f"{wl.name}: {WORKLOAD_KIND[wl.name.rsplit('_', 1)[0].split('256')[0]]}, "
                               f"{len(shapes)} tensors, {wl.numel} parameters, rank {wl.rank}, "
                               f"{wl.cap_bytes >> 20} MiB buckets ({nb})",
                   "rank": wl.rank, "buckets": nb, "parameters": wl.numel, "mode": args.mode,
                   "streams": nstreams if args.mode == "bucket" else 1,
                   "pct_hbm_peak": round(100 * gbs / HBM_PEAK_GBS, 2),
                   "gradient_elements_per_s": round(wl.numel / (ms * 1e-3), 1),
                   "algorithmic_bytes_per_step": step_bytes,
                   "kernels": {k: {kk: round(vv, 3) for kk, vv in v.items()} for k, v in kern.items()}},
        "roofline": roof,
    }
    res["config"]["step_ms"] = {"mean": round(float(t_step.mean()), 4), "std": round(float(t_step.std()), 4),
                                "median": round(float(np.median(t_step)), 4),
                                "p_step_mean": round(float(t_step[0::2].mean()), 4),
                                "q_step_mean": round(float(t_step[1::2].mean()), 4)}
    res["config"]["mall_flushed"] = {"mean_ms": round(float(t_flush.mean()), 4),
                                     "gbs": round(step_bytes / (float(t_flush.mean()) * 1e-3) / 1e9, 2)}
    if ms_other is not None:
        res["config"][f"ms_per_step_{other}_mode"] = round(ms_other, 4)
        res["config"][f"gbs_{other}_mode"] = round(step_bytes / (ms_other * 1e-3) / 1e9, 2)
    # copy probe: device-to-device copy of 1 GiB, the achievable streaming ceiling on this GPU
    src = torch.empty(1 << 28, dtype=torch.float32, device=dev).normal_()
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    c0.record(main)
    for _ in range(10):
        dst.copy_(src)
    c1.record(main)
    torch.cuda.synchronize()
    copy_gbs = 10 * 2 * src.numel() * 4 / (c0.elapsed_time(c1) * 1e-3) / 1e9
    res["config"]["copy_probe_gbs"] = round(copy_gbs, 1)
    res["config"]["pct_of_copy_probe"] = round(100 * gbs / copy_gbs, 2)
    del src, dst

    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(wl)
    res["cpu_baseline_host"] = {"cpu": platform.processor() or platform.machine(),
                                "affinity_cores": len(os.sched_getaffinity(0))}
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
