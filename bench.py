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
event-timed average launch duration, and its HBM traffic from the workload's rocprofv3 counter
file when that was taken on the current kernel sources); the streaming ceilings of the probe
kernels (libacp_probe.so: the compress kernels' 2-read-1-write mix and the decompress kernels'
write-only stream) and the step's fraction of their mix; the CPU oracle's throughput on a bounded
sample of the same workload; with --compare-powersgd, Power-SGD's compress and step times beside
ACP-SGD's on the same workload.
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
    pools = threadpool_info()
    threads = max([i.get("num_threads", 1) for i in pools] or [1])
    blas = ", ".join(sorted({f"{i.get('internal_api')} {i.get('version')}" for i in pools if i.get("user_api") == "blas"}))
    return {"value": round(steps * step_bytes / elapsed / 1e9, 4), "unit": "GB/s", "cores": int(threads),
            "kind": "oracle",
            "sample": f"{wl.name}: all {len(lay.buckets)} buckets, steps 1-{steps}, fp64 NumPy "
                      f"({blas or 'BLAS'}, {threads} threads), {elapsed:.1f} s of oracle work"}


def host_info():
    """The host the CPU baseline ran on: CPU model, cores this process may use, BLAS pools."""
    from threadpoolctl import threadpool_info
    model = platform.processor() or platform.machine()
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    pools = [{"api": i.get("internal_api"), "version": i.get("version"), "threads": i.get("num_threads")}
             for i in threadpool_info() if i.get("user_api") == "blas"]
    return {"cpu": model, "affinity_cores": len(os.sched_getaffinity(0)), "blas": pools}


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
PROFILES = os.path.join(os.path.dirname(os.path.abspath(__file__)), "profiles")
METRIC_NAME = {"conv256x576": "one 256x576 matrix", "resnet50": "ResNet-50", "resnet152": "ResNet-152",
               "bert_base": "BERT-base", "bert_large": "BERT-large"}


def traffic_file(workload: str) -> str:
    """Per-kernel HBM bytes of a workload's benchmark from rocprofv3 counters (pmc_summary)."""
    return os.path.join(PROFILES, f"{workload}_traffic.txt")


def metric_of(wl) -> str:
    base, r = wl.name.rsplit("_r", 1)
    return f"ACP-SGD compress+decompress gradient GB/s and % HBM peak, {METRIC_NAME[base]} r={r}"


def kernel_source_hash() -> str:
    """Fingerprint of the code of the kernel sources and of the planner that sets their tiles and
    launches: comments and blank lines are left out, so that a reworded comment keeps counters
    that were taken on the same code."""
    import hashlib
    import re
    csrc = os.path.join(os.path.dirname(os.path.abspath(__file__)), "paper_2306_08881_amd", "csrc")
    h = hashlib.sha256()
    for f in ("kernels.hip", "wide.hip", "device.hpp", "acp_internal.hpp", "plan.cpp", "probe.hip"):
        text = open(os.path.join(csrc, f), encoding="utf-8").read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        lines = (re.sub(r"//.*", "", ln).rstrip() for ln in text.splitlines())
        h.update("\n".join(ln for ln in lines if ln).encode())
    return h.hexdigest()[:16]


PROBE_FLOATS = 1 << 28  # 1 GiB per probe array


def pmc_summary(fetch_csv: str, write_csv: str, workload: str):
    """Per-kernel HBM bytes per dispatch from FETCH_SIZE / WRITE_SIZE runs, each scaled by what
    the counter reads for the streaming probe of known bytes (k_probe_rrw over 1 GiB arrays:
    2 GiB read, 1 GiB written), written to profiles/traffic.txt with the kernel source hash they
    were taken on."""
    import csv
    from collections import defaultdict

    def load(path):
        d = defaultdict(list)
        for r in csv.DictReader(open(path)):
            d[r["Kernel_Name"]].append(float(r["Counter_Value"]))
        return d

    f, w = load(fetch_csv), load(write_csv)
    gib_kib = PROBE_FLOATS * 4 / 1024.0
    probe_f = [v for k, vs in f.items() if "k_probe_rrw" in k for v in vs]
    probe_w = [v for k, vs in w.items() if "k_probe_rrw" in k for v in vs]
    # every footprint of the probe moves the same bytes per dispatch
    sf = 2 * gib_kib / (sum(probe_f) / len(probe_f))
    sw = gib_kib / (sum(probe_w) / len(probe_w))
    out = {"source_hash": kernel_source_hash(), "workload": workload, "fetch_scale": round(sf, 4),
           "write_scale": round(sw, 4), "kernels": {}}
    print(f"| kernel | dispatches | FETCH_SIZE KiB/dispatch | WRITE_SIZE KiB/dispatch | HBM bytes/dispatch (scaled) |")
    print("|---|---|---|---|---|")
    for name in sorted(f):
        if "acp::" not in name and "k_probe" not in name:
            continue
        fv, wv = f[name], w.get(name, [0.0])
        fa, wa = sum(fv) / len(fv), sum(wv) / len(wv)
        hbm = (fa * sf + wa * sw) * 1024
        short = name[name.find("k_"):name.find("(", name.find("k_"))] if "k_" in name else name
        out["kernels"][short] = {"dispatches": len(fv), "fetch_kib": round(fa, 1), "write_kib": round(wa, 1),
                                 "hbm_bytes": round(hbm, 1)}
        print(f"| {short} | {len(fv)} | {fa:.0f} | {wa:.0f} | {hbm:.4g} |")
    print(f"\nscale factors from the probe k_probe_rrw (2 GiB read, 1 GiB written per dispatch): "
          f"FETCH_SIZE x{sf:.4f}, WRITE_SIZE x{sw:.4f}")
    os.makedirs(PROFILES, exist_ok=True)
    json.dump(out, open(traffic_file(workload), "w"), indent=1)


def measured_traffic(workload: str, family: str):
    """(HBM bytes per launch of the dominant kernel family, provenance text) from the workload's
    counter file, or (None, reason) when the counters were taken on other kernel sources."""
    path = traffic_file(workload)
    rel = os.path.relpath(path, os.path.dirname(os.path.abspath(__file__)))
    try:
        t = json.load(open(path))
    except (OSError, ValueError):
        return None, f"no counters: {rel} is missing"
    if t.get("source_hash") != kernel_source_hash() or t.get("workload") not in (None, workload):
        return None, f"no counters: {rel} was taken on other kernel sources"
    sym = next((k[2] for k in kernel_families(4) + kernel_families(8) + kernel_families(64) + kernel_families(256) if k[0] == family), None)
    ks = [v for k, v in t["kernels"].items() if sym and k.startswith(sym)]
    if not ks:
        return None, f"no counters for {sym} in {rel}"
    # dispatch-weighted bytes per launch of the family (its launches of every class)
    tot = sum(v["hbm_bytes"] * v["dispatches"] for v in ks)
    n = sum(v["dispatches"] for v in ks)
    src = (f"{rel}: rocprofv3 --pmc FETCH_SIZE, then WRITE_SIZE, over this benchmark on kernel sources "
           f"{t['source_hash']}, not measured in this run; each counter scaled by what it reads for the "
           f"probe k_probe_rrw of known bytes (FETCH_SIZE x{t['fetch_scale']}, WRITE_SIZE x{t['write_scale']})")
    return (round(tot / n, 1) if n else None), src


def probe_ceilings(dev, stream):
    """Streaming ceilings of this GPU from the probe kernels (libacp_probe.so) over 1 GiB arrays:
    the compress kernels' mix (read M, read E, write E in place) and the decompress kernels'
    (write only), both nontemporal, each the best of 4, 8, 16 and 32 KB per workgroup; and the
    step's mix of the two (12 B : 4 B per element)."""
    import ctypes as C
    import torch
    lib = C.CDLL(os.path.join(os.path.dirname(os.path.abspath(__file__)), "paper_2306_08881_amd",
                              "libacp_probe.so"))
    lib.acp_probe_rrw.argtypes = [C.c_void_p, C.c_void_p, C.c_int64, C.c_int, C.c_void_p]
    lib.acp_probe_w.argtypes = [C.c_void_p, C.c_int64, C.c_float, C.c_int, C.c_void_p]
    m = torch.empty(PROBE_FLOATS, dtype=torch.float32, device=dev).normal_()
    e = torch.zeros_like(m)
    sp = stream.cuda_stream

    def rate(fn, nbytes, reps=10):
        for _ in range(3):
            if fn() != 0:
                raise RuntimeError("probe launch failed")
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(stream)
        for _ in range(reps):
            fn()
        b.record(stream)
        torch.cuda.synchronize()
        return reps * nbytes / (a.elapsed_time(b) * 1e-3) / 1e9

    rrw = {kb: rate(lambda: lib.acp_probe_rrw(m.data_ptr(), e.data_ptr(), PROBE_FLOATS, kb, sp), 12 * PROBE_FLOATS)
           for kb in (4, 8, 16, 32)}
    w = {kb: rate(lambda: lib.acp_probe_w(e.data_ptr(), PROBE_FLOATS, 1.0, kb, sp), 4 * PROBE_FLOATS)
         for kb in (4, 8, 16, 32)}
    del m, e
    best_rrw, best_w = max(rrw.values()), max(w.values())
    mix = 16.0 / (12.0 / best_rrw + 4.0 / best_w)
    return {"compress_mix_gbs": round(best_rrw, 1), "write_gbs": round(best_w, 1), "step_mix_gbs": round(mix, 1),
            "by_kb_per_workgroup": {"compress_mix": {k: round(v, 1) for k, v in rrw.items()},
                                    "write": {k: round(v, 1) for k, v in w.items()}},
            "probe": "k_probe_rrw (e = m + e in place) and k_probe_w (fill), 1 GiB arrays, nontemporal, "
                     "best of 4-32 KB per workgroup and stream"}


def compare_powersgd(acp, wl, shapes, gsets, fbuf, out, dev, stream, steps, warmup, step_no):
    """ACP-SGD and Power-SGD (Algorithm 1, left, with error feedback) on the same workload and
    resident gradients, all buckets per call: per step, events around the compress calls (ACP-SGD:
    acp_compress_all; Power-SGD: acp_powersgd_p_all and acp_powersgd_q_all, the all-reduces being
    the identity of one worker) and around the decompress call."""
    import numpy as np
    import torch
    from paper_2306_08881_amd.acp import Acp

    def phases(step_fn, n):
        ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(n)]
        torch.cuda.synchronize()
        for e in ev:
            step_fn(e)
        torch.cuda.synchronize()
        c = np.array([e[0].elapsed_time(e[1]) for e in ev])
        d = np.array([e[1].elapsed_time(e[2]) for e in ev])
        return float(c.mean()), float(d.mean()), float((c + d).mean())

    def acp_step(e):
        step_no[0] += 1
        t = step_no[0]
        e[0].record(stream)
        acp.compress_all(t, gsets[t % 2], fbuf, stream=stream)
        e[1].record(stream)
        acp.decompress_all(t, fbuf, out, stream=stream)
        e[2].record(stream)

    if step_no[0] % 2:
        acp_step([torch.cuda.Event() for _ in range(3)])
    a_c, a_d, a_s = phases(acp_step, steps)

    ps = Acp(shapes, wl.rank, seed=wl.seed, cap_bytes=wl.cap_bytes, device=dev, powersgd=True)
    nb = ps.num_buckets()
    info = [ps.bucket_info(b) for b in range(nb)]
    pbuf = [torch.zeros(max(i[2], 4), dtype=torch.float32, device=dev) for i in info]
    qbuf = [torch.zeros(max(i[3], 4), dtype=torch.float32, device=dev) for i in info]
    k = [0]

    def psgd_step(e):
        k[0] += 1
        t = k[0]
        g = gsets[t % 2]
        e[0].record(stream)
        ps.powersgd_p_all(t, g, pbuf, stream=stream)
        ps.powersgd_q_all(t, g, pbuf, qbuf, stream=stream)
        e[1].record(stream)
        ps.powersgd_decompress_all(t, qbuf, out, stream=stream)
        e[2].record(stream)

    for _ in range(warmup):
        psgd_step([torch.cuda.Event() for _ in range(3)])
    p_c, p_d, p_s = phases(psgd_step, steps)
    ps.close()
    return {"acp_compress_ms": round(a_c, 4), "acp_decompress_ms": round(a_d, 4), "acp_step_ms": round(a_s, 4),
            "powersgd_compress_ms": round(p_c, 4), "powersgd_decompress_ms": round(p_d, 4),
            "powersgd_step_ms": round(p_s, 4),
            "compress_time_ratio": round(p_c / a_c, 3), "step_time_ratio": round(p_s / a_s, 3),
            "bytes_per_compressed_element": {"acp": 16, "powersgd": 24},
            "note": "events around each call group of every step (a pass of its own); Power-SGD's "
                    "compress is both halves (P product, orthogonalisation of the all-reduced P, Q "
                    "product), ACP-SGD's one product with the orthogonalisation of the reused factor"}


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
    ap.add_argument("--mode", choices=["all", "bucket", "graph"], default="all",
                    help="all: acp_compress_all / acp_decompress_all (every bucket in one launch per "
                         "kernel kind); bucket: acp_compress / acp_decompress per bucket; graph: the "
                         "all-bucket calls of one odd and one even step captured into two HIP graphs "
                         "and replayed in turn")
    ap.add_argument("--compare", action="store_true",
                    help="also time the other mode and report it in config")
    ap.add_argument("--compare-powersgd", action="store_true",
                    help="also run Power-SGD (Algorithm 1, left, with error feedback) on the same "
                         "workload and report its compress and step times beside ACP-SGD's")
    ap.add_argument("--pmc-summary", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="summarise two rocprofv3 --pmc runs of this benchmark (FETCH_SIZE, then "
                         "WRITE_SIZE counter_collection.csv) and exit")
    args = ap.parse_args()
    if args.pmc_summary:
        pmc_summary(*args.pmc_summary, workload=args.workload)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported "
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
    graphs = []     # [odd step, even step] after capture()
    replayed = [0]  # replays so far: the context's step record does not count them

    def one_step(mode, stream=None):
        if mode == "graph":
            replayed[0] += 1
            graphs[(replayed[0] - 1) % 2].replay()
            return
        step_no[0] += 1
        t = step_no[0]
        g = gsets[t % 2]
        if mode == "all":
            st = main if stream is None else stream
            acp.compress_all(t, g, fbuf, stream=st)
            acp.decompress_all(t, fbuf, out, stream=st)
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

    def capture():
        """One odd and one even step of the all-bucket calls captured into HIP graphs (at steady
        state: the step's kernel arguments then depend only on its parity).  Capture enqueues
        nothing; replays of the pair, in turn, run the steps."""
        assert step_no[0] % 2 == 0 and step_no[0] >= 2
        side = torch.cuda.Stream(device=dev)
        side.wait_stream(main)
        for _ in range(2):
            gr = torch.cuda.CUDAGraph()
            with torch.cuda.graph(gr, stream=side):
                one_step("all", stream=torch.cuda.current_stream())
            graphs.append(gr)
        main.wait_stream(side)

    other = "bucket" if args.mode != "bucket" else "all"
    eager = "all" if args.mode == "graph" else args.mode
    for _ in range(max(args.warmup, 2)):
        one_step(eager)
    if step_no[0] % 2:  # start every timed region on a P-step
        one_step(eager)
    if args.mode == "graph":
        capture()
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
        timed(steps, eager)
        n, sec, by = acp.profile_stop()
        if n:
            kern[name] = {"launches": n, "avg_launch_us": sec / n * 1e6, "bytes_per_launch": by / n,
                          "gbs": by / sec / 1e9, "ms_per_step": sec / steps * 1e3}
            if fam == fams[4][1] and 8 <= wl.rank < 128:
                kern[name]["note"] = ("the Gram finish (k_wfact, k_chol) runs on the context's second "
                                      "stream beside the decompress: its events time that span, most of "
                                      "which the decompress hides")
    # the dominant kernel: the Q-step kernel, the longest-running single kernel of the step (one
    # launch per Q-step); at rank 4 the P-step time is split over one k_pfused launch per column
    # class
    dom = fams[1][0] if fams[1][0] in kern else max(kern, key=lambda k: kern[k]["ms_per_step"])
    dk = kern[dom]
    step_bytes, bp, bq, bd, nc, n1 = algorithmic_bytes(wl, wl.rank)
    traffic, traffic_src = measured_traffic(wl.name, dom)
    gbs = step_bytes / (ms * 1e-3) / 1e9
    roof = {"bound": "hbm", "achieved": round(dk["gbs"], 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(dk["gbs"] / HBM_PEAK_GBS, 4),
            "traffic": traffic,
            "traffic_source": traffic_src,
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
        "metric": metric_of(wl),
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
                   "kernels": {k: {kk: round(vv, 3) if isinstance(vv, float) else vv for kk, vv in v.items()}
                       for k, v in kern.items()}},
        "roofline": roof,
    }
    res["config"]["step_ms"] = {"mean": round(float(t_step.mean()), 4), "std": round(float(t_step.std()), 4),
                                "median": round(float(np.median(t_step)), 4),
                                "p_step_mean": round(float(t_step[0::2].mean()), 4),
                                "q_step_mean": round(float(t_step[1::2].mean()), 4)}
    res["config"]["mall_flushed"] = {"mean_ms": round(float(t_flush.mean()), 4),
                                     "gbs": round(step_bytes / (float(t_flush.mean()) * 1e-3) / 1e9, 2)}
    if args.mode == "graph":
        ms_eager = timed(steps, "all")
        res["config"]["ms_per_step_all_mode_uncaptured"] = round(ms_eager, 4)
        res["config"]["gbs_all_mode_uncaptured"] = round(step_bytes / (ms_eager * 1e-3) / 1e9, 2)
    if ms_other is not None:
        res["config"][f"ms_per_step_{other}_mode"] = round(ms_other, 4)
        res["config"][f"gbs_{other}_mode"] = round(step_bytes / (ms_other * 1e-3) / 1e9, 2)
    if args.compare_powersgd:
        res["config"]["powersgd"] = compare_powersgd(acp, wl, shapes, gsets, fbuf, out, dev, main, steps,
                                                     args.warmup, step_no)
    ceil = probe_ceilings(dev, main)
    ceil["pct_of_step_mix"] = round(100 * gbs / ceil["step_mix_gbs"], 2)
    res["config"]["ceilings"] = ceil
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(wl)
    res["cpu_baseline_host"] = host_info()
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
