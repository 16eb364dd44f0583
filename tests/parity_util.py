"""Shared driver of the GPU parity tests: run the library (through the C ABI binding) and the
oracle on the same seeded inputs and compare per layer.

Inputs: gradient of tensor l at step t is ``synthgrad.gradient(wl, l, key(t))``.  ``mode``:
* "fresh": key(t) = t (a new gradient every step);
* "fixed": key(t) = 1 (the same gradient every step);
* "pool3": key(t) = (t - 1) % 3 + 1 (three gradient sets in turn; keeps the large models'
  input generation to three sets).
"""

from __future__ import annotations

import sys
import time
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence

import numpy as np
import torch

import synthgrad as sg
from oracle.acp import AcpOracle
from paper_2306_08881_amd.acp import Acp

TOL = 1e-4   # relative Frobenius error per layer and quantity


def key_of(mode: str, t: int) -> int:
    if mode == "fresh":
        return t
    if mode == "fixed":
        return 1
    if mode == "pool3":
        return (t - 1) % 3 + 1
    raise ValueError(mode)


def rel_err(x: np.ndarray, ref: np.ndarray) -> float:
    x = np.asarray(x, dtype=np.float64).reshape(-1)
    ref = np.asarray(ref, dtype=np.float64).reshape(-1)
    num = np.linalg.norm(x - ref)
    den = np.linalg.norm(ref)
    return num / den if den > 0 else num


def log(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def tids_by_name(wl: sg.Workload, names: Sequence[str]) -> List[int]:
    idx = {p.name: i for i, p in enumerate(wl.params)}
    return [idx[n] for n in names]


@dataclass
class Report:
    worst: Dict[str, float] = field(default_factory=dict)
    failures: List[str] = field(default_factory=list)

    def add(self, what: str, tid: int, t: int, err: float, tol: float = TOL):
        k = what
        self.worst[k] = max(self.worst.get(k, 0.0), err)
        if not err <= tol:
            self.failures.append(f"t={t} tensor {tid} {what}: rel err {err:.3e} > {tol:g}")


class Runner:
    """One library context plus the device buffers of every bucket."""

    def __init__(self, shapes, rank, seed=0, cap=25 << 20, world=1, ef=True, device="cuda:0",
                 grouped=False, reuse=True):
        self.dev = torch.device(device)
        self.grouped = grouped  # step() through acp_compress_all / acp_decompress_all
        self.acp = Acp(shapes, rank, seed=seed, cap_bytes=cap, world_size=world, ef=ef, device=self.dev,
                       reuse=reuse)
        self.nb = self.acp.num_buckets()
        self.info = [self.acp.bucket_info(b) for b in range(self.nb)]
        self.lay = [self.acp.layout(b) for b in range(self.nb)]
        self.where = {}
        for b in range(self.nb):
            tids, go, fp, fq, comp = self.lay[b]
            for k, tid in enumerate(tids):
                self.where[int(tid)] = (b, int(go[k]), int(fp[k]), int(fq[k]), bool(comp[k]))
        self.shapes = [tuple(s) for s in shapes]
        self.rank = rank
        nf = [max(i[2], i[3]) for i in self.info]
        self.fbuf = [torch.zeros(max(n, 4), dtype=torch.float32, device=self.dev) for n in nf]
        self.out = [torch.zeros(i[1], dtype=torch.float32, device=self.dev) for i in self.info]
        self.ebuf = [torch.zeros(i[1], dtype=torch.float32, device=self.dev) for i in self.info]

    def pack(self, grads: Dict[int, np.ndarray]) -> List[torch.Tensor]:
        """Device gradient buckets from per-tensor host arrays."""
        bufs = []
        for b in range(self.nb):
            host = np.empty(self.info[b][1], dtype=np.float32)
            tids, go, *_ = self.lay[b]
            for k, tid in enumerate(tids):
                g = grads[int(tid)].reshape(-1)
                host[go[k]:go[k] + g.size] = g
            bufs.append(torch.from_numpy(host).to(self.dev))
        return bufs

    def step(self, t: int, gbufs: Sequence[torch.Tensor], buckets: Optional[Sequence[int]] = None):
        if self.grouped and buckets is None:  # the launch configuration bench.py times
            self.acp.compress_all(t, gbufs, self.fbuf)
            self.acp.decompress_all(t, self.fbuf, self.out)
            return
        for b in (range(self.nb) if buckets is None else buckets):
            self.acp.compress(t, b, gbufs[b], self.fbuf[b])
            self.acp.decompress(t, b, self.fbuf[b], self.out[b])

    def factor_slice(self, t: int, tid: int) -> np.ndarray:
        b, go, fp, fq, comp = self.where[tid]
        off = fp if t % 2 == 1 else fq
        shp = self.shapes[tid]
        n = shp[0]
        m = int(np.prod(shp[1:])) if len(shp) > 1 else 1
        size = (n if t % 2 == 1 else m) * self.rank if comp else int(np.prod(shp))
        return self.fbuf[b][off:off + size].cpu().numpy()

    def out_slice(self, tid: int) -> np.ndarray:
        b, go, *_ = self.where[tid]
        numel = int(np.prod(self.shapes[tid]))
        return self.out[b][go:go + numel].cpu().numpy()

    def error_slice(self, tid: int) -> np.ndarray:
        b, go, *_ = self.where[tid]
        self.acp.error(b, self.ebuf[b])
        numel = int(np.prod(self.shapes[tid]))
        return self.ebuf[b][go:go + numel].cpu().numpy()

    def ortho(self, t: int, tid: int) -> np.ndarray:
        shp = self.shapes[tid]
        n, m = shp[0], int(np.prod(shp[1:]))
        rows = m if t % 2 == 1 else n
        out = torch.zeros(rows * self.rank, dtype=torch.float32, device=self.dev)
        self.acp.factor(tid, "Q" if t % 2 == 1 else "P", out)
        return out.cpu().numpy()


def compare_step(run: Runner, orc: AcpOracle, t: int, tids: Sequence[int], emits: Dict[int, np.ndarray],
                 outs: Dict[int, np.ndarray], rep: Report, tol: float = TOL):
    torch.cuda.synchronize()
    for tid in tids:
        st = orc.state[tid]
        if st.plan.compressed:
            rep.add("emitted factor", tid, t, rel_err(run.factor_slice(t, tid), emits[tid]), tol)
            rep.add("orthonormal factor", tid, t, rel_err(run.ortho(t, tid), st.ortho), tol)
            rep.add("M_hat", tid, t, rel_err(run.out_slice(tid), outs[tid]), tol)
            if st.E is not None:
                rep.add("E", tid, t, rel_err(run.error_slice(tid), st.E), tol)
        else:
            # raw vectors: packed, summed over one worker and divided by 1 -> exact
            rep.add("vector message", tid, t, float(np.abs(run.factor_slice(t, tid) - emits[tid]).max()), 0.0)
            rep.add("vector output", tid, t, float(np.abs(run.out_slice(tid) - outs[tid].reshape(-1)).max()), 0.0)


def read_state_into(run: Runner, orc: AcpOracle, t_done: int, tids: Sequence[int]):
    """Give the oracle the device state after step ``t_done`` (reused factors and E)."""
    torch.cuda.synchronize()
    for tid in tids:
        st = orc.state[tid]
        if st.plan.compressed:
            n, m, r = st.plan.n, st.plan.m, run.rank
            for which, rows in (("P", n), ("Q", m)):
                buf = torch.zeros(rows * r, dtype=torch.float32, device=run.dev)
                run.acp.factor(tid, which, buf)
                val = buf.cpu().numpy().astype(np.float64).reshape(rows, r)
                if which == "P":
                    st.P = val
                else:
                    st.Q = val
            if st.E is not None:
                st.E = run.error_slice(tid).astype(np.float64).reshape(n, m)
        st.step, st.pending = t_done, None


def run_parity(wl: sg.Workload, mode: str, steps: int, check: Sequence[int], tids: Sequence[int],
               ef: bool = True, tol: float = TOL, free: Optional[int] = None,
               device="cuda:0", grouped: bool = False, reuse: bool = True) -> Report:
    """Parity over ``steps`` steps, comparing the sampled tensors at the ``check`` steps.

    Steps 1..``free`` run free: the oracle carries its own fp64 state from step 1.  At a
    checked step t > ``free`` the oracle is re-synced: it takes the device's reused factors and
    E after step t - 1 and computes step t from them, which checks that step's arithmetic.
    (Error feedback integrates every rounding difference, and with a fresh gradient each step
    any fp32 execution drifts away from an fp64 one exponentially with the step count, so
    free-running agreement is only meaningful over the first steps.)
    """
    free = steps if free is None else free
    shapes = [p.shape for p in wl.params]
    t0 = time.time()
    run = Runner(shapes, wl.rank, wl.seed, wl.cap_bytes, ef=ef, device=device, grouped=grouped, reuse=reuse)
    orc = AcpOracle(shapes, wl.rank, seed=wl.seed, cap_bytes=wl.cap_bytes, ef=ef, tensor_ids=tids,
                    reuse=reuse)
    rep = Report()
    cache: Dict[int, List[torch.Tensor]] = {}
    host_cache: Dict[int, Dict[int, np.ndarray]] = {}
    for t in range(1, steps + 1):
        key = key_of(mode, t)
        if key in cache:
            gbufs, grads = cache[key], host_cache[key]
        else:
            grads = sg.gradient_set(wl, key)
            gbufs = run.pack(grads)
            if mode != "fresh":
                cache[key] = gbufs
                host_cache[key] = {tid: grads[tid] for tid in tids}
        resync = t > free and t in check
        if resync:
            read_state_into(run, orc, t - 1, tids)
        run.step(t, gbufs)
        if t <= free or resync:
            emits, outs = {}, {}
            for tid in tids:
                emits[tid] = orc.compress_tensor(t, tid, grads[tid])
                outs[tid] = orc.decompress_tensor(t, tid, emits[tid])
            if t in check:
                compare_step(run, orc, t, tids, emits, outs, rep, tol)
                log(f"  {wl.name} t={t}{' (re-synced)' if resync else ''}: worst so far " +
                    ", ".join(f"{k} {v:.2e}" for k, v in rep.worst.items()) + f" ({time.time() - t0:.0f}s)")
        if mode == "fresh":
            del gbufs
    run.acp.close()
    return rep
