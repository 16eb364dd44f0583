"""Full-size GPU parity: every tensor of a workload against the fp64 oracle, and the drift of a few
tracked tensors over 100 free-running steps against an fp32 envelope.

All buckets run through the all-bucket calls (the launch configuration the benchmark times).
Schedule of a run of ``steps`` steps:

* t = 1 .. ``free_all`` (4): a fresh gradient set keyed t for every tensor.  The oracle runs every
  tensor free-running from step 1, and every tensor is compared at each of these steps.
* t in ``resync`` (50, 99, 100): a fresh gradient set keyed t.  The oracle restarts every tensor
  from the device's state after step t - 1 (its reused factors and E) and computes step t, and
  every tensor is compared: this checks the arithmetic of that step at every layer.
* the other steps take the resident sets of steps 1-4 in turn.
* tracked tensors take a fresh gradient keyed t at every step (written into their slots of the
  resident set).  A free-running fp64 oracle and a free-running fp32 re-implementation
  (``tests/fp32_ref.py``) run them for all steps.  Up to step ``free_check`` (10) the device must
  agree with the free-running oracle within the parity bar; at the ``drift`` steps (50, 99, 100)
  its distance from the free-running oracle must stay inside the envelope that the independent
  fp32 run gives on the same tensor and inputs: at most max(TOL, ENVELOPE x the fp32 run's).

Compared per compressed tensor: the emitted (local) factor, the orthonormal factor, M_hat and E,
each by relative Frobenius error <= TOL and by its largest element error <= MAXREL x the RMS of
the oracle's values (a few wrong elements of a large layer move the Frobenius error by little).
Raw vectors must be bit-exact.
"""

from __future__ import annotations

import time
from dataclasses import dataclass, field
from typing import Dict, List, Sequence

import numpy as np
import torch

import synthgrad as sg
from oracle.acp import AcpOracle
from tests import parity_util as PU
from tests.fp32_ref import Fp32Tensor

TOL = PU.TOL        # relative Frobenius error per layer and quantity
MAXREL = 1e-3       # largest element error over the RMS of the oracle's values
ENVELOPE = 10.0     # drift bar: the device may drift up to this many times the fp32 run's distance


def max_rel(x: np.ndarray, ref: np.ndarray) -> float:
    x = np.asarray(x, dtype=np.float64).reshape(-1)
    ref = np.asarray(ref, dtype=np.float64).reshape(-1)
    if ref.size == 0:
        return 0.0
    rms = np.linalg.norm(ref) / np.sqrt(ref.size)
    d = float(np.max(np.abs(x - ref)))
    return d / rms if rms > 0 else d


@dataclass
class FullReport:
    worst: Dict[str, float] = field(default_factory=dict)
    where: Dict[str, str] = field(default_factory=dict)
    failures: List[str] = field(default_factory=list)
    compared: int = 0

    def add(self, what: str, tid: int, t: int, err: float, tol: float):
        if err > self.worst.get(what, -1.0):
            self.worst[what] = err
            self.where[what] = f"t={t} tensor {tid}"
        if not err <= tol:
            self.failures.append(f"t={t} tensor {tid} {what}: {err:.3e} > {tol:g}")

    def summary(self) -> str:
        return ", ".join(f"{k} {v:.2e} ({self.where[k]})" for k, v in self.worst.items())


class Snapshot:
    """Host copies of the device results after a step: factor buffers, outputs, E and the
    factors of every compressed tensor, each read in one transfer per bucket."""

    def __init__(self, run: PU.Runner, t: int, tids: Sequence[int]):
        torch.cuda.synchronize()
        self.run, self.t = run, t
        self.fbuf = [f.cpu().numpy() for f in run.fbuf]
        self.out = [o.cpu().numpy() for o in run.out]
        self.e = []
        for b in range(run.nb):
            if run.acp.ef:
                run.acp.error(b, run.ebuf[b])
            self.e.append(run.ebuf[b].cpu().numpy() if run.acp.ef else None)
        # the factors P_t and Q_t of every compressed tensor: one device buffer, one transfer
        self.fac: Dict[int, Dict[str, np.ndarray]] = {}
        mats = [tid for tid in tids if run.where[tid][4]]
        sizes = []
        for tid in mats:
            n, m = self._nm(tid)
            sizes += [n * run.rank, m * run.rank]
        if mats:
            dev = torch.empty(int(sum(sizes)), dtype=torch.float32, device=run.dev)
            off = 0
            for tid in mats:
                n, m = self._nm(tid)
                for which, rows in (("P", n), ("Q", m)):
                    run.acp.factor(tid, which, dev[off:off + rows * run.rank])
                    off += rows * run.rank
            host = dev.cpu().numpy()
            off = 0
            for tid in mats:
                n, m = self._nm(tid)
                self.fac[tid] = {}
                for which, rows in (("P", n), ("Q", m)):
                    self.fac[tid][which] = host[off:off + rows * run.rank].reshape(rows, run.rank)
                    off += rows * run.rank

    def _nm(self, tid):
        shp = self.run.shapes[tid]
        return shp[0], int(np.prod(shp[1:]))

    def factor_msg(self, tid: int) -> np.ndarray:
        b, go, fp, fq, comp = self.run.where[tid]
        off = fp if self.t % 2 == 1 else fq
        n, m = self._nm(tid)
        size = (n if self.t % 2 == 1 else m) * self.run.rank if comp else int(np.prod(self.run.shapes[tid]))
        return self.fbuf[b][off:off + size]

    def out_of(self, tid: int) -> np.ndarray:
        b, go, *_ = self.run.where[tid]
        return self.out[b][go:go + int(np.prod(self.run.shapes[tid]))]

    def e_of(self, tid: int) -> np.ndarray:
        b, go, *_ = self.run.where[tid]
        return self.e[b][go:go + int(np.prod(self.run.shapes[tid]))]

    def ortho_of(self, tid: int) -> np.ndarray:
        return self.fac[tid]["Q" if self.t % 2 == 1 else "P"]


def compare_all(snap: Snapshot, orc: AcpOracle, t: int, tids: Sequence[int], emits, outs,
                rep: FullReport):
    for tid in tids:
        st = orc.state[tid]
        if st.plan.compressed:
            pairs = [("emitted factor", snap.factor_msg(tid), emits[tid]),
                     ("orthonormal factor", snap.ortho_of(tid), st.ortho),
                     ("M_hat", snap.out_of(tid), outs[tid])]
            if st.E is not None:
                pairs.append(("E", snap.e_of(tid), st.E))
            for what, x, ref in pairs:
                rep.add(what, tid, t, PU.rel_err(x, ref), TOL)
                rep.add(what + " max element", tid, t, max_rel(x, ref), MAXREL)
        else:
            rep.add("vector message", tid, t, float(np.abs(snap.factor_msg(tid) - emits[tid]).max()), 0.0)
            rep.add("vector output", tid, t, float(np.abs(snap.out_of(tid) - outs[tid].reshape(-1)).max()), 0.0)
        rep.compared += 1


def oracle_from_device(run: PU.Runner, wl: sg.Workload, snap: Snapshot, t_done: int,
                       tids: Sequence[int], ef: bool) -> AcpOracle:
    """A fresh oracle over ``tids`` holding the device's state after step ``t_done``."""
    shapes = [p.shape for p in wl.params]
    orc = AcpOracle(shapes, wl.rank, seed=wl.seed, cap_bytes=wl.cap_bytes, ef=ef, tensor_ids=tids)
    for tid in tids:
        st = orc.state[tid]
        if st.plan.compressed:
            st.P = snap.fac[tid]["P"].astype(np.float64)
            st.Q = snap.fac[tid]["Q"].astype(np.float64)
            if st.E is not None:
                st.E = snap.e_of(tid).astype(np.float64).reshape(st.plan.n, st.plan.m)
        st.step, st.pending = t_done, None
    return orc


def oracle_step(orc: AcpOracle, t: int, tids: Sequence[int], grads):
    emits, outs = {}, {}
    for tid in tids:
        emits[tid] = orc.compress_tensor(t, tid, grads[tid])
        outs[tid] = orc.decompress_tensor(t, tid, emits[tid])
    return emits, outs


def run_full_parity(wl: sg.Workload, tracked: Sequence[str], steps: int = 100, free_all: int = 4,
                    resync: Sequence[int] = (50, 99, 100), free_check: int = 10,
                    drift: Sequence[int] = (50, 99, 100), ef: bool = True, threads: int = 16):
    """Returns (report of the all-tensor comparisons, drift rows: (t, tensor, quantity, device
    distance, fp32 distance))."""
    t0 = time.time()
    shapes = [p.shape for p in wl.params]
    all_tids = list(range(len(shapes)))
    trk = PU.tids_by_name(wl, tracked)
    run = PU.Runner(shapes, wl.rank, wl.seed, wl.cap_bytes, ef=ef, grouped=True)
    orc_all = AcpOracle(shapes, wl.rank, seed=wl.seed, cap_bytes=wl.cap_bytes, ef=ef)
    orc_trk = AcpOracle(shapes, wl.rank, seed=wl.seed, cap_bytes=wl.cap_bytes, ef=ef, tensor_ids=trk)
    f32 = {tid: Fp32Tensor(wl.seed, tid, orc_trk.state[tid].plan.n, orc_trk.state[tid].plan.m, wl.rank)
           for tid in trk if orc_trk.state[tid].plan.compressed}
    rep = FullReport()
    drift_rows = []
    resident: List[List[torch.Tensor]] = []
    for t in range(1, steps + 1):
        fresh = t <= free_all or t in resync
        if fresh:
            grads = sg.gradient_set(wl, t, threads=threads)
            gbufs = run.pack(grads)
            if t <= free_all:
                resident.append(gbufs)
        else:
            gbufs = resident[(t - 1) % len(resident)]
        # tracked tensors: a fresh gradient keyed t at every step
        g_trk = {tid: sg.gradient(wl, tid, t) for tid in trk}
        if not fresh:
            for tid in trk:
                b, go, *_ = run.where[tid]
                g = torch.from_numpy(g_trk[tid].reshape(-1).copy()).to(run.dev)
                gbufs[b][go:go + g.numel()].copy_(g)
        snap_prev = None
        if t in resync and t > free_all:
            snap_prev = Snapshot(run, t - 1, all_tids)
        run.step(t, gbufs)
        # the tracked tensors' free-running fp64 oracle and fp32 re-implementation
        e_trk, o_trk = oracle_step(orc_trk, t, trk, g_trk)
        o32 = {tid: f.step(t, g_trk[tid]) for tid, f in f32.items()}
        if t <= free_all:
            emits, outs = oracle_step(orc_all, t, all_tids, grads)
            compare_all(Snapshot(run, t, all_tids), orc_all, t, all_tids, emits, outs, rep)
            PU.log(f"  {wl.name} t={t} all {len(all_tids)} tensors (free-running): {rep.summary()} "
                   f"({time.time() - t0:.0f}s)")
            if t == free_all:
                del orc_all
        elif t in resync:
            orc_rs = oracle_from_device(run, wl, snap_prev, t - 1, all_tids, ef)
            del snap_prev
            emits, outs = oracle_step(orc_rs, t, all_tids, grads)
            compare_all(Snapshot(run, t, all_tids), orc_rs, t, all_tids, emits, outs, rep)
            del orc_rs
            PU.log(f"  {wl.name} t={t} all {len(all_tids)} tensors (re-synced): {rep.summary()} "
                   f"({time.time() - t0:.0f}s)")
        if t == free_check or t in drift:
            snap = Snapshot(run, t, trk)
            if t == free_check:
                compare_all(snap, orc_trk, t, trk, e_trk, o_trk, rep)
                PU.log(f"  {wl.name} t={t} tracked tensors (free-running): {rep.summary()}")
            if t in drift:
                for tid, f in f32.items():
                    st = orc_trk.state[tid]
                    d_out = PU.rel_err(snap.out_of(tid), o_trk[tid])
                    f_out = PU.rel_err(o32[tid], o_trk[tid])
                    d_e = PU.rel_err(snap.e_of(tid), st.E) if st.E is not None else 0.0
                    f_e = PU.rel_err(f.E, st.E) if st.E is not None else 0.0
                    drift_rows.append((t, tid, "M_hat", d_out, f_out))
                    drift_rows.append((t, tid, "E", d_e, f_e))
                    PU.log(f"  {wl.name} t={t} tensor {tid} {wl.params[tid].name}: free-running distance "
                           f"from fp64, device / fp32 re-implementation: M_hat {d_out:.2e} / {f_out:.2e}, "
                           f"E {d_e:.2e} / {f_e:.2e}")
        if fresh and t > free_all:
            del gbufs
        if fresh:
            del grads
    run.acp.close()
    PU.log(f"  {wl.name}: {rep.compared} tensor comparisons, worst {rep.summary()} ({time.time() - t0:.0f}s)")
    return rep, drift_rows


def drift_failures(rows) -> List[str]:
    out = []
    for t, tid, what, dev, f32 in rows:
        bar = max(TOL, ENVELOPE * f32)
        if not dev <= bar:
            out.append(f"t={t} tensor {tid} {what}: device drift {dev:.3e} > max({TOL:g}, "
                       f"{ENVELOPE:g} x fp32 drift {f32:.3e})")
    return out
