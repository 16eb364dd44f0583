"""GPU parity of the no-reuse ablation and of Power-SGD against the fp64 oracle.

* No reuse (Section V-B): ACP-SGD whose reused factor is drawn anew every step on the device
  from the step-keyed counter-based generator; compared with ``AcpOracle(reuse=False)``.
* Power-SGD with error feedback (Algorithm 1, left): the three calls per step through the C ABI,
  per bucket and all-bucket, compared with ``PowerSgdOracle``: the P message, the Q message, the
  orthonormal P, the kept Q, M_hat and E per layer (relative Frobenius <= 1e-4), raw vectors
  bit-exact.  Steps 1-4 run free; later steps re-sync the oracle from the device's Q and E (the
  subspace iteration compounds fp32 rounding the way ACP-SGD's does).
"""

from __future__ import annotations

from typing import Dict, List, Sequence

import numpy as np
import pytest
import torch

import synthgrad as sg
from oracle.acp import AcpOracle, PowerSgdOracle
from paper_2306_08881_amd.acp import Acp
from tests import parity_util as PU
from tests.test_gpu_parity import RAGGED, RANK256, _assert_ok

pytestmark = pytest.mark.gpu

TOL = PU.TOL


def _require_gpu():
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible")


# ------------------------------------------------------------------------------ no reuse

def _custom_workload(shapes, rank, steps, seed=3):
    params = [sg.Param(f"t{i}", tuple(s)) for i, s in enumerate(shapes)]
    return sg.Workload("custom", params, rank, steps, lambda p: 0.05, seed=seed, cap_bytes=1 << 16)


@pytest.mark.parametrize("rank", [1, 4, 8, 32, 64, 128])
@pytest.mark.parametrize("ef", [True, False])
def test_no_reuse_ragged(rank, ef):
    """Every tensor at every step; the fresh factor is drawn on the device."""
    _require_gpu()
    wl = _custom_workload(RAGGED, rank, 8)
    rep = PU.run_parity(wl, "fresh", 8, range(1, 9), list(range(len(RAGGED))), ef=ef, free=4, reuse=False)
    _assert_ok(rep)


def test_no_reuse_rank256():
    _require_gpu()
    wl = _custom_workload(RANK256, 256, 4)
    rep = PU.run_parity(wl, "fresh", 4, range(1, 5), list(range(len(RANK256))), free=2, reuse=False)
    _assert_ok(rep)


@pytest.mark.parametrize("name", ["bert_large_r4", "bert_large_r32"])
def test_no_reuse_bert_large_grouped(name):
    """Sampled BERT-large tensors through the all-bucket calls, four free-running steps."""
    _require_gpu()
    wl = sg.WORKLOADS[name]
    names = ["embeddings.word_embeddings.weight", "embeddings.LayerNorm.weight",
             "encoder.layer.0.attention.self.query.weight", "encoder.layer.11.intermediate.dense.weight",
             "encoder.layer.23.output.dense.weight", "encoder.layer.23.output.dense.bias"]
    rep = PU.run_parity(wl, "fresh", 4, (1, 2, 3, 4), PU.tids_by_name(wl, names), grouped=True, reuse=False)
    _assert_ok(rep)


# ------------------------------------------------------------------------------ Power-SGD

class PsgdRunner:
    """One Power-SGD library context and the device buffers of every bucket."""

    def __init__(self, shapes, rank, seed=0, cap=25 << 20, world=1, ef=True, grouped=False):
        self.dev = torch.device("cuda:0")
        self.acp = Acp(shapes, rank, seed=seed, cap_bytes=cap, world_size=world, ef=ef, device=self.dev,
                       powersgd=True)
        self.grouped, self.rank, self.ef = grouped, rank, ef
        self.shapes = [tuple(s) for s in shapes]
        self.nb = self.acp.num_buckets()
        self.info = [self.acp.bucket_info(b) for b in range(self.nb)]
        self.lay = [self.acp.layout(b) for b in range(self.nb)]
        self.where = {}
        for b in range(self.nb):
            tids, go, fp, fq, comp = self.lay[b]
            for k, tid in enumerate(tids):
                self.where[int(tid)] = (b, int(go[k]), int(fp[k]), int(fq[k]), bool(comp[k]))
        z = lambda n: torch.zeros(max(n, 4), dtype=torch.float32, device=self.dev)
        self.pbuf = [z(i[2]) for i in self.info]
        self.qbuf = [z(i[3]) for i in self.info]
        self.out = [z(i[1]) for i in self.info]
        self.ebuf = [z(i[1]) for i in self.info]

    def pack(self, grads):
        return PU.Runner.pack(self, grads)

    def step(self, t, gbufs, allreduce=None):
        """One step; ``allreduce(list_of_buffers)`` replaces each half's buffers by their sums
        (identity at world size 1)."""
        if self.grouped:
            self.acp.powersgd_p_all(t, gbufs, self.pbuf)
            if allreduce:
                allreduce(self.pbuf)
            self.acp.powersgd_q_all(t, gbufs, self.pbuf, self.qbuf)
            if allreduce:
                allreduce(self.qbuf)
            self.acp.powersgd_decompress_all(t, self.qbuf, self.out)
            return
        for b in range(self.nb):
            self.acp.powersgd_p(t, b, gbufs[b], self.pbuf[b])
        if allreduce:
            allreduce(self.pbuf)
        for b in range(self.nb):
            self.acp.powersgd_q(t, b, gbufs[b], self.pbuf[b], self.qbuf[b])
        if allreduce:
            allreduce(self.qbuf)
        for b in range(self.nb):
            self.acp.powersgd_decompress(t, b, self.qbuf[b], self.out[b])

    def host(self):
        torch.cuda.synchronize()
        res = {"p": [x.cpu().numpy() for x in self.pbuf], "q": [x.cpu().numpy() for x in self.qbuf],
               "out": [x.cpu().numpy() for x in self.out], "e": []}
        for b in range(self.nb):
            if self.ef:
                self.acp.error(b, self.ebuf[b])
            res["e"].append(self.ebuf[b].cpu().numpy() if self.ef else None)
        return res

    def nm(self, tid):
        s = self.shapes[tid]
        return s[0], int(np.prod(s[1:]))

    def factor(self, tid, which):
        n, m = self.nm(tid)
        rows = n if which == "P" else m
        buf = torch.zeros(rows * self.rank, dtype=torch.float32, device=self.dev)
        self.acp.factor(tid, which, buf)
        return buf.cpu().numpy().reshape(rows, self.rank)


def _compare(run: PsgdRunner, orc: PowerSgdOracle, t: int, tids, host, msgs, outs, rep: PU.Report):
    for tid in tids:
        b, go, fp, fq, comp = run.where[tid]
        st = orc.state[tid]
        numel = int(np.prod(run.shapes[tid]))
        if comp:
            n, m = run.nm(tid)
            r = run.rank
            rep.add("P message", tid, t, PU.rel_err(host["p"][b][fp:fp + n * r], msgs[tid][0]))
            rep.add("Q message", tid, t, PU.rel_err(host["q"][b][fq:fq + m * r], msgs[tid][1]))
            rep.add("orthonormal P", tid, t, PU.rel_err(run.factor(tid, "P"), st.P))
            rep.add("kept Q", tid, t, PU.rel_err(run.factor(tid, "Q"), st.Q))
            rep.add("M_hat", tid, t, PU.rel_err(host["out"][b][go:go + numel], outs[tid]))
            if st.E is not None:
                rep.add("E", tid, t, PU.rel_err(host["e"][b][go:go + numel], st.E))
        else:
            rep.add("vector message", tid, t, float(np.abs(host["q"][b][fq:fq + numel] - msgs[tid][1]).max()), 0.0)
            rep.add("vector output", tid, t, float(np.abs(host["out"][b][go:go + numel] - outs[tid].reshape(-1)).max()), 0.0)


def _resync(run: PsgdRunner, orc: PowerSgdOracle, t_done: int, tids, host):
    for tid in tids:
        st = orc.state[tid]
        if st.plan.compressed:
            st.Q = run.factor(tid, "Q").astype(np.float64)
            if st.E is not None:
                b, go, *_ = run.where[tid]
                n, m = run.nm(tid)
                st.E = host["e"][b][go:go + n * m].astype(np.float64).reshape(n, m)
        st.step, st.phase = t_done, 0


def run_psgd_parity(wl: sg.Workload, steps: int, tids: Sequence[int], ef=True, free=4, grouped=False,
                    world=1) -> PU.Report:
    shapes = [p.shape for p in wl.params]
    run = PsgdRunner(shapes, wl.rank, wl.seed, wl.cap_bytes, world=world, ef=ef, grouped=grouped)
    orc = PowerSgdOracle(shapes, wl.rank, seed=wl.seed, cap_bytes=wl.cap_bytes, world_size=world, ef=ef,
                         tensor_ids=tids)
    rep = PU.Report()
    host = None
    for t in range(1, steps + 1):
        if t > free:
            _resync(run, orc, t - 1, tids, host)
        grads = sg.gradient_set(wl, t, tensor_ids=None, threads=16)
        run.step(t, run.pack(grads))
        msgs, outs = {}, {}
        for tid in tids:
            ep = orc.compress_p_tensor(t, tid, grads[tid])
            eq = orc.compress_q_tensor(t, tid, ep)
            msgs[tid] = (ep, eq)
            outs[tid] = orc.decompress_tensor(t, tid, eq)
        host = run.host()
        _compare(run, orc, t, tids, host, msgs, outs, rep)
        PU.log(f"  power-sgd {wl.name} r={wl.rank} t={t}{' (re-synced)' if t > free else ''}: " +
               ", ".join(f"{k} {v:.2e}" for k, v in rep.worst.items()))
    run.acp.close()
    return rep


@pytest.mark.parametrize("rank", [1, 2, 4, 8, 32, 64, 128])
@pytest.mark.parametrize("ef", [True, False])
def test_powersgd_ragged(rank, ef):
    _require_gpu()
    wl = _custom_workload(RAGGED, rank, 8)
    _assert_ok(run_psgd_parity(wl, 8, list(range(len(RAGGED))), ef=ef))


def test_powersgd_rank256():
    _require_gpu()
    wl = _custom_workload(RANK256, 256, 4)
    _assert_ok(run_psgd_parity(wl, 4, list(range(len(RANK256))), free=2))


@pytest.mark.parametrize("name", ["bert_large_r4", "bert_large_r32"])
def test_powersgd_bert_large_every_tensor(name):
    """Every BERT-large tensor at steps 1-3 through the all-bucket calls (the benchmark's)."""
    _require_gpu()
    wl = sg.WORKLOADS[name]
    _assert_ok(run_psgd_parity(wl, 3, list(range(len(wl.params))), grouped=True))


@pytest.mark.parametrize("rank", [4, 32])
def test_powersgd_grouped_equals_per_bucket(rank):
    """The all-bucket calls give bitwise the per-bucket calls' results."""
    _require_gpu()
    wl = _custom_workload(RAGGED + [(700, 640), (96,)], rank, 4)
    shapes = [p.shape for p in wl.params]
    a = PsgdRunner(shapes, rank, wl.seed, wl.cap_bytes)
    g = PsgdRunner(shapes, rank, wl.seed, wl.cap_bytes, grouped=True)
    assert a.nb > 2
    for t in range(1, 5):
        bufs = a.pack(sg.gradient_set(wl, t))
        a.step(t, bufs)
        g.step(t, bufs)
        ha, hg = a.host(), g.host()
        for k in ha:
            for x, y in zip(ha[k], hg[k]):
                assert np.array_equal(x, y), (t, k)


def test_powersgd_three_workers_loopback():
    """p = 3 workers on one GPU, the all-reduces are sums of their buffers."""
    _require_gpu()
    shapes = [(96, 80), (80,), (64, 3, 3, 3)]
    k, r = 3, 4
    runs = [PsgdRunner(shapes, r, world=k) for _ in range(k)]
    orcs = [PowerSgdOracle(shapes, r, world_size=k) for _ in range(k)]
    rng = np.random.default_rng(2)
    for t in range(1, 7):
        grads = [{i: rng.standard_normal(s).astype(np.float32) for i, s in enumerate(shapes)} for _ in range(k)]
        bufs = [ru.pack(gr) for ru, gr in zip(runs, grads)]
        for ru, bb in zip(runs, bufs):
            ru.acp.powersgd_p(t, 0, bb[0], ru.pbuf[0])
        psum = sum(ru.pbuf[0] for ru in runs)
        for ru, bb in zip(runs, bufs):
            ru.acp.powersgd_q(t, 0, bb[0], psum, ru.qbuf[0])
        qsum = sum(ru.qbuf[0] for ru in runs)
        for ru in runs:
            ru.acp.powersgd_decompress(t, 0, qsum, ru.out[0])
        for tid in range(len(shapes)):
            p_agg = sum(o.compress_p_tensor(t, tid, gr[tid]) for o, gr in zip(orcs, grads))
            q_agg = sum(o.compress_q_tensor(t, tid, p_agg) for o in orcs)
            outs = [o.decompress_tensor(t, tid, q_agg) for o in orcs]
            for w, ru in enumerate(runs):
                h = ru.host()
                b, go, *_ = ru.where[tid]
                numel = int(np.prod(shapes[tid]))
                assert PU.rel_err(h["out"][b][go:go + numel], outs[w]) <= TOL, (t, tid, w)
                if orcs[w].error(tid) is not None:
                    assert PU.rel_err(h["e"][b][go:go + numel], orcs[w].error(tid)) <= TOL, (t, tid, w)
        for tid in (0, 2):  # every worker keeps bitwise the same Q
            q0 = runs[0].factor(tid, "Q")
            for ru in runs[1:]:
                assert np.array_equal(ru.factor(tid, "Q"), q0)


def test_powersgd_sequencing():
    _require_gpu()
    from paper_2306_08881_amd import _lib as L
    ru = PsgdRunner([(32, 24)], 4)
    g = ru.pack({0: np.ones((32, 24), np.float32)})
    with pytest.raises(L.AcpError) as e:
        ru.acp.powersgd_q(1, 0, g[0], ru.pbuf[0], ru.qbuf[0])
    assert e.value.status == L.ACP_E_STEP
    ru.acp.powersgd_p(1, 0, g[0], ru.pbuf[0])
    with pytest.raises(L.AcpError) as e:
        ru.acp.error(0, ru.ebuf[0])                      # the arena holds M + E between the halves
    assert e.value.status == L.ACP_E_STEP
    with pytest.raises(L.AcpError) as e:
        ru.acp.powersgd_decompress(1, 0, ru.qbuf[0], ru.out[0])
    assert e.value.status == L.ACP_E_STEP
    with pytest.raises(L.AcpError) as e:
        ru.acp.compress(1, 0, g[0], ru.pbuf[0])          # an ACP-SGD call on a Power-SGD context
    assert e.value.status == L.ACP_E_UNSUPPORTED
    ru.acp.powersgd_q(1, 0, g[0], ru.pbuf[0], ru.qbuf[0])
    ru.acp.powersgd_decompress(1, 0, ru.qbuf[0], ru.out[0])
    ru.acp.powersgd_p(2, 0, g[0], ru.pbuf[0])
