"""GPU determinism, checkpoint/resume and full-size invariants (no oracle needed).

* two runs from the same seed and inputs are bitwise identical (the reductions are
  deterministic, which a data-parallel job needs so that all ranks keep the same factor);
* exporting the state at step k and importing it into a fresh context continues bitwise
  like the uninterrupted run;
* at the full BERT-large size, every element obeys E_t + M_hat_t = M_t + E_{t-1} (p = 1) and
  every orthonormal factor has Q^T Q = I on its kept columns.
"""

import numpy as np
import pytest
import torch

import synthgrad as sg
from tests import parity_util as PU

pytestmark = pytest.mark.gpu


def _snap(run, t):
    torch.cuda.synchronize()
    out = [o.clone() for o in run.out]
    fb = [f.clone() for f in run.fbuf]
    es = []
    for b in range(run.nb):
        run.acp.error(b, run.ebuf[b])
        es.append(run.ebuf[b].clone())
    return out, fb, es


def _same(a, b):
    return all(torch.equal(x, y) for xs, ys in zip(a, b) for x, y in zip(xs, ys))


def _resnet_inputs(run, wl, t):
    return run.pack(sg.gradient_set(wl, t))


def test_bitwise_repeatable_and_resume():
    wl = sg.WORKLOADS["resnet50_r4"]
    shapes = [p.shape for p in wl.params]
    inputs = {}

    def inp(run, t):
        if t not in inputs:
            inputs[t] = run.pack(sg.gradient_set(wl, t))
        return inputs[t]

    a = PU.Runner(shapes, 4)
    snaps_a = []
    for t in range(1, 7):
        a.step(t, inp(a, t))
        snaps_a.append(_snap(a, t))
        if t == 3:
            ckpt = a.acp.get_state()
    b = PU.Runner(shapes, 4)
    for t in range(1, 7):
        b.step(t, inp(b, t))
        assert _same(_snap(b, t), snaps_a[t - 1]), f"run-to-run difference at step {t}"
    c = PU.Runner(shapes, 4)
    c.acp.set_state(ckpt)
    for t in range(4, 7):
        c.step(t, inp(c, t))
        assert _same(_snap(c, t), snaps_a[t - 1]), f"resume difference at step {t}"


def test_checkpoint_rejects_other_context():
    from paper_2306_08881_amd import _lib as L
    a = PU.Runner([(32, 24)], 4)
    ckpt = a.acp.get_state()
    b = PU.Runner([(32, 24)], 8)
    with pytest.raises(L.AcpError) as e:
        b.acp.set_state(ckpt)
    assert e.value.status == L.ACP_E_STATE


@pytest.mark.parametrize("name", ["bert_large_r4"])
def test_full_size_residual_identity(name):
    wl = sg.WORKLOADS[name]
    shapes = [p.shape for p in wl.params]
    run = PU.Runner(shapes, wl.rank)
    e_prev = [torch.zeros_like(o) for o in run.out]
    worst = 0.0
    for t in range(1, 5):
        gb = run.pack(sg.gradient_set(wl, t))
        run.step(t, gb)
        torch.cuda.synchronize()
        for b in range(run.nb):
            run.acp.error(b, run.ebuf[b])
            tids, go, fp, fq, comp = run.lay[b]
            lhs = run.ebuf[b].double() + run.out[b].double()
            rhs = gb[b].double() + e_prev[b].double()
            for k, tid in enumerate(tids):
                if not comp[k]:
                    continue
                n = int(np.prod(shapes[tid]))
                sl = slice(int(go[k]), int(go[k]) + n)
                err = (torch.linalg.norm(lhs[sl] - rhs[sl]) / torch.linalg.norm(rhs[sl])).item()
                worst = max(worst, err)
                assert err <= 1e-5, (t, tid, err)
            e_prev[b] = run.ebuf[b].clone()
        # orthonormal factors of every matrix
        for tid, s in enumerate(shapes):
            if len(s) < 2:
                continue
            rows = int(np.prod(s[1:])) if t % 2 == 1 else s[0]
            f = torch.zeros(rows * wl.rank, device=run.dev)
            run.acp.factor(tid, "Q" if t % 2 == 1 else "P", f)
            F = f.view(rows, wl.rank).double()
            g = F.T @ F
            assert torch.allclose(g, torch.eye(wl.rank, dtype=torch.float64, device=run.dev), atol=1e-5), (t, tid)
    PU.log(f"  full-size residual identity worst {worst:.2e}")
