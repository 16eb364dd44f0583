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
    """Outputs, the message the step wrote (its parity's length of each factor buffer) and E."""
    torch.cuda.synchronize()
    out = [o.clone() for o in run.out]
    fb = [f[:(i[2] if t % 2 else i[3])].clone() for f, i in zip(run.fbuf, run.info)]
    es = []
    for b in range(run.nb):
        run.acp.error(b, run.ebuf[b])
        es.append(run.ebuf[b].clone())
    return out, fb, es


def _same(a, b):
    return all(torch.equal(x, y) for xs, ys in zip(a, b) for x, y in zip(xs, ys))


def _resnet_inputs(run, wl, t):
    return run.pack(sg.gradient_set(wl, t))


WIDE_SHAPES = [(96, 80), (33, 5, 7), (40,), (70, 130), (17,), (64, 64), (200, 36)]
# rank-split kernels, Gram partials over several slices, the blocked Cholesky
SPLIT_SHAPES = [(300, 520), (40,), (2100, 300), (270, 1000)]


@pytest.mark.parametrize("case", ["resnet50_r4", "wide_r16_after_p", "wide_r32_after_q",
                                  "split_r128_after_p", "split_r256_after_q"])
def test_bitwise_repeatable_and_resume(case):
    """Repeat runs agree bitwise; resuming from a checkpoint continues bitwise.  The wide cases
    checkpoint a rank-16 context after a P-step (its arena holds X) and a rank-32 context after
    a Q-step (its arena holds F); the split cases do the same at ranks 128 and 256."""
    if case == "resnet50_r4":
        wl = sg.WORKLOADS["resnet50_r4"]
        shapes, rank, cap, at = [p.shape for p in wl.params], 4, 25 << 20, 3
    else:
        rank, at = {"wide_r16_after_p": (16, 3), "wide_r32_after_q": (32, 4),
                    "split_r128_after_p": (128, 3), "split_r256_after_q": (256, 4)}[case]
        shapes, cap = (WIDE_SHAPES, 1 << 15) if case.startswith("wide") else (SPLIT_SHAPES, 1 << 20)
        wl = sg.Workload(case, [sg.Param(f"t{i}", s) for i, s in enumerate(shapes)], rank, 8,
                         lambda p: 0.05, seed=11)
    inputs = {}

    def inp(run, t):
        if t not in inputs:
            inputs[t] = run.pack(sg.gradient_set(wl, t))
        return inputs[t]

    a = PU.Runner(shapes, rank, cap=cap)
    snaps_a = []
    for t in range(1, 7):
        a.step(t, inp(a, t))
        snaps_a.append(_snap(a, t))
        if t == at:
            ckpt = a.acp.get_state()
    b = PU.Runner(shapes, rank, cap=cap)
    for t in range(1, 7):
        b.step(t, inp(b, t))
        assert _same(_snap(b, t), snaps_a[t - 1]), f"run-to-run difference at step {t}"
    c = PU.Runner(shapes, rank, cap=cap)
    c.acp.set_state(ckpt)
    for t in range(at + 1, 7):
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


@pytest.mark.parametrize("name", ["bert_large_r4", "bert_large_r32", "bert_large_r64", "bert_large_r128",
                                  "bert_large_r256"])
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


def _grouped_vs_per_bucket(shapes, rank, grads_of, steps, cap=25 << 20):
    a = PU.Runner(shapes, rank, cap=cap)
    b = PU.Runner(shapes, rank, cap=cap)
    for t in range(1, steps + 1):
        gb = a.pack(grads_of(t))
        a.step(t, gb)
        b.acp.compress_all(t, gb, b.fbuf)
        b.acp.decompress_all(t, b.fbuf, b.out)
        assert _same(_snap(a, t), _snap(b, t)), f"grouped call differs at step {t}"
    return a.nb


@pytest.mark.parametrize("name", ["resnet50_r4", "bert_base_r4", "bert_base_r32"])
def test_grouped_calls_equal_per_bucket_calls(name):
    wl = sg.WORKLOADS[name]
    shapes = [p.shape for p in wl.params]
    _grouped_vs_per_bucket(shapes, wl.rank, lambda t: sg.gradient_set(wl, t), 4)


def test_grouped_calls_over_several_launch_groups():
    g = np.random.default_rng(7)
    shapes = [(int(g.integers(8, 200)), int(g.integers(8, 300))) if i % 3 else (int(g.integers(1, 500)),)
              for i in range(150)]
    params = [sg.Param(f"t{i}", s) for i, s in enumerate(shapes)]
    wl = sg.Workload("many", params, 4, 4, lambda p: 0.1, seed=5)
    nb = _grouped_vs_per_bucket(shapes, 4, lambda t: sg.gradient_set(wl, t), 4, cap=1 << 14)
    assert nb > 64


@pytest.mark.parametrize("rank", [16, 32, 64])
def test_mixed_calls_and_reload_in_place(rank):
    """From rank 8 to 64 a decompress also forms the next compress's orthogonal factor and the
    context records it: per-bucket and all-bucket calls in alternation, and a state load into the
    same context (which must drop the record while the slots hold the early factor), continue
    bitwise like plain per-bucket calls."""
    shapes = WIDE_SHAPES if rank < 64 else SPLIT_SHAPES
    cap = 1 << 15 if rank < 64 else 1 << 20
    wl = sg.Workload(f"mixed_r{rank}", [sg.Param(f"t{i}", s) for i, s in enumerate(shapes)], rank, 8,
                     lambda p: 0.05, seed=13)
    a = PU.Runner(shapes, rank, cap=cap)
    b = PU.Runner(shapes, rank, cap=cap)
    assert a.nb >= 2
    for t in range(1, 9):
        gb = a.pack(sg.gradient_set(wl, t))
        a.step(t, gb)
        if t % 2:  # all-bucket compress, per-bucket decompress
            b.acp.compress_all(t, gb, b.fbuf)
            for k in range(b.nb):
                b.acp.decompress(t, k, b.fbuf[k], b.out[k])
        else:      # per-bucket compress, all-bucket decompress
            for k in range(b.nb):
                b.acp.compress(t, k, gb[k], b.fbuf[k])
            b.acp.decompress_all(t, b.fbuf, b.out)
        assert _same(_snap(a, t), _snap(b, t)), f"mixed calls differ at step {t}"
        if t == 3:
            ckpt = b.acp.get_state()
        if t == 5:  # back to step 3 in the same context, then steps 4 and 5 again
            b.acp.set_state(ckpt)
            for u in (4, 5):
                gu = b.pack(sg.gradient_set(wl, u))
                b.step(u, gu)
            assert _same(_snap(a, t), _snap(b, t)), "reload in place differs at step 5"
    PU.log(f"  rank {rank}: mixed calls and an in-place reload bitwise equal to per-bucket calls")


def test_grouped_call_sequencing():
    from paper_2306_08881_amd import _lib as L
    shapes = [(32, 24), (24,), (40, 16)]
    run = PU.Runner(shapes, 4, cap=1 << 10)
    assert run.nb >= 2
    gb = run.pack({i: np.ones(s, np.float32) for i, s in enumerate(shapes)})
    run.acp.compress(1, 0, gb[0], run.fbuf[0])          # bucket 0 ahead of the others
    with pytest.raises(L.AcpError) as e:
        run.acp.compress_all(1, gb, run.fbuf)
    assert e.value.status == L.ACP_E_STEP
    run.acp.decompress(1, 0, run.fbuf[0], run.out[0])
    for b in range(1, run.nb):
        run.acp.compress(1, b, gb[b], run.fbuf[b])
        run.acp.decompress(1, b, run.fbuf[b], run.out[b])
    run.acp.compress_all(2, gb, run.fbuf)
    with pytest.raises(L.AcpError) as e:
        run.acp.compress_all(3, gb, run.fbuf)
    assert e.value.status == L.ACP_E_STEP
    run.acp.decompress_all(2, run.fbuf, run.out)
