"""GPU parity of libacp.so against the fp64 oracle (per layer, relative Frobenius <= 1e-4).

Compared per layer: the emitted (local) factor, the orthonormal factor, M_hat and E; raw vectors
must be bit-exact.  Small cases compare every tensor at every step.  The five full-size workloads
(ResNet-50, ResNet-152, BERT-base r = 4 and 32, BERT-large r = 4 and 32) run all buckets through
the all-bucket calls, as the benchmark does, and compare every tensor at steps 1-4 (free-running)
and 50, 99, 100 (re-synced), plus tracked tensors free-running over all 100 steps against an fp32
drift envelope (tests/full_parity.py).  The rank sweep (r = 64, 128, 256) compares sampled tensors
at steps 1, 2, 3, 4, 10 (free-running), 50, 99 and 100 (re-synced).
"""

import numpy as np
import pytest
import torch

import synthgrad as sg
from oracle.acp import AcpOracle, LoopbackOracle
from tests import full_parity as FP
from tests import parity_util as PU

pytestmark = pytest.mark.gpu

CHECK = (1, 2, 3, 4, 10, 50, 99, 100)
FREE = 10


def _require_gpu():
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible")


def _assert_ok(rep):
    PU.log("  worst: " + ", ".join(f"{k} {v:.2e}" for k, v in rep.worst.items()))
    assert not rep.failures, "\n".join(rep.failures[:20])


@pytest.mark.parametrize("mode", ["fresh", "fixed"])
def test_single_conv_every_step(mode):
    _require_gpu()
    wl = sg.WORKLOADS["conv256x576_r4"]
    rep = PU.run_parity(wl, mode, wl.steps, range(1, wl.steps + 1), [0])
    _assert_ok(rep)


# tensors tracked over all 100 steps (fresh gradient every step, free-running fp64 oracle and
# fp32 re-implementation beside the device): ResNets
RESNET_TRACKED = ["layer1.0.conv1.weight", "layer1.0.conv2.weight", "layer3.2.conv3.weight",
                  "layer4.2.conv2.weight", "fc.weight", "fc.bias"]
RESNET152_TRACKED = ["layer2.7.conv2.weight", "layer3.35.conv3.weight", "layer4.0.downsample.0.weight",
                     "fc.weight", "layer3.20.bn2.bias"]
BERT_TRACKED = ["embeddings.position_embeddings.weight", "encoder.layer.0.attention.self.query.weight",
                "encoder.layer.0.attention.self.query.bias", "encoder.layer.5.intermediate.dense.weight",
                "encoder.layer.5.output.dense.weight"]


def _assert_full(rep, drift_rows):
    PU.log("  worst: " + rep.summary())
    bad = rep.failures + FP.drift_failures(drift_rows)
    assert not bad, "\n".join(bad[:20])


@pytest.mark.parametrize("name,tracked", [("resnet50_r4", RESNET_TRACKED), ("resnet152_r4", RESNET152_TRACKED),
                                          ("bert_base_r4", BERT_TRACKED), ("bert_base_r32", BERT_TRACKED),
                                          ("bert_large_r4", BERT_TRACKED), ("bert_large_r32", BERT_TRACKED)])
def test_every_tensor_100_steps(name, tracked):
    """Every tensor compared with the oracle at t = 1-4 (free-running, fresh gradients) and at
    t = 50, 99, 100 (re-synced, fresh gradients); tracked tensors free-running for 100 steps."""
    _require_gpu()
    rep, drift_rows = FP.run_full_parity(sg.WORKLOADS[name], tracked)
    _assert_full(rep, drift_rows)


BERT_SAMPLE = ["embeddings.word_embeddings.weight", "embeddings.position_embeddings.weight",
               "embeddings.LayerNorm.weight", "encoder.layer.0.attention.self.query.weight",
               "encoder.layer.0.attention.self.query.bias", "encoder.layer.5.intermediate.dense.weight",
               "encoder.layer.5.output.dense.weight", "encoder.layer.11.attention.output.dense.weight",
               "encoder.layer.23.attention.output.dense.weight", "encoder.layer.23.output.dense.weight"]


@pytest.mark.parametrize("name", ["bert_large_r64", "bert_large_r128", "bert_large_r256"])
def test_bert_large_rank_sweep_100_steps(name):
    """Rank sweep: sampled BERT-large tensors over 100 steps, through the all-bucket calls (the
    oracle's Gram-Schmidt takes seconds per factor at these ranks, so not every tensor)."""
    _require_gpu()
    wl = sg.WORKLOADS[name]
    names = list(BERT_SAMPLE)
    if wl.rank >= 256:
        # the oracle's Gram-Schmidt of the 30522 x 256 embedding factor takes about 20 s per
        # even step; test_bert_large_r256_embedding compares that matrix at steps 1 and 2
        names.remove("embeddings.word_embeddings.weight")
    rep = PU.run_parity(wl, "pool3", 100, CHECK, PU.tids_by_name(wl, names), free=FREE, grouped=True)
    _assert_ok(rep)


def test_bert_large_r256_embedding():
    """The 30522 x 1024 token embedding at rank 256 (30 Gram slices of its P factor, the blocked
    Cholesky of the 2 x 2 split) at steps 1 and 2, every element compared, all buckets running."""
    _require_gpu()
    wl = sg.WORKLOADS["bert_large_r256"]
    rep = PU.run_parity(wl, "fresh", 2, (1, 2), PU.tids_by_name(wl, ["embeddings.word_embeddings.weight"]),
                        grouped=True)
    _assert_ok(rep)


def _custom(shapes, rank, steps=12, cap=1 << 16, ef=True, mode="fresh", free=4):
    """Every tensor at every step: free-running for ``free`` steps, re-synced afterwards (a
    matrix whose rank r is close to min(n, m) amplifies rounding differences fastest)."""
    params = [sg.Param(f"t{i}", tuple(s)) for i, s in enumerate(shapes)]
    wl = sg.Workload("custom", params, rank, steps, lambda p: 0.05, seed=3, cap_bytes=cap)
    tids = list(range(len(shapes)))
    return PU.run_parity(wl, mode, steps, range(1, steps + 1), tids, ef=ef, free=free)


RAGGED = [(37, 3, 3), (5, 7), (129, 1030), (64,), (300, 147), (3,), (1000, 2048), (33, 65),
          (2, 900), (17, 4100), (260, 4608), (7, 5121)]


@pytest.mark.parametrize("rank", [1, 2, 4, 8, 16, 32, 64, 128, 256])
def test_ragged_shapes_all_ranks(rank):
    _require_gpu()
    _assert_ok(_custom(RAGGED, rank))


# rank 256 (the four waves of a workgroup split the rank; W in 2 x 2 blocks): ragged column
# tails, row counts just past r, a factor of 2100 rows (two Q-step chunks, several Gram slices)
RANK256 = [(257, 333), (2100, 300), (64,), (270, 1000)]


@pytest.mark.parametrize("ef", [True, False])
def test_rank256_ragged(ef):
    _require_gpu()
    _assert_ok(_custom(RANK256, 256, ef=ef))


# rows of at most 512 columns (the narrow rank-4 kernels): every lane shape (16, 32, 64 lanes,
# one or two float4 groups), ragged row counts, and a 3-element vector that leaves the factor
# offsets after it unaligned (those matrices take the general kernels)
NARROW = [(37, 8), (5, 12), (130, 64), (64,), (33, 128), (300, 256), (3,), (17, 500), (250, 512),
          (41, 36), (64, 64), (9, 132), (70, 4, 2, 2)]


@pytest.mark.parametrize("ef", [True, False])
def test_narrow_rows(ef):
    _require_gpu()
    _assert_ok(_custom(NARROW, 4, ef=ef))


# rank-4 matrices whose rows or factor offsets are not 16-byte aligned and that fit one
# workgroup (at most 256 rows and 512 columns: taken whole inside the row kernels' launches),
# at the limits and just past them (the general kernels), behind a 3-element vector that
# misaligns everything after it
SMALL = [(3,), (5, 5), (256, 512), (256, 511), (257, 147), (64, 3, 7, 7), (200, 513), (9, 2, 2),
         (255, 6), (6, 255)]


# rank-4 rows of 516 to 768 columns (three-wave P-step launch) and of 3076 to 4096 columns
# (eight-wave P-step launch): at both ends of those ranges and just past them, ragged row counts,
# beside a 1024-column matrix of the four-wave launches and a vector
THREE_WAVE = [(300, 516), (9, 768), (1000, 768), (129, 640), (64,), (37, 772), (260, 1024),
              (2, 512), (4100, 700), (37, 3076), (300, 4096), (5, 4000), (70, 3072), (33, 4100)]


@pytest.mark.parametrize("ef", [True, False])
def test_three_wave_rows(ef):
    _require_gpu()
    _assert_ok(_custom(THREE_WAVE, 4, ef=ef))


@pytest.mark.parametrize("ef", [True, False])
def test_small_unaligned_matrices(ef):
    _require_gpu()
    _assert_ok(_custom(SMALL, 4, ef=ef))


def test_error_feedback_off():
    _require_gpu()
    _assert_ok(_custom(RAGGED[:6] + [(256, 64, 3, 3)], 4, ef=False))


@pytest.mark.parametrize("rank", [8, 64, 128])
def test_error_feedback_off_mfma_ranks(rank):
    """Without error feedback the MFMA kernels read no E and write none (one-wave and
    rank-split kernels)."""
    _require_gpu()
    _assert_ok(_custom([(300, 1030), (64,), (129, 2048), (1000, 520)], rank, ef=False))


def test_single_bucket_of_vectors_and_tiny_cap():
    _require_gpu()
    _assert_ok(_custom([(10,), (20,), (8, 8), (30,)], 2, cap=16))


def test_zero_gradient_then_nonzero():
    _require_gpu()
    shapes = [(48, 40)]
    run = PU.Runner(shapes, 4)
    orc = AcpOracle(shapes, 4)
    zero = np.zeros((48, 40), np.float32)
    g2 = np.random.default_rng(0).standard_normal((48, 40)).astype(np.float32)
    for t, g in ((1, zero), (2, g2), (3, g2), (4, g2)):
        run.step(t, run.pack({0: g}))
        e = orc.compress_tensor(t, 0, g)
        o = orc.decompress_tensor(t, 0, e)
        torch.cuda.synchronize()
        if t == 1:
            assert np.all(run.factor_slice(t, 0) == 0) and np.all(run.out_slice(0) == 0)
            assert np.all(run.error_slice(0) == 0)
        if t == 2:  # orth(0) = 0 on both sides: Q = 0, M_hat = 0, E = M'
            assert np.all(run.ortho(t, 0) == 0) and np.all(run.factor_slice(t, 0) == 0)
            assert np.all(run.out_slice(0) == 0)
            assert np.array_equal(run.error_slice(0), g2.reshape(-1))
        assert PU.rel_err(run.out_slice(0), o) <= PU.TOL
        assert PU.rel_err(run.error_slice(0), orc.error(0)) <= PU.TOL


@pytest.mark.parametrize("rank,k", [(8, 3), (16, 5), (32, 10), (64, 20), (128, 40), (256, 100)])
def test_rank_deficient_high_rank(rank, k):
    """Gradients of exact rank k < r: from step 2 on the orthogonalisation drops r - k columns of
    the reused factor (r <= 64: the one-wave Cholesky; r = 128 and 256: kept and dropped pivots
    in the blocked Cholesky's first blocks, dropped ones only after them), on both sides alike.
    The kept columns' Gram-Schmidt is as ill-conditioned as a random k x k matrix, which scales
    the fp32 rounding difference from the fp64 oracle and makes it compound from step to step,
    so the oracle is re-synced from the device state before every step after the first: each
    step's arithmetic is checked on its own."""
    _require_gpu()
    shapes = [(300, 520)]
    run = PU.Runner(shapes, rank)
    orc = AcpOracle(shapes, rank)
    rng = np.random.default_rng(5)
    a = rng.standard_normal((300, k))
    b = rng.standard_normal((520, k))
    for t in range(1, 7):
        g = (a @ rng.standard_normal((k, k)) @ b.T / k).astype(np.float32)
        if t > 1:
            PU.read_state_into(run, orc, t - 1, [0])
        run.step(t, run.pack({0: g}))
        emit = orc.compress_tensor(t, 0, g)
        out = orc.decompress_tensor(t, 0, emit)
        torch.cuda.synchronize()
        st = orc.state[0]
        errs = {"emitted factor": PU.rel_err(run.factor_slice(t, 0), emit),
                "orthonormal factor": PU.rel_err(run.ortho(t, 0), st.ortho),
                "M_hat": PU.rel_err(run.out_slice(0), out),
                # after a Q-step E is zero up to rounding (the kept columns span M'), so its
                # error is measured against the gradient's norm
                "E": float(np.linalg.norm(run.error_slice(0) - orc.error(0).reshape(-1))
                           / max(np.linalg.norm(orc.error(0)), np.linalg.norm(g)))}
        PU.log(f"  rank {rank}, gradient rank {k}, t={t}: " + ", ".join(f"{n} {v:.2e}" for n, v in errs.items()))
        assert all(v <= PU.TOL for v in errs.values()), (t, errs)
        # the dropped columns are zero on both sides, the kept ones orthonormal
        f = run.ortho(t, 0).reshape(-1, rank).astype(np.float64)
        dropped = np.all(f == 0, axis=0)
        assert np.array_equal(dropped, np.all(st.ortho.reshape(-1, rank) == 0, axis=0)), t
        assert t == 1 or dropped.sum() == rank - k, (t, dropped.sum())
        kept = f[:, ~dropped]
        assert np.allclose(kept.T @ kept, np.eye(kept.shape[1]), atol=1e-5), t


def test_three_workers_loopback():
    """p = 3 workers on one GPU; the caller's all-reduce is a sum of their factor buffers."""
    _require_gpu()
    shapes = [(96, 80), (80,), (64, 3, 3, 3)]
    k = 3
    runs = [PU.Runner(shapes, 4, world=k) for _ in range(k)]
    lb = LoopbackOracle(k, shapes, 4)
    g = np.random.default_rng(1)
    for t in range(1, 9):
        grads = [{i: g.standard_normal(s).astype(np.float32) for i, s in enumerate(shapes)} for _ in range(k)]
        bufs = [r.pack(gr) for r, gr in zip(runs, grads)]
        for r, bb in zip(runs, bufs):
            r.acp.compress(t, 0, bb[0], r.fbuf[0])
        agg = sum(r.fbuf[0] for r in runs)
        for r in runs:
            r.acp.decompress(t, 0, agg, r.out[0])
        for tid in range(len(shapes)):
            outs, _ = lb.step_tensor(t, tid, [gr[tid] for gr in grads])
            for w, r in enumerate(runs):
                assert PU.rel_err(r.out_slice(tid), outs[w]) <= PU.TOL, (t, tid, w)
                if lb.workers[w].state[tid].E is not None:
                    assert PU.rel_err(r.error_slice(tid), lb.workers[w].error(tid)) <= PU.TOL
        # every worker keeps bitwise the same reused factor
        for tid in (0, 2):
            f0 = runs[0].ortho(t, tid)
            for r in runs[1:]:
                assert np.array_equal(r.ortho(t, tid), f0)


def test_step_sequencing_errors():
    _require_gpu()
    from paper_2306_08881_amd import _lib as L
    run = PU.Runner([(32, 24)], 4)
    g = run.pack({0: np.ones((32, 24), np.float32)})
    with pytest.raises(L.AcpError) as e:
        run.acp.compress(2, 0, g[0], run.fbuf[0])
    assert e.value.status == L.ACP_E_STEP
    with pytest.raises(L.AcpError) as e:
        run.acp.decompress(1, 0, run.fbuf[0], run.out[0])
    assert e.value.status == L.ACP_E_STEP
    run.acp.compress(1, 0, g[0], run.fbuf[0])
    with pytest.raises(L.AcpError) as e:
        run.acp.compress(1, 0, g[0], run.fbuf[0])
    assert e.value.status == L.ACP_E_STEP
    with pytest.raises(L.AcpError) as e:
        run.acp.decompress(2, 0, run.fbuf[0], run.out[0])
    assert e.value.status == L.ACP_E_STEP
    with pytest.raises(L.AcpError) as e:
        run.acp.compress(1, 0, g[0], g[0])                # factor buffer overlapping the gradient
    assert e.value.status in (L.ACP_E_STEP, L.ACP_E_INVALID)
    run.acp.decompress(1, 0, run.fbuf[0], run.out[0])
    run.acp.compress(2, 0, g[0], run.fbuf[0])
    run.acp.decompress(2, 0, run.fbuf[0], run.out[0])
