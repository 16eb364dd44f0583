"""Pins of the oracle's ACP-SGD step (Algorithm 2) to mathematics it must obey.

None of these re-types the oracle's formula: they check identities and limits
that any correct implementation satisfies (the residual/projection identities
of error feedback, exact recovery of rank-r gradients, convergence of the
alternation to the top-r singular subspace from a brute-force SVD, the
equivalence with Power-SGD that the paper states, and the k-worker semantics).
``test_planted_mistakes_are_caught`` plants plausible mistakes in the oracle's
per-matrix step and checks that the same suite rejects each of them.
"""

import numpy as np
import pytest

import oracle.acp as A
from oracle.gs import gram_schmidt

RTOL = 1e-12


def rel(x, y):
    d = np.linalg.norm(np.asarray(x) - np.asarray(y))
    s = max(np.linalg.norm(y), 1e-300)
    return d / s


def _rng(seed):
    return np.random.default_rng(seed)


# ---------------------------------------------------------------- invariant checks
# Each returns a list of failure strings; the tests assert it is empty, and the
# planted-mistake test asserts it is not.

def check_residual_identities(seed=0):
    bad = []
    g = _rng(seed)
    n, m, r = 13, 9, 3
    for t in (1, 2, 3, 4):
        M = g.standard_normal((n, m))
        E = g.standard_normal((n, m)) * 0.3
        P_prev, Q_prev = g.standard_normal((n, r)), g.standard_normal((m, r))
        try:
            bad += _residual_case(t, M, E, P_prev, Q_prev, r)
        except Exception as e:  # shape errors from a transposed operand
            bad.append(f"t={t}: {type(e).__name__}")
    return bad


def _residual_case(t, M, E, P_prev, Q_prev, r):
    bad = []
    emit, ortho, E_new = A.compress_matrix(t, M, E, P_prev, Q_prev)
    M_hat, P, Q = A.decompress_matrix(t, emit, ortho, 1)
    Mp = M + E
    if rel(E_new + M_hat, Mp) > RTOL:
        bad.append(f"t={t}: E + M_hat != M + E_prev")
    if abs(np.linalg.norm(E_new) ** 2 + np.linalg.norm(M_hat) ** 2 - np.linalg.norm(Mp) ** 2) \
            > 1e-10 * np.linalg.norm(Mp) ** 2:
        bad.append(f"t={t}: Pythagoras")
    if t % 2 == 1:
        if np.abs(E_new @ Q).max() > 1e-10 * np.abs(Mp).max():
            bad.append(f"t={t}: E Q_hat != 0")
        if rel(Q, gram_schmidt(Q_prev)) > 1e-10 or rel(emit, Mp @ Q) > RTOL:
            bad.append(f"t={t}: P-step factors")
    else:
        if np.abs(P.T @ E_new).max() > 1e-10 * np.abs(Mp).max():
            bad.append(f"t={t}: P_hat^T E != 0")
        if np.abs(P.T @ P - np.eye(r)).max() > 1e-10:
            bad.append(f"t={t}: P_hat not orthonormal")
    return bad


def _run_single(M_seq, r, ef, n, m, seed=0):
    orc = A.AcpOracle([(n, m)], r, seed=seed, ef=ef)
    outs, errs = [], []
    for t, M in enumerate(M_seq, start=1):
        e = orc.compress_tensor(t, 0, M)
        outs.append(orc.decompress_tensor(t, 0, e))
        errs.append(None if orc.error(0) is None else orc.error(0).copy())
    return outs, errs


def check_exact_rank(seed=1):
    bad = []
    g = _rng(seed)
    n, m, r = 14, 11, 3
    Au, Bv = g.standard_normal((n, r)), g.standard_normal((m, r))
    Ms = [Au @ g.standard_normal((r, r)) @ Bv.T for _ in range(8)]
    try:
        outs, _ = _run_single(Ms, r, ef=False, n=n, m=m, seed=seed)
        for t in range(2, 9):
            if rel(outs[t - 1], Ms[t - 1]) > 1e-10:
                bad.append(f"no-EF rank-r gradient not recovered at t={t}")
        outs, errs = _run_single(Ms, r, ef=True, n=n, m=m, seed=seed)
        for t in range(2, 9, 2):
            if np.abs(errs[t - 1]).max() > 1e-10 * np.abs(Ms[t - 1]).max():
                bad.append(f"EF Q-step t={t}: E != 0")
            if rel(outs[t - 1], Ms[t - 1] + errs[t - 2]) > 1e-10:
                bad.append(f"EF Q-step t={t}: M_hat != M + E_prev")
    except Exception as e:
        bad.append(f"exact rank: {type(e).__name__}: {e}")
    return bad


def planted_matrix(n=12, m=9, r=2, seed=3):
    g = _rng(seed)
    U, _ = np.linalg.qr(g.standard_normal((n, n)))
    V, _ = np.linalg.qr(g.standard_normal((m, m)))
    k = min(n, m)
    s = 8.0 * 0.5 ** np.arange(k)
    return (U[:, :k] * s) @ V[:, :k].T, U[:, :k], s, V[:, :k]


def check_convergence(seed=3):
    bad = []
    n, m, r = 12, 9, 2
    M, U, s, V = planted_matrix(n, m, r, seed)
    try:
        orc = A.AcpOracle([(n, m)], r, seed=seed, ef=False)
        for t in range(1, 61):
            e = orc.compress_tensor(t, 0, M)
            out = orc.decompress_tensor(t, 0, e)
        st = orc.state[0]
        Ur, Vr = np.linalg.svd(M)[0][:, :r], np.linalg.svd(M)[2][:r].T
        Ph, Qh = gram_schmidt(st.P), gram_schmidt(st.Q)
        sin_p = np.linalg.norm(Ph - Ur @ (Ur.T @ Ph), 2)
        sin_q = np.linalg.norm(Qh - Vr @ (Vr.T @ Qh), 2)
        if sin_p > 1e-10 or sin_q > 1e-10:
            bad.append(f"subspace not reached: {sin_p:.2e} {sin_q:.2e}")
        ey = np.sqrt((s[r:] ** 2).sum())
        if abs(np.linalg.norm(M - out) - ey) > 1e-10 * s[0]:
            bad.append("Eckart-Young error not reached")
        for j in range(r):
            if min(np.abs(Ph[:, j] - Ur[:, j]).max(), np.abs(Ph[:, j] + Ur[:, j]).max()) > 1e-8:
                bad.append(f"column {j} is not +-u_{j}")
    except Exception as e:
        bad.append(f"convergence: {type(e).__name__}: {e}")
    return bad


def check_powersgd_equivalence(seed=4):
    bad = []
    g = _rng(seed)
    n, m, r = 10, 8, 3
    try:
        orc = A.AcpOracle([(n, m)], r, seed=seed, ef=False)
        for t in (1, 2):
            orc.decompress_tensor(t, 0, orc.compress_tensor(t, 0, g.standard_normal((n, m))))
        M = g.standard_normal((n, m))
        Q_prev = orc.state[0].Q.copy()
        orc.decompress_tensor(3, 0, orc.compress_tensor(3, 0, M))
        out = orc.decompress_tensor(4, 0, orc.compress_tensor(4, 0, M))
        ref, _ = A.powersgd_matrix([M], Q_prev)
        if rel(out, ref) > 1e-10:
            bad.append("two alternate steps != one Power-SGD step")
    except Exception as e:
        bad.append(f"power-sgd: {type(e).__name__}: {e}")
    return bad


def check_loopback(seed=5, k=3):
    bad = []
    g = _rng(seed)
    n, m, r = 9, 7, 2
    try:
        lb = A.LoopbackOracle(k, [(n, m)], r, seed=seed)
        for t in range(1, 7):
            grads = [g.standard_normal((n, m)) for _ in range(k)]
            Eprev = [w.error(0).copy() for w in lb.workers]
            outs, _ = lb.step_tensor(t, 0, grads)
            for w in lb.workers[1:]:
                if not (np.array_equal(w.state[0].P, lb.workers[0].state[0].P)
                        and np.array_equal(w.state[0].Q, lb.workers[0].state[0].Q)):
                    bad.append(f"t={t}: reused factors differ across workers")
            if any(rel(o, outs[0]) > 0 for o in outs[1:]):
                bad.append(f"t={t}: returned gradients differ across workers")
            lhs = sum(w.error(0) for w in lb.workers) + k * outs[0]
            rhs = sum(G + Ep for G, Ep in zip(grads, Eprev))
            if rel(lhs, rhs) > 1e-12:
                bad.append(f"t={t}: sum E + p M_hat != sum M'")
    except Exception as e:
        bad.append(f"loopback: {type(e).__name__}: {e}")
    return bad


ALL_CHECKS = [check_residual_identities, check_exact_rank, check_convergence,
              check_powersgd_equivalence, check_loopback]


# ---------------------------------------------------------------- tests

@pytest.mark.parametrize("check", ALL_CHECKS, ids=lambda c: c.__name__)
def test_invariant(check):
    assert check() == []


@pytest.mark.parametrize("seed", range(1, 6))
def test_residual_identities_many_seeds(seed):
    assert check_residual_identities(seed) == []


def test_full_rank_factor_is_exact():
    g = _rng(6)
    n, m = 6, 5
    M, E = g.standard_normal((n, m)), g.standard_normal((n, m))
    # r = m: the P-step projector Q Q^T is the identity
    emit, ortho, E_new = A.compress_matrix(1, M, E, g.standard_normal((n, m)), g.standard_normal((m, m)))
    assert np.abs(E_new).max() < 1e-12
    # r = n: the Q-step projector P P^T is the identity
    emit, ortho, E_new = A.compress_matrix(2, M, E, g.standard_normal((n, n)), g.standard_normal((m, n)))
    assert np.abs(E_new).max() < 1e-12


def test_p_steps_not_exact_with_ef():
    """With EF on, P-steps after t=1 are not exact for rank-r input (the claim is Q-steps only)."""
    g = _rng(1)
    n, m, r = 14, 11, 3
    Au, Bv = g.standard_normal((n, r)), g.standard_normal((m, r))
    Ms = [Au @ g.standard_normal((r, r)) @ Bv.T for _ in range(5)]
    _, errs = _run_single(Ms, r, ef=True, n=n, m=m, seed=1)
    assert np.abs(errs[2]).max() > 1e-6


def test_zero_gradient_degenerate_case():
    n, m, r = 8, 6, 2
    orc = A.AcpOracle([(n, m)], r, seed=0)
    e1 = orc.compress_tensor(1, 0, np.zeros((n, m)))
    assert np.all(e1 == 0)
    out1 = orc.decompress_tensor(1, 0, e1)
    assert np.all(out1 == 0) and np.all(orc.error(0) == 0)
    M2 = _rng(7).standard_normal((n, m))
    e2 = orc.compress_tensor(2, 0, M2)          # P_hat = orth(0) = 0, so Q = 0
    assert np.all(orc.state[0].ortho == 0) and np.all(e2 == 0)
    out2 = orc.decompress_tensor(2, 0, e2)
    assert np.all(out2 == 0) and np.array_equal(orc.error(0), M2)


def test_reuse_off_is_a_fresh_projection():
    n, m, r = 12, 9, 2
    M, *_ = planted_matrix(n, m, r, 3)
    orc = A.AcpOracle([(n, m)], r, seed=3, ef=False, reuse=False)
    errs = []
    for t in range(1, 41):
        out = orc.decompress_tensor(t, 0, orc.compress_tensor(t, 0, M))
        errs.append(np.linalg.norm(M - out))
        Qh = orc.state[0].ortho
        if t % 2 == 1:
            assert rel(out, M @ Qh @ Qh.T) < 1e-12
    # without reuse the error does not settle to the Eckart-Young bound
    assert np.std(errs[-10:]) > 1e-3


def test_vectors_pass_through_and_mean():
    lb = A.LoopbackOracle(2, [(5,), (6, 7)], 2, seed=0)
    g = _rng(8)
    v = [g.standard_normal(5) for _ in range(2)]
    outs, agg = lb.step_tensor(1, 0, v)
    assert np.allclose(outs[0], (v[0] + v[1]) / 2, rtol=0, atol=1e-15)


def test_step_order_enforced():
    orc = A.AcpOracle([(6, 5)], 2)
    with pytest.raises(ValueError):
        orc.compress_tensor(2, 0, np.zeros((6, 5)))
    orc.compress_tensor(1, 0, np.zeros((6, 5)))
    with pytest.raises(ValueError):
        orc.compress_tensor(2, 0, np.zeros((6, 5)))
    with pytest.raises(ValueError):
        orc.decompress_tensor(2, 0, np.zeros(12))


def test_bucket_view_matches_tensor_view():
    import synthgrad as sg
    wl = sg.WORKLOADS["resnet50_r4"]
    shapes = [p.shape for p in wl.params]
    a = A.AcpOracle(shapes, 4, tensor_ids=None)
    b_idx = 3  # the last bucket holds the first (smallest) layers
    tids = a.layout.buckets[b_idx].tids
    grads = {t: sg.gradient(wl, t, 1) for t in tids}
    buf = a.compress_bucket(1, b_idx, grads)
    outs = a.decompress_bucket(1, b_idx, buf)
    c = A.AcpOracle(shapes, 4, tensor_ids=tids)
    for t in tids:
        e = c.compress_tensor(1, t, grads[t])
        assert np.array_equal(outs[t], c.decompress_tensor(1, t, e))


# ---------------------------------------------------------------- planted mistakes

def _mutant(kind):
    def f(t, M, E, P_prev, Q_prev):
        Mp = np.asarray(M, dtype=np.float64) + (E if E is not None else 0)
        odd = (t % 2 == 1) if kind != "parity" else (t % 2 == 0)
        if kind == "no_orth":
            ortho_fn = lambda X: X
        else:
            ortho_fn = gram_schmidt
        if odd:
            q = ortho_fn(Q_prev)
            src = M if kind == "drop_ef_in_product" else Mp
            p = np.asarray(src, dtype=np.float64) @ q
            if kind == "sign":
                En = Mp + p @ q.T
            elif kind == "drop_ef_in_residual":
                En = np.asarray(M, dtype=np.float64) - p @ q.T
            else:
                En = Mp - p @ q.T
            return p, q, (En if E is not None else None)
        p = ortho_fn(Q_prev if kind == "wrong_factor" else P_prev)
        q = (Mp @ p) if kind == "transpose" else Mp.T @ p
        En = Mp - p @ q.T
        if kind == "sign":
            En = Mp + p @ q.T
        return q, p, (En if E is not None else None)

    return f


@pytest.mark.parametrize("kind", ["no_orth", "sign", "drop_ef_in_product", "drop_ef_in_residual",
                                  "parity", "transpose", "wrong_factor"])
def test_planted_mistakes_are_caught(monkeypatch, kind):
    monkeypatch.setattr(A, "compress_matrix", _mutant(kind))
    failures = [f for c in ALL_CHECKS for f in c()]
    assert failures, f"mistake {kind!r} went unnoticed"
