"""Pins of the oracle's Power-SGD with error feedback (Algorithm 1, left; the error applied as
Algorithm 2 applies it) to mathematics it must obey.

None of these re-types the oracle's formula: they check the error-feedback identities, exact
recovery of a rank-r gradient by one power iteration, convergence of repeated steps on a fixed
matrix to the top-r singular subspace of a brute-force SVD, the k-worker identity of the sums,
and that no-EF steps agree with the plain Algorithm 1 form.  ``test_planted_mistakes_are_caught``
plants plausible mistakes in the two halves of the step and checks that the suite rejects each.
"""

import numpy as np
import pytest

import oracle.acp as A
from oracle.gs import gram_schmidt

RTOL = 1e-12


def rel(x, y):
    return np.linalg.norm(np.asarray(x) - np.asarray(y)) / max(np.linalg.norm(y), 1e-300)


def _step(workers, t, tid, grads):
    """One Power-SGD step of tensor ``tid`` over k workers whose all-reduces are sums."""
    p_agg = sum(w.compress_p_tensor(t, tid, g) for w, g in zip(workers, grads))
    q_agg = sum(w.compress_q_tensor(t, tid, p_agg) for w in workers)
    return [w.decompress_tensor(t, tid, q_agg) for w in workers]


def check_ef_identities(seed=0):
    bad = []
    g = np.random.default_rng(seed)
    n, m, r = 13, 9, 3
    try:
        w = A.PowerSgdOracle([(n, m)], r, seed=seed)
        for t in range(1, 6):
            M = g.standard_normal((n, m))
            Mp = M + w.error(0)
            out = _step([w], t, 0, [M])[0]
            E, P = w.error(0), w.state[0].P
            if rel(E + out, Mp) > RTOL:
                bad.append(f"t={t}: E + M_hat != M + E_prev")
            if abs(np.linalg.norm(E) ** 2 + np.linalg.norm(out) ** 2 - np.linalg.norm(Mp) ** 2) \
                    > 1e-10 * np.linalg.norm(Mp) ** 2:
                bad.append(f"t={t}: Pythagoras")
            if np.abs(P.T @ E).max() > 1e-10 * np.abs(Mp).max():
                bad.append(f"t={t}: P^T E != 0")
            if np.abs(P.T @ P - np.eye(r)).max() > 1e-10:
                bad.append(f"t={t}: P not orthonormal")
    except Exception as e:  # shape errors from a transposed operand
        bad.append(f"identities: {type(e).__name__}: {e}")
    return bad


def check_exact_rank(seed=1):
    """A gradient of exact rank r is recovered by one power iteration from a generic Q: with
    E_0 = 0 every step returns M_t itself and leaves E = 0."""
    bad = []
    g = np.random.default_rng(seed)
    n, m, r = 14, 11, 3
    A_, B_ = g.standard_normal((n, r)), g.standard_normal((m, r))
    try:
        for ef in (True, False):
            w = A.PowerSgdOracle([(n, m)], r, seed=seed, ef=ef)
            for t in range(1, 6):
                M = A_ @ g.standard_normal((r, r)) @ B_.T
                out = _step([w], t, 0, [M])[0]
                if rel(out, M) > 1e-10:
                    bad.append(f"ef={ef} t={t}: rank-r gradient not recovered")
                if ef and np.abs(w.error(0)).max() > 1e-10 * np.abs(M).max():
                    bad.append(f"t={t}: E != 0 for a rank-r gradient")
    except Exception as e:
        bad.append(f"exact rank: {type(e).__name__}: {e}")
    return bad


def check_convergence(seed=3):
    """No error feedback, a fixed matrix: the steps are subspace iteration on M M^T, so P tends to
    the top-r left singular vectors (column by column, up to sign) and the error of M_hat to the
    Eckart-Young bound, both from a brute-force SVD."""
    bad = []
    n, m, r = 12, 9, 2
    g = np.random.default_rng(seed)
    U, _ = np.linalg.qr(g.standard_normal((n, n)))
    V, _ = np.linalg.qr(g.standard_normal((m, m)))
    s = 8.0 * 0.5 ** np.arange(m)
    M = (U[:, :m] * s) @ V.T
    try:
        w = A.PowerSgdOracle([(n, m)], r, seed=seed, ef=False)
        for t in range(1, 41):
            out = _step([w], t, 0, [M])[0]
        Ur = np.linalg.svd(M)[0][:, :r]
        P = w.state[0].P
        if np.linalg.norm(P - Ur @ (Ur.T @ P), 2) > 1e-10:
            bad.append("subspace not reached")
        for j in range(r):
            if min(np.abs(P[:, j] - Ur[:, j]).max(), np.abs(P[:, j] + Ur[:, j]).max()) > 1e-8:
                bad.append(f"column {j} is not +-u_{j}")
        if abs(np.linalg.norm(M - out) - np.sqrt((s[r:] ** 2).sum())) > 1e-10 * s[0]:
            bad.append("Eckart-Young error not reached")
    except Exception as e:
        bad.append(f"convergence: {type(e).__name__}: {e}")
    return bad


def check_loopback(seed=5, k=3):
    """k workers: all keep the same Q, return the same gradient, and with error feedback the
    errors and the returned mean add up to the workers' M' (E from each worker's local Q)."""
    bad = []
    g = np.random.default_rng(seed)
    n, m, r = 9, 7, 2
    try:
        ws = [A.PowerSgdOracle([(n, m)], r, seed=seed, world_size=k) for _ in range(k)]
        for t in range(1, 6):
            grads = [g.standard_normal((n, m)) for _ in range(k)]
            Eprev = [w.error(0).copy() for w in ws]
            outs = _step(ws, t, 0, grads)
            if any(not np.array_equal(w.state[0].Q, ws[0].state[0].Q) for w in ws[1:]):
                bad.append(f"t={t}: reused Q differs across workers")
            if any(rel(o, outs[0]) > 0 for o in outs[1:]):
                bad.append(f"t={t}: returned gradients differ")
            lhs = sum(w.error(0) for w in ws) + k * outs[0]
            rhs = sum(G + Ep for G, Ep in zip(grads, Eprev))
            if rel(lhs, rhs) > 1e-12:
                bad.append(f"t={t}: sum E + p M_hat != sum M'")
    except Exception as e:
        bad.append(f"loopback: {type(e).__name__}: {e}")
    return bad


def check_plain_algorithm_1(seed=6, k=2):
    """Without error feedback the three calls are Algorithm 1's Power-SGD over k workers."""
    bad = []
    g = np.random.default_rng(seed)
    n, m, r = 10, 8, 3
    try:
        ws = [A.PowerSgdOracle([(n, m)], r, seed=seed, world_size=k, ef=False) for _ in range(k)]
        for t in range(1, 4):
            grads = [g.standard_normal((n, m)) for _ in range(k)]
            Q_prev = ws[0].state[0].Q.copy()
            outs = _step(ws, t, 0, grads)
            ref, Q_ref = A.powersgd_matrix(grads, Q_prev)
            if rel(outs[0], ref) > 1e-12 or rel(ws[0].state[0].Q, Q_ref) > 1e-12:
                bad.append(f"t={t}: differs from Algorithm 1")
    except Exception as e:
        bad.append(f"algorithm 1: {type(e).__name__}: {e}")
    return bad


def check_ef_resends_the_residual(seed=7):
    """Error feedback at work: after a full-rank gradient, a zero gradient still sends the
    residual, M' = E_1 (P = E_1 Q), so M_hat_2 != 0 and the energy moves from E to M_hat."""
    bad = []
    g = np.random.default_rng(seed)
    n, m, r = 12, 10, 2
    try:
        w = A.PowerSgdOracle([(n, m)], r, seed=seed)
        _step([w], 1, 0, [g.standard_normal((n, m))])
        E1 = w.error(0).copy()
        out = _step([w], 2, 0, [np.zeros((n, m))])[0]
        if np.linalg.norm(out) < 1e-3 * np.linalg.norm(E1):
            bad.append("a zero gradient sent nothing: the residual was not fed back")
        if abs(np.linalg.norm(w.error(0)) ** 2 + np.linalg.norm(out) ** 2 - np.linalg.norm(E1) ** 2) \
                > 1e-10 * np.linalg.norm(E1) ** 2:
            bad.append("the fed-back residual is not split between E_2 and M_hat_2")
    except Exception as e:
        bad.append(f"feedback: {type(e).__name__}: {e}")
    return bad


ALL_CHECKS = [check_ef_identities, check_exact_rank, check_convergence, check_loopback,
              check_plain_algorithm_1, check_ef_resends_the_residual]


@pytest.mark.parametrize("check", ALL_CHECKS, ids=lambda c: c.__name__)
def test_invariant(check):
    assert check() == []


def test_vectors_and_sequencing():
    w = A.PowerSgdOracle([(5,), (6, 7)], 2, seed=0, world_size=2)
    v = np.arange(5.0)
    assert np.array_equal(w.compress_p_tensor(1, 0, v), v)
    assert np.array_equal(w.compress_q_tensor(1, 0, 2 * v), v)   # the raw vector again
    assert np.array_equal(w.decompress_tensor(1, 0, 2 * v), v)   # second all-reduce / p
    with pytest.raises(ValueError):
        w.compress_q_tensor(1, 1, np.zeros(12))                   # second half before the first
    w.compress_p_tensor(1, 1, np.zeros((6, 7)))
    with pytest.raises(ValueError):
        w.decompress_tensor(1, 1, np.zeros(14))                   # decompress before the second half


# ---------------------------------------------------------------- planted mistakes

def _mutants(kind):
    real_p, real_q = A.powersgd_p, A.powersgd_q

    def p(M, E, Q_prev):
        if kind == "drop_ef_in_product":
            P, Mp = real_p(M, E, Q_prev)
            return np.asarray(M, dtype=np.float64) @ Q_prev, Mp
        return real_p(M, E, Q_prev)

    def q(Mp, P_agg, ef):
        if kind == "no_orth":
            P = P_agg
        else:
            P = gram_schmidt(P_agg)
        Q = (Mp @ P) if kind == "transpose" else Mp.T @ P
        if not ef:
            return Q, P, None
        if kind == "sign":
            return Q, P, Mp + P @ Q.T
        if kind == "unorthogonalised_residual":
            return Q, P, Mp - P_agg @ Q.T
        return Q, P, Mp - P @ Q.T

    return p, q


@pytest.mark.parametrize("kind", ["no_orth", "transpose", "sign", "drop_ef_in_product",
                                  "unorthogonalised_residual"])
def test_planted_mistakes_are_caught(monkeypatch, kind):
    p, q = _mutants(kind)
    monkeypatch.setattr(A, "powersgd_p", p)
    monkeypatch.setattr(A, "powersgd_q", q)
    failures = [f for c in ALL_CHECKS for f in c()]
    assert failures, f"mistake {kind!r} went unnoticed"
