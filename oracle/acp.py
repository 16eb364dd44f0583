"""Oracle ACP-SGD with error feedback, step by step, in float64.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Per compressed gradient matrix M_t (n x m) the state is the previous factors
P_{t-1} (n x r), Q_{t-1} (m x r) and the error E_{t-1} (n x m).  Algorithm 2:

* odd t (P-step): Q_t = orth(Q_{t-1});  P_t = (M_t + E_{t-1}) Q_t;
  E_t = M_t + E_{t-1} - P_t Q_t^T;  then P_t is all-reduced.
* even t (Q-step): P_t = orth(P_{t-1});  Q_t = (M_t + E_{t-1})^T P_t;
  E_t = M_t + E_{t-1} - P_t Q_t^T;  then Q_t is all-reduced.
* the step returns P_t Q_t^T with the aggregated factor.

Readings taken where the paper is silent (each listed in the design notes):

* t starts at 1, so the first step is a P-step and P0 is drawn but unused.
* E_t uses the local factor, computed before the all-reduce; the returned
  product and the factor kept for the next step use the aggregated one.
* the all-reduce sums (Section II-A aggregates the workers' gradients by addition), and the
  returned gradient is divided by the number of workers p, as S-SGD's mean.
* vector-shaped gradients pass through: sent raw, summed and divided by p.
* E_0 = 0 and P0, Q0 come from ``oracle.rng``.
* without error feedback (ablation, Section V-B) M' = M and no E is kept;
  without reuse the reused factor is replaced by a fresh standard normal draw
  every step: the initial factors' counter-based generator keyed by the step
  as well (``rng.fresh_factor``), so that the device can draw the same values.
"""

from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence

import numpy as np

from . import layout as L
from . import rng
from .gs import gram_schmidt


# ---- one matrix, Algorithm 2 --------------------------------------------------------------

def compress_matrix(t: int, M: np.ndarray, E: Optional[np.ndarray], P_prev: np.ndarray,
                    Q_prev: np.ndarray):
    """Algorithm 2 up to the all-reduce for one matrix.

    ``E`` is E_{t-1}, or None without error feedback.  Returns
    ``(emit, ortho, E_t)``: the local factor to be all-reduced (P_t on odd t,
    Q_t on even t), the orthogonalised reused factor (Q_t on odd t, P_t on
    even t) and the new error (None without error feedback).
    """
    Mp = np.asarray(M, dtype=np.float64)
    if E is not None:
        Mp = Mp + E
    if t % 2 == 1:
        q = gram_schmidt(Q_prev)        # Q_t = orth(Q_{t-1})
        p = Mp @ q                      # P_t = (M_t + E_{t-1}) Q_t
        E_new = Mp - p @ q.T if E is not None else None
        return p, q, E_new
    p = gram_schmidt(P_prev)            # P_t = orth(P_{t-1})
    q = Mp.T @ p                        # Q_t = (M_t + E_{t-1})^T P_t
    E_new = Mp - p @ q.T if E is not None else None
    return q, p, E_new


def decompress_matrix(t: int, agg: np.ndarray, ortho: np.ndarray, world_size: int):
    """Algorithm 2 after the all-reduce: returns (M_hat, P_t, Q_t) with the aggregated factor."""
    if t % 2 == 1:
        P, Q = agg, ortho
    else:
        P, Q = ortho, agg
    return (P @ Q.T) / world_size, P, Q


def powersgd_p(M: np.ndarray, E: Optional[np.ndarray], Q_prev: np.ndarray):
    """First half of a Power-SGD step (Algorithm 1, left) for one matrix, with error feedback.

    M' = M_t + E_{t-1} (M_t without error feedback) and the local P_t = M' Q_{t-1}, which the
    workers all-reduce before the second half.  Returns (P_t, M').
    """
    Mp = np.asarray(M, dtype=np.float64)
    if E is not None:
        Mp = Mp + E
    return Mp @ Q_prev, Mp


def powersgd_q(Mp: np.ndarray, P_agg: np.ndarray, ef: bool):
    """Second half: P_t = orth(all-reduced P_t); the local Q_t = M'^T P_t, all-reduced next;
    with error feedback E_t = M' - P_t Q_t^T with the local Q_t (before the all-reduce, where
    Algorithm 2 updates E).  Returns (Q_t, P_t, E_t or None)."""
    p = gram_schmidt(P_agg)
    q = Mp.T @ p
    return q, p, (Mp - p @ q.T if ef else None)


def powersgd_matrix(Ms: Sequence[np.ndarray], Q_prev: np.ndarray):
    """Power-SGD compression of Algorithm 1 (left) over the workers' matrices ``Ms``.

    P = all-reduce(M Q_{t-1}); P = orth(P); Q = all-reduce(M^T P); returns
    (P Q^T / p, Q) with the sums taken over workers and the mean returned.
    """
    Ms = [np.asarray(M, dtype=np.float64) for M in Ms]
    P = sum(M @ Q_prev for M in Ms)
    P = gram_schmidt(P)
    Q = sum(M.T @ P for M in Ms)
    return (P @ Q.T) / len(Ms), Q


# ---- the whole model ------------------------------------------------------------------------

@dataclass
class TensorState:
    plan: L.TensorPlan
    P: Optional[np.ndarray] = None       # reused factor state, float64
    Q: Optional[np.ndarray] = None
    E: Optional[np.ndarray] = None
    step: int = 0                        # last completed step
    pending: Optional[int] = None        # step compressed but not yet decompressed
    ortho: Optional[np.ndarray] = None   # orthogonalised factor of the pending / last step
    emit: Optional[np.ndarray] = None    # local factor (or raw vector) of the last compress


class AcpOracle:
    """ACP-SGD with error feedback over a model's fused buckets (one worker).

    ``tensor_ids`` restricts the state to a subset of tensors; every per-layer
    quantity depends only on that layer's own inputs, so a sample of layers of
    a large model is computed exactly as in the full model.
    """

    def __init__(self, shapes: Sequence[Sequence[int]], rank: int, seed: int = 0,
                 cap_bytes: int = L.DEFAULT_CAP_BYTES, world_size: int = 1, ef: bool = True,
                 reuse: bool = True, tensor_ids: Optional[Sequence[int]] = None):
        self.layout = L.plan(shapes, rank, cap_bytes)
        self.rank, self.seed, self.world_size = rank, seed, world_size
        self.ef, self.reuse = ef, reuse
        ids = range(len(shapes)) if tensor_ids is None else tensor_ids
        self.state: Dict[int, TensorState] = {}
        for tid in ids:
            pl = self.layout.tensors[tid]
            st = TensorState(pl)
            if pl.compressed:
                st.P = rng.init_factor(seed, tid, "P", pl.n, rank).astype(np.float64)
                st.Q = rng.init_factor(seed, tid, "Q", pl.m, rank).astype(np.float64)
                if ef:
                    st.E = np.zeros((pl.n, pl.m), dtype=np.float64)
            self.state[tid] = st

    def _fresh(self, tid: int, t: int, which: str, rows: int) -> np.ndarray:
        return rng.fresh_factor(self.seed, tid, which, rows, self.rank, t).astype(np.float64)

    def compress_tensor(self, t: int, tid: int, grad: np.ndarray) -> np.ndarray:
        """Local message of one tensor at step t, flattened (a factor or the raw vector)."""
        st = self.state[tid]
        if t != st.step + 1 or st.pending is not None:
            raise ValueError(f"tensor {tid}: step {t} out of order (last {st.step})")
        pl = st.plan
        g = np.asarray(grad, dtype=np.float64)
        if not pl.compressed:
            st.emit = g.reshape(-1).copy()
        else:
            M = g.reshape(pl.n, pl.m)
            P_prev, Q_prev = st.P, st.Q
            if not self.reuse:
                P_prev = self._fresh(tid, t, "P", pl.n)
                Q_prev = self._fresh(tid, t, "Q", pl.m)
            emit, st.ortho, E_new = compress_matrix(t, M, st.E, P_prev, Q_prev)
            st.E = E_new
            st.emit = emit.reshape(-1).copy()
        st.pending = t
        return st.emit

    def decompress_tensor(self, t: int, tid: int, agg: np.ndarray) -> np.ndarray:
        """Returned gradient of one tensor (its shape) from the aggregated message."""
        st = self.state[tid]
        if st.pending != t:
            raise ValueError(f"tensor {tid}: decompress({t}) without compress({t})")
        pl = st.plan
        agg = np.asarray(agg, dtype=np.float64)
        if not pl.compressed:
            out = (agg / self.world_size).reshape(pl.shape)
        else:
            rows = pl.n if t % 2 == 1 else pl.m
            M_hat, st.P, st.Q = decompress_matrix(t, agg.reshape(rows, self.rank), st.ortho,
                                                  self.world_size)
            out = M_hat.reshape(pl.shape)
        st.pending, st.step = None, t
        return out

    # bucket-level view: factor buffers laid out as in ``layout``

    def compress_bucket(self, t: int, b: int, grads: Dict[int, np.ndarray]) -> np.ndarray:
        bk = self.layout.buckets[b]
        size = bk.fac_elems_p if t % 2 == 1 else bk.fac_elems_q
        offs = bk.fac_off_p if t % 2 == 1 else bk.fac_off_q
        buf = np.zeros(size, dtype=np.float64)
        for tid, off in zip(bk.tids, offs):
            e = self.compress_tensor(t, tid, grads[tid])
            buf[off:off + e.size] = e
        return buf

    def decompress_bucket(self, t: int, b: int, agg: np.ndarray) -> Dict[int, np.ndarray]:
        bk = self.layout.buckets[b]
        offs = bk.fac_off_p if t % 2 == 1 else bk.fac_off_q
        out = {}
        for tid, off in zip(bk.tids, offs):
            size = self.layout.tensors[tid].factor_elems(self.rank, "P" if t % 2 == 1 else "Q")
            out[tid] = self.decompress_tensor(t, tid, agg[off:off + size])
        return out

    def error(self, tid: int) -> Optional[np.ndarray]:
        return self.state[tid].E


class LoopbackOracle:
    """k workers with the same seed and their own local gradients; the all-reduce is a sum."""

    def __init__(self, k: int, shapes: Sequence[Sequence[int]], rank: int, seed: int = 0, **kw):
        self.workers: List[AcpOracle] = [AcpOracle(shapes, rank, seed, world_size=k, **kw)
                                         for _ in range(k)]

    def step_tensor(self, t: int, tid: int, grads: Sequence[np.ndarray]):
        """One step of one tensor: returns (per-worker M_hat, the summed message)."""
        emits = [w.compress_tensor(t, tid, g) for w, g in zip(self.workers, grads)]
        agg = sum(emits)
        return [w.decompress_tensor(t, tid, agg) for w in self.workers], agg


@dataclass
class PsgdTensorState:
    plan: L.TensorPlan
    Q: Optional[np.ndarray] = None       # Q_{t-1}: the all-reduced Q of the last step (Q0 first)
    E: Optional[np.ndarray] = None
    Mp: Optional[np.ndarray] = None      # M' between the two halves of a step
    P: Optional[np.ndarray] = None       # orthonormal P_t of the last second half
    step: int = 0
    phase: int = 0                       # 0: idle, 1: P sent, 2: Q sent
    emit_p: Optional[np.ndarray] = None
    emit_q: Optional[np.ndarray] = None


class PowerSgdOracle:
    """Power-SGD with error feedback (Algorithm 1, left) over a model's tensors, one worker.

    Per step t and compressed tensor, in three calls with an all-reduce after each of the first
    two: ``compress_p_tensor`` (M' = M + E, local P = M' Q_{t-1}), ``compress_q_tensor`` (P =
    orth(all-reduced P), local Q = M'^T P, E = M' - P Q^T), ``decompress_tensor`` (M_hat = P
    Q_agg^T / p; Q_agg is reused at t + 1).  Q_0 is the same draw as ACP-SGD's (``rng``).
    Vectors are sent raw in both halves; the returned vector is the second all-reduce / p.
    """

    def __init__(self, shapes: Sequence[Sequence[int]], rank: int, seed: int = 0,
                 cap_bytes: int = L.DEFAULT_CAP_BYTES, world_size: int = 1, ef: bool = True,
                 tensor_ids: Optional[Sequence[int]] = None):
        self.layout = L.plan(shapes, rank, cap_bytes)
        self.rank, self.seed, self.world_size, self.ef = rank, seed, world_size, ef
        ids = range(len(shapes)) if tensor_ids is None else tensor_ids
        self.state: Dict[int, PsgdTensorState] = {}
        for tid in ids:
            pl = self.layout.tensors[tid]
            st = PsgdTensorState(pl)
            if pl.compressed:
                st.Q = rng.init_factor(seed, tid, "Q", pl.m, rank).astype(np.float64)
                if ef:
                    st.E = np.zeros((pl.n, pl.m), dtype=np.float64)
            self.state[tid] = st

    def compress_p_tensor(self, t: int, tid: int, grad: np.ndarray) -> np.ndarray:
        st = self.state[tid]
        if t != st.step + 1 or st.phase != 0:
            raise ValueError(f"tensor {tid}: first half of step {t} out of order")
        g = np.asarray(grad, dtype=np.float64)
        if st.plan.compressed:
            p, st.Mp = powersgd_p(g.reshape(st.plan.n, st.plan.m), st.E, st.Q)
            st.emit_p = p.reshape(-1).copy()
        else:
            st.Mp = g.reshape(-1).copy()
            st.emit_p = st.Mp.copy()
        st.phase = 1
        return st.emit_p

    def compress_q_tensor(self, t: int, tid: int, p_agg: np.ndarray) -> np.ndarray:
        st = self.state[tid]
        if t != st.step + 1 or st.phase != 1:
            raise ValueError(f"tensor {tid}: second half of step {t} out of order")
        if st.plan.compressed:
            P_agg = np.asarray(p_agg, dtype=np.float64).reshape(st.plan.n, self.rank)
            q, st.P, E_new = powersgd_q(st.Mp, P_agg, self.ef)
            st.E = E_new
            st.emit_q = q.reshape(-1).copy()
        else:
            st.emit_q = st.Mp.copy()
        st.Mp = None
        st.phase = 2
        return st.emit_q

    def decompress_tensor(self, t: int, tid: int, q_agg: np.ndarray) -> np.ndarray:
        st = self.state[tid]
        if t != st.step + 1 or st.phase != 2:
            raise ValueError(f"tensor {tid}: decompress({t}) before both halves")
        agg = np.asarray(q_agg, dtype=np.float64)
        if st.plan.compressed:
            st.Q = agg.reshape(st.plan.m, self.rank)
            out = ((st.P @ st.Q.T) / self.world_size).reshape(st.plan.shape)
        else:
            out = (agg / self.world_size).reshape(st.plan.shape)
        st.phase, st.step = 0, t
        return out

    def error(self, tid: int) -> Optional[np.ndarray]:
        return self.state[tid].E
