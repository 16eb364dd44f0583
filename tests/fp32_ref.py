"""A plain float32 re-implementation of one tensor's ACP-SGD step (Algorithm 2), for the drift
envelope.

It is written here, in the tests, independently of both the device library and the fp64 oracle:
NumPy float32 arithmetic with a Householder QR (numpy.linalg.qr, columns signed so that R has a
positive diagonal).  It is neither a reference for parity nor part of the product; it shows how far
*an* fp32 execution of the same method on the same inputs drifts from the fp64 oracle when every
step takes a fresh gradient and error feedback integrates the rounding differences.
"""

from __future__ import annotations

import numpy as np

from oracle import rng


def _orth32(a: np.ndarray) -> np.ndarray:
    q, r = np.linalg.qr(a.astype(np.float32))
    s = np.sign(np.diag(r)).astype(np.float32)
    s[s == 0] = 1
    return (q * s).astype(np.float32)


class Fp32Tensor:
    """One compressed tensor's state (P, Q, E in float32) at world size 1."""

    def __init__(self, seed: int, tid: int, n: int, m: int, rank: int):
        self.n, self.m = n, m
        self.P = rng.init_factor(seed, tid, "P", n, rank).astype(np.float32)
        self.Q = rng.init_factor(seed, tid, "Q", m, rank).astype(np.float32)
        self.E = np.zeros((n, m), np.float32)

    def step(self, t: int, grad: np.ndarray) -> np.ndarray:
        """Step t on the float32 gradient; returns M_hat (n x m)."""
        Mp = grad.reshape(self.n, self.m).astype(np.float32) + self.E
        if t % 2:
            self.Q = _orth32(self.Q)
            self.P = (Mp @ self.Q).astype(np.float32)
        else:
            self.P = _orth32(self.P)
            self.Q = (Mp.T @ self.P).astype(np.float32)
        out = (self.P @ self.Q.T).astype(np.float32)
        self.E = (Mp - out).astype(np.float32)
        return out
