"""Oracle orthogonalisation: Gram-Schmidt, applied twice, in float64.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Algorithms 1 and 2 orthogonalise the reused factor before the product; the
implementation notes (Section IV-C) use a reduced QR decomposition.  The
result taken here is the Gram-Schmidt factor: the thin QR factor whose R has a
positive diagonal, which is unique for a full-column-rank input (a Householder
QR gives the same columns up to sign).  The columns are produced left to
right; each is projected against the earlier ones twice ("twice is enough",
Giraud, Langou and Rozloznik, 2005) and normalised.

Rank deficiency, on which the paper is silent: a column whose norm is zero, or
whose residual after the projections is at most ``tau`` times its original
norm, is set to zero (tau = 1e-4).  A zero column then takes no part in later
projections.
"""

from __future__ import annotations

import numpy as np

TAU = 1e-4


def gram_schmidt(a: np.ndarray, tau: float = TAU) -> np.ndarray:
    a = np.array(a, dtype=np.float64, copy=True)
    k, r = a.shape
    q = np.zeros((k, r), dtype=np.float64)
    for j in range(r):
        v = a[:, j].copy()
        norm_a = float(np.sqrt(v @ v))
        for _ in range(2):
            for i in range(j):
                v -= (q[:, i] @ v) * q[:, i]
        norm_v = float(np.sqrt(v @ v))
        if norm_a == 0.0 or norm_v <= tau * norm_a:
            continue
        q[:, j] = v / norm_v
    return q
