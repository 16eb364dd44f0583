"""Oracle draw of the initial low-rank factors P0 and Q0.

TEST INFRASTRUCTURE ONLY (see the package docstring).

The paper initialises P0 and Q0 from an i.i.d. standard normal distribution
(Section IV-A, "Power-SGD" and "Error-feedback").  It names no generator, so
the library and this oracle each implement the same published counter-based
generator, which makes the draw a pure function of (seed, tensor, factor,
element) and independent of bucket layout:

* SplitMix64's output finaliser ``mix`` (Steele, Lea and Flood, "Fast
  splittable pseudorandom number generators", OOPSLA 2014, with the
  finaliser constants of Stafford's variant 13), with golden-ratio increment
  gamma = 0x9E3779B97F4A7C15.  The generator with state x yields mix(x + k
  gamma) as its k-th output (k = 1, 2, ...).
* stream key: s = mix(seed XOR mix(2 * tensor_id + f)), f = 0 for P0 and 1
  for Q0.
* fresh factors of the no-reuse ablation (Section V-B: ACP-SGD "without
  reuse" draws the factor it would have reused anew at every step): the same
  generator with the step t >= 1 in the high half of the key,
  s = mix(seed XOR mix(t 2^32 + 2 * tensor_id + f)); t = 0 is P0 / Q0.
* element i (row-major): a = mix(s + (2i + 1) gamma), b = mix(s + (2i + 2) gamma),
  u1 = ((a >> 11) + 1) 2^-53 in (0, 1], u2 = (b >> 11) 2^-53 in [0, 1).
* Box-Muller (Box and Muller, 1958): z = sqrt(-2 ln u1) cos(2 pi u2) in
  float64 with the C library's ``log`` and ``cos`` (Python's ``math`` module
  calls the same functions), then rounded to the nearest float32.
"""

from __future__ import annotations

import math

import numpy as np

MASK64 = (1 << 64) - 1
GAMMA = 0x9E3779B97F4A7C15
MIX_M1 = 0xBF58476D1CE4E5B9
MIX_M2 = 0x94D049BB133111EB
TWO_PI = 2.0 * math.pi  # the float64 nearest to 2 pi


def mix(z: int) -> int:
    """SplitMix64 output finaliser on a Python int (mod 2^64)."""
    z &= MASK64
    z = ((z ^ (z >> 30)) * MIX_M1) & MASK64
    z = ((z ^ (z >> 27)) * MIX_M2) & MASK64
    return z ^ (z >> 31)


def splitmix64_stream(state: int, count: int) -> list:
    """The first ``count`` outputs of SplitMix64 started at ``state``."""
    return [mix(state + k * GAMMA) for k in range(1, count + 1)]


def _mix_vec(z: np.ndarray) -> np.ndarray:
    z = z.astype(np.uint64, copy=True)
    z ^= z >> np.uint64(30)
    z *= np.uint64(MIX_M1)
    z ^= z >> np.uint64(27)
    z *= np.uint64(MIX_M2)
    z ^= z >> np.uint64(31)
    return z


def stream_key(seed: int, tensor_id: int, factor: int, step: int = 0) -> int:
    return mix((seed & MASK64) ^ mix((step << 32) + 2 * tensor_id + factor))


def uniforms(seed: int, tensor_id: int, factor: int, count: int, step: int = 0):
    """(u1, u2) float64 arrays of the Box-Muller inputs for elements 0..count-1."""
    s = np.uint64(stream_key(seed, tensor_id, factor, step))
    i = np.arange(count, dtype=np.uint64)
    g = np.uint64(GAMMA)
    with np.errstate(over="ignore"):
        a = _mix_vec(s + (np.uint64(2) * i + np.uint64(1)) * g)
        b = _mix_vec(s + (np.uint64(2) * i + np.uint64(2)) * g)
    u1 = ((a >> np.uint64(11)) + np.uint64(1)).astype(np.float64) * 2.0 ** -53
    u2 = (b >> np.uint64(11)).astype(np.float64) * 2.0 ** -53
    return u1, u2


_log = np.frompyfunc(math.log, 1, 1)
_cos = np.frompyfunc(math.cos, 1, 1)


def normals(seed: int, tensor_id: int, factor: int, count: int, step: int = 0) -> np.ndarray:
    """float32 standard normals of one factor, element by element."""
    u1, u2 = uniforms(seed, tensor_id, factor, count, step)
    rad = np.sqrt(-2.0 * _log(u1).astype(np.float64))
    ang = _cos(TWO_PI * u2).astype(np.float64)
    return (rad * ang).astype(np.float32)


def init_factor(seed: int, tensor_id: int, which: str, rows: int, r: int) -> np.ndarray:
    """P0 (``which='P'``, rows = n) or Q0 (``which='Q'``, rows = m) as a float32 rows x r array."""
    f = 0 if which == "P" else 1
    return normals(seed, tensor_id, f, rows * r).reshape(rows, r)


def fresh_factor(seed: int, tensor_id: int, which: str, rows: int, r: int, step: int) -> np.ndarray:
    """The factor drawn anew at step ``step`` >= 1 without reuse, float32 rows x r."""
    f = 0 if which == "P" else 1
    return normals(seed, tensor_id, f, rows * r, step).reshape(rows, r)
