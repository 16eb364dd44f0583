"""Seeded synthetic gradients for the benchmark workloads.

Every value is a float32 drawn from numpy's Philox counter-based generator
keyed by ``SeedSequence([seed, tensor_id, key])``, so any single tensor at any
step can be regenerated on its own without producing the rest of the model.
The float32 array is the canonical input: it is uploaded to the device as is
and widened exactly to float64 for the CPU oracle.

Value distributions (the workloads' stated recipe):

* single 3x3 conv: N(0, 0.01^2)
* ResNets: N(0, 1/fan_in) for weights (fan_in = product of all dims but the
  first), N(0, 1/numel) for 1-D tensors
* BERTs: N(0, 0.02^2) for every tensor

This module computes no part of the compressor.
"""

from __future__ import annotations

import math
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field
from typing import Callable, Dict, Iterable, List, Optional

import numpy as np

from . import shapes as S


def _sigma_const(value: float) -> Callable[[S.Param], float]:
    return lambda p: value


def _sigma_fan_in(p: S.Param) -> float:
    if len(p.shape) >= 2:
        fan_in = 1
        for d in p.shape[1:]:
            fan_in *= d
        return 1.0 / math.sqrt(fan_in)
    return 1.0 / math.sqrt(p.numel)


@dataclass(frozen=True)
class Workload:
    name: str
    params: List[S.Param] = field(repr=False)
    rank: int
    steps: int
    sigma: Callable[[S.Param], float] = field(repr=False)
    seed: int = 0
    cap_bytes: int = 25 * 1024 * 1024

    @property
    def ndims(self) -> List[int]:
        return [len(p.shape) for p in self.params]

    @property
    def dims(self) -> List[int]:
        return [d for p in self.params for d in p.shape]

    @property
    def numel(self) -> int:
        return sum(p.numel for p in self.params)


def _make() -> Dict[str, Workload]:
    w = {}
    w["conv256x576_r4"] = Workload("conv256x576_r4", S.single_conv(), 4, 10, _sigma_const(0.01))
    w["resnet50_r4"] = Workload("resnet50_r4", S.resnet50(), 4, 100, _sigma_fan_in)
    w["resnet152_r4"] = Workload("resnet152_r4", S.resnet152(), 4, 100, _sigma_fan_in)
    for r in (4, 32):
        w[f"bert_base_r{r}"] = Workload(f"bert_base_r{r}", S.bert_base(), r, 100, _sigma_const(0.02))
        w[f"bert_large_r{r}"] = Workload(f"bert_large_r{r}", S.bert_large(), r, 100, _sigma_const(0.02))
    # the rank sweep on the BERT-large shapes continues at r = 64, 128 and 256
    for r in (64, 128, 256):
        w[f"bert_large_r{r}"] = Workload(f"bert_large_r{r}", S.bert_large(), r, 100, _sigma_const(0.02))
    return w


WORKLOADS: Dict[str, Workload] = _make()


def gradient(wl: Workload, tensor_id: int, key: int) -> np.ndarray:
    """float32 gradient of parameter ``tensor_id`` (registration index) for input ``key``."""
    p = wl.params[tensor_id]
    g = np.random.Generator(np.random.Philox(np.random.SeedSequence([wl.seed, tensor_id, key])))
    z = g.standard_normal(p.numel, dtype=np.float32)
    z *= np.float32(wl.sigma(p))
    return z.reshape(p.shape)


def gradient_set(wl: Workload, key: int, tensor_ids: Optional[Iterable[int]] = None,
                 threads: int = 8) -> Dict[int, np.ndarray]:
    """Gradients of several tensors for one key, generated on a thread pool."""
    ids = list(range(len(wl.params))) if tensor_ids is None else list(tensor_ids)
    with ThreadPoolExecutor(max(1, threads)) as ex:
        arrs = list(ex.map(lambda i: gradient(wl, i, key), ids))
    return dict(zip(ids, arrs))


def zero_gradient(wl: Workload, tensor_id: int) -> np.ndarray:
    return np.zeros(wl.params[tensor_id].shape, dtype=np.float32)
