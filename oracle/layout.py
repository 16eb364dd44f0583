"""Oracle layout planner: which gradients are compressed, their matrix shape,
the tensor-fusion buckets and the offsets inside each bucket's buffers.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Rules, each with the passage it follows:

* Reshape and eligibility (Section IV-C, implementation): vector-shaped
  parameters are not compressed; every other parameter is reshaped into a
  matrix.  The matrix is n x m with n = the first dimension (output channels,
  output features, vocabulary) and m = the product of the remaining ones.  A
  tensor whose matrix has r >= min(n, m) gains nothing from a rank-r
  factorisation and is passed through like a vector.
* Buckets (Section IV-B, "Buffer Size"; 25 MB default of PyTorch-DDP): the
  tensors are visited in backward order (reverse registration order); each
  whole tensor is appended to the open bucket and the bucket is closed as soon
  as its size reaches the cap.  MB is read as MiB.  With this rule the
  ResNet-50 gradients (97.5 MB) form 4 buckets, as the paper states.
* Factor buffer (Section IV-B and IV-C): the tensor copied into the fusion
  buffer is the compressed factor (P, n x r, on P-steps; Q, m x r, on
  Q-steps) or, for uncompressed tensors, the raw gradient.  Each bucket's
  factor buffer holds them packed in bucket order.
* Compressed fusion (Section IV-B, "Buffer Size"): the compressed buffer size
  is the gradient buffer size scaled by the compression rate, computed
  separately for P and for Q, and P (Q) tensors are grouped with it by the
  same closing rule.
"""

from __future__ import annotations

from dataclasses import dataclass, field
from math import prod
from typing import List, Sequence, Tuple

MIB = 1 << 20
DEFAULT_CAP_BYTES = 25 * MIB
ELEM_BYTES = 4  # fp32 gradients


@dataclass(frozen=True)
class TensorPlan:
    tid: int            # registration index
    shape: Tuple[int, ...]
    numel: int
    compressed: bool
    n: int              # matrix rows (dim 0); numel for passthrough tensors
    m: int              # matrix columns (product of the rest); 1 for passthrough

    def factor_elems(self, r: int, parity: str) -> int:
        """Elements this tensor contributes to a P-step ('P') or Q-step ('Q') factor buffer."""
        if not self.compressed:
            return self.numel
        return self.n * r if parity == "P" else self.m * r


@dataclass
class Bucket:
    tids: List[int] = field(default_factory=list)
    grad_off: List[int] = field(default_factory=list)   # element offset of each tensor in the gradient bucket
    fac_off_p: List[int] = field(default_factory=list)  # element offset in the P-step factor buffer
    fac_off_q: List[int] = field(default_factory=list)  # element offset in the Q-step factor buffer
    grad_elems: int = 0
    fac_elems_p: int = 0
    fac_elems_q: int = 0


def plan_tensor(tid: int, shape: Sequence[int], r: int) -> TensorPlan:
    shape = tuple(int(d) for d in shape)
    numel = prod(shape) if shape else 1
    if len(shape) >= 2:
        n, m = shape[0], prod(shape[1:])
        if r < min(n, m):
            return TensorPlan(tid, shape, numel, True, n, m)
    return TensorPlan(tid, shape, numel, False, numel, 1)


def plan_tensors(shapes: Sequence[Sequence[int]], r: int) -> List[TensorPlan]:
    return [plan_tensor(i, s, r) for i, s in enumerate(shapes)]


def group_backward(sizes_bytes: Sequence[int], cap_bytes: float) -> List[List[int]]:
    """Greedy grouping in backward order: indices into ``sizes_bytes`` (registration order).

    A group is closed once its byte size reaches ``cap_bytes``; a tensor larger
    than the cap therefore closes the group it lands in.
    """
    groups: List[List[int]] = []
    cur: List[int] = []
    cur_bytes = 0
    for i in reversed(range(len(sizes_bytes))):
        cur.append(i)
        cur_bytes += sizes_bytes[i]
        if cur_bytes >= cap_bytes:
            groups.append(cur)
            cur, cur_bytes = [], 0
    if cur:
        groups.append(cur)
    return groups


def plan_buckets(plans: Sequence[TensorPlan], r: int, cap_bytes: int = DEFAULT_CAP_BYTES) -> List[Bucket]:
    buckets = []
    for group in group_backward([p.numel * ELEM_BYTES for p in plans], cap_bytes):
        b = Bucket()
        for tid in group:
            p = plans[tid]
            b.tids.append(tid)
            b.grad_off.append(b.grad_elems)
            b.fac_off_p.append(b.fac_elems_p)
            b.fac_off_q.append(b.fac_elems_q)
            b.grad_elems += p.numel
            b.fac_elems_p += p.factor_elems(r, "P")
            b.fac_elems_q += p.factor_elems(r, "Q")
        buckets.append(b)
    return buckets


@dataclass
class Layout:
    rank: int
    cap_bytes: int
    tensors: List[TensorPlan]
    buckets: List[Bucket]

    @property
    def numel(self) -> int:
        return sum(t.numel for t in self.tensors)

    def bucket_of(self, tid: int) -> Tuple[int, int]:
        """(bucket index, position inside the bucket) of a tensor."""
        for bi, b in enumerate(self.buckets):
            if tid in b.tids:
                return bi, b.tids.index(tid)
        raise KeyError(tid)


def plan(shapes: Sequence[Sequence[int]], r: int, cap_bytes: int = DEFAULT_CAP_BYTES) -> Layout:
    tensors = plan_tensors(shapes, r)
    return Layout(r, cap_bytes, tensors, plan_buckets(tensors, r, cap_bytes))


# ---- quantities the paper prints about the layout -------------------------------------------

def factor_totals(layout: Layout) -> Tuple[int, int]:
    """Total elements sent on a P-step and on a Q-step (factors plus raw vectors)."""
    p = sum(t.factor_elems(layout.rank, "P") for t in layout.tensors)
    q = sum(t.factor_elems(layout.rank, "Q") for t in layout.tensors)
    return p, q


def compression_rates(layout: Layout) -> Tuple[float, float]:
    """Compression rates of P-steps and Q-steps: sent elements over gradient elements."""
    p, q = factor_totals(layout)
    return p / layout.numel, q / layout.numel


def compressed_fusion_groups(layout: Layout) -> Tuple[List[List[int]], List[List[int]]]:
    """P and Q fusion groups with the cap scaled by each compression rate."""
    rate_p, rate_q = compression_rates(layout)
    sizes_p = [t.factor_elems(layout.rank, "P") * ELEM_BYTES for t in layout.tensors]
    sizes_q = [t.factor_elems(layout.rank, "Q") * ELEM_BYTES for t in layout.tensors]
    return (group_backward(sizes_p, layout.cap_bytes * rate_p),
            group_backward(sizes_q, layout.cap_bytes * rate_q))


def powersgd_ratio(layout: Layout) -> float:
    """Power-SGD sends both P and Q every step: N / ((sum n + sum m) r + N_1)."""
    p, q = factor_totals(layout)
    n1 = sum(t.numel for t in layout.tensors if not t.compressed)
    return layout.numel / (p + q - n1)


def acp_ratio(layout: Layout) -> float:
    """ACP-SGD sends P or Q, alternately: N / ((sum n + sum m) r / 2 + N_1)."""
    p, q = factor_totals(layout)
    n1 = sum(t.numel for t in layout.tensors if not t.compressed)
    return layout.numel / ((p + q - 2 * n1) / 2 + n1)
