"""Seeded synthetic inputs shared by the CPU oracle and the device path.

Holds workload shape lists and a Philox-keyed gradient generator; it contains
none of the compressor's arithmetic.
"""

from .shapes import Param, resnet50, resnet152, bert_base, bert_large, single_conv  # noqa: F401
from .grads import WORKLOADS, Workload, gradient, gradient_set, zero_gradient  # noqa: F401
