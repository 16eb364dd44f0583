"""ACP-SGD gradient compressor for AMD Instinct MI355X (gfx950).

The compressor of arXiv 2306.08881 (alternate compressed Power-SGD with error feedback,
Algorithm 2) behind the C ABI of include/acp.h, built as libacp.so from csrc/ with hipcc.
``paper_2306_08881_amd.acp.Acp`` is the Python binding.
"""

from ._lib import AcpError, load  # noqa: F401
