"""acp_compress_noalloc, the compress entry point that allocates nothing (its Q-step partial sums
go to the library's static device array instead of the state block), against acp_compress.

Two contexts with the same shapes, rank and seed take the same gradients, one through each
entry point; both decompress through acp_decompress.  The factor buffers, the outputs and E must
be bitwise equal (same kernels, same order of every sum).  The cases run in a row in one process,
each with less Q-step scratch than the one before, so each later call runs over what the earlier
ones left in the array.
"""

import numpy as np
import pytest
import torch

from tests import parity_util as PU

pytestmark = pytest.mark.gpu

# (rank, shapes): partial sums per case fall from 2.0 MiB to 0.9 MiB to 0.1 MiB
CASES = [(32, [(2048, 1024), (1024,), (600, 520)]),
         (4, [(3000, 1024), (64,), (600, 520), (37, 3, 3)]),
         (4, [(300, 512), (64,)])]


def _run_case(rank, shapes, seed):
    ref = PU.Runner(shapes, rank, seed=seed)
    new = PU.Runner(shapes, rank, seed=seed)
    rng = np.random.default_rng(seed)
    for t in range(1, 5):
        grads = {i: (0.02 * rng.standard_normal(s)).astype(np.float32) for i, s in enumerate(shapes)}
        gb = ref.pack(grads)
        for b in range(ref.nb):
            ref.acp.compress(t, b, gb[b], ref.fbuf[b])
            new.acp.compress_noalloc(t, b, gb[b], new.fbuf[b])
        torch.cuda.synchronize()
        for b in range(ref.nb):
            assert torch.equal(ref.fbuf[b], new.fbuf[b]), (rank, t, b, "factor buffer")
            ref.acp.decompress(t, b, ref.fbuf[b], ref.out[b])
            new.acp.decompress(t, b, new.fbuf[b], new.out[b])
            ref.acp.error(b, ref.ebuf[b])
            new.acp.error(b, new.ebuf[b])
        torch.cuda.synchronize()
        for b in range(ref.nb):
            assert torch.equal(ref.out[b], new.out[b]), (rank, t, b, "M_hat")
            assert torch.equal(ref.ebuf[b], new.ebuf[b]), (rank, t, b, "E")
        PU.log(f"  noalloc rank {rank} {shapes[0]}: step {t} bitwise equal")
    ref.acp.close()
    new.acp.close()


def test_noalloc_matches_compress_calls_in_a_row():
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible")
    for k, (rank, shapes) in enumerate(CASES):
        _run_case(rank, shapes, seed=11 + k)
