"""Replays of captured steps against eager calls: the all-bucket calls of one odd and one even step
captured into HIP graphs (as `bench.py --mode graph` does) and replayed in turn must give bitwise
the results of calling the library for every step.

A second context runs every step eagerly on the same inputs.  Each step's gradients are written
into the captured input buffers by an eager copy before the replay, and every replay is compared
with the eager step (outputs and factor buffers bitwise; E and the factors after even steps,
where the context's host-side record of the last step's parity, which replays do not advance,
matches the device).  The captured calls enqueue no memset.
"""

import numpy as np
import pytest
import torch

from tests import parity_util as PU
from tests.test_gpu_parity import RAGGED

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("rank", [4, 32])
@pytest.mark.parametrize("ef", [True, False])
def test_captured_steps_replay_like_eager_calls(rank, ef):
    if not torch.cuda.is_available():
        pytest.fail("no GPU visible")
    shapes = RAGGED + [(700, 1024), (96,), (2048, 4096)]
    eager = PU.Runner(shapes, rank, cap=1 << 22, ef=ef, grouped=True)
    capt = PU.Runner(shapes, rank, cap=1 << 22, ef=ef, grouped=True)
    assert eager.nb > 2
    rng = np.random.default_rng(7)

    def grads():
        return {i: (0.02 * rng.standard_normal(s)).astype(np.float32) for i, s in enumerate(shapes)}

    inputs = capt.pack(grads())  # the buffers the graphs read
    for t in (1, 2):
        g = grads()
        for dst, src in zip(inputs, capt.pack(g)):
            dst.copy_(src)
        eager.step(t, eager.pack(g))
        capt.step(t, inputs)
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    graphs = []
    for t in (3, 4):
        gr = torch.cuda.CUDAGraph()
        with torch.cuda.graph(gr, stream=side):
            capt.acp.compress_all(t, inputs, capt.fbuf)
            capt.acp.decompress_all(t, capt.fbuf, capt.out)
        graphs.append(gr)
    torch.cuda.current_stream().wait_stream(side)
    for t in range(3, 13):
        g = grads()
        eager.step(t, eager.pack(g))
        for dst, src in zip(inputs, capt.pack(g)):
            dst.copy_(src)
        graphs[0 if t % 2 else 1].replay()
        torch.cuda.synchronize()
        for b in range(eager.nb):
            assert torch.equal(eager.out[b], capt.out[b]), (t, b, "output")
            assert torch.equal(eager.fbuf[b], capt.fbuf[b]), (t, b, "factor buffer")
        if t % 2 == 0:
            for tid, s in enumerate(shapes):
                if eager.where[tid][4]:
                    assert np.array_equal(eager.ortho(t, tid), capt.ortho(t, tid)), (t, tid)
                    if ef:
                        assert np.array_equal(eager.error_slice(tid), capt.error_slice(tid)), (t, tid)
        PU.log(f"  rank {rank} ef={ef}: replay of step {t} bitwise equal to the eager step")
    eager.acp.close()
    capt.acp.close()
