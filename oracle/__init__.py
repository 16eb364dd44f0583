"""Plain fp64 CPU oracle for the ACP-SGD compressor (arXiv 2306.08881).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports, calls or
links this package: only the tests, the smoke check and the benchmark's
CPU-baseline leg use it.  It shares no code with the device library; the two
meet only in the seeded input generator ``synthgrad``.

Modules:

* ``layout``  - eligibility, reshape, tensor-fusion buckets and factor-buffer
                offsets (Section IV-B "Tensor Fusion" / "Buffer Size",
                Section IV-C).
* ``rng``     - the counter-based draw of the initial factors P0, Q0
                (Section IV-A, "Error-feedback": i.i.d. standard normal).
* ``gs``      - Gram-Schmidt orthogonalisation (the "Orthogonalize" of
                Algorithms 1 and 2).
* ``acp``     - ACP-SGD with error feedback, step by step (Algorithm 2),
                Power-SGD (Algorithm 1, left) and a k-worker loopback.

Every function is written for clarity, not speed.
"""
