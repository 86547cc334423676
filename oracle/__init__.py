"""CPU oracles of the selective-SSM mixer shard and what is built around it.

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the benchmark's
CPU-baseline leg, never by the GPU product path. ``mixer`` is the float64 Mamba-1 mixer
oracle; ``naive`` is an independent pure-Python per-token loop that pins it (and the
other oracles) on tiny shapes; ``codec`` is the quantized exchange, ``mamba2`` the
Mamba-2 (SSD) mixer and ``layer`` the residual stream, the norms and stacks of layers.
"""
