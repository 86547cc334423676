"""CPU oracle of the selective-SSM mixer shard.

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the benchmark's
CPU-baseline leg, never by the GPU product path. ``mixer`` is the float64 oracle;
``naive`` is an independent pure-Python per-token loop that pins it on tiny shapes.
"""
