"""Selective-SSM (Mamba) mixer on one tensor-parallel channel shard, native to MI355X (gfx950).

The compute lives in a C-ABI shared library of hand-written HIP kernels
(``csrc/``, declared in ``include/ssm_shard.h``); ``binding`` marshals torch tensors
into it. ``synth`` draws the seeded synthetic inputs.
"""
__all__ = ["synth"]
