"""Batch-1 decode step of a dense decoder on MI355X (gfx950).

The compute path is ``libaio.so`` (hand-written HIP kernels behind the C ABI in
``include/aio.h``); ``binding`` marshals torch device tensors into it.
"""
