"""HetPipe's data-parallel hot path on MI355X (gfx950).

One pipeline stage's CNN training step (implicit-GEMM convolutions and FC
layers on MFMA, batch-norm, ReLU, pooling, softmax cross-entropy) and the Wave
Synchronous Parallel weight update (local update, wave accumulation, push and
pull against a parameter server in device memory), behind the C ABI of
include/hetpipe.h.  ``hetpipe`` is the ctypes binding, ``nets`` the stage
layer lists, ``workloads`` the five configurations and ``driver`` the
simulation of several virtual workers on one GPU.
"""
