"""MI355X-native mixed chunked-prefill + decode attention over a paged KV cache.

The hot path of one serving iteration shaped by SlidingServe's scheduler (a
batch B = {(c_i, u_i)} of chunk and decode requests, Sec. 3.2), executed by
hand-written gfx950 HIP kernels behind the C ABI of ``include/ssa.h``.

Modules:
  ssa       ctypes binding of libssa.so (the C names)
  device    a batch resident on the GPU with its plan, output and workspace
  workload  seeded synthetic batches shaped like the paper's workloads
  build     compiles libssa.so in-tree for gfx950
"""
__all__ = ["ssa", "device", "workload", "build"]
