"""libkf355: MI355X (gfx950) HIP kernels for the memory-bound segmented
reductions Kernel Forge specialises -- row softmax, GroupNorm and
adaptive_avgpool2d -- behind a C ABI, with a thin ctypes binding."""
