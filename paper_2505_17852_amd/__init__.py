"""MI355X (gfx950) implementation of one CD-RGE training step for stacked-LSTM
language models: HIP kernels behind the C ABI in include/zo.h, with a thin
ctypes binding (``zo``) and seeded synthetic workloads (``workloads``)."""
