"""MI355X-native Kalman Delta Network hot path (arXiv 2609.07816).

The compute lives in ``libkdn.so`` (HIP kernels for gfx950 behind a C ABI, declared in
``include/kdn.h``). ``paper_2609_07816_amd.kdn`` is the thin ctypes binding; ``workloads`` draws
seeded synthetic inputs.
"""
