"""MI355X-native population decode for verifier-free evolution (Squeeze Evolve).

``sevo``          thin ctypes binding of libsevo.so (the C ABI in include/sevo.h)
``synth``         seeded synthetic inputs (host); ``device_inputs`` on the GPU
``build``         compiles libsevo.so (hipcc, gfx950) and the host generator
Submodules are imported on demand so that the input generator can be used
without loading the HIP library.
"""
__version__ = "0.1.0"
