"""MI355X-native DISCO spherical convolution (forward and transposed).

The compute path lives in ``libdisco.so`` (HIP kernels for gfx950 behind a
C ABI declared in ``include/disco.h``).  ``paper_2209_13603_amd.disco`` is the
thin ctypes binding; ``paper_2209_13603_amd.synth`` holds the seeded workload
inputs.  The library is loaded on first use and a missing or unbuilt library
raises immediately: there is no CPU fallback.
"""
__all__ = ["disco", "synth"]
