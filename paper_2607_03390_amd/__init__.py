"""TemporalGS hot path on MI355X: HIP kernels behind a C-ABI (``libtgs.so``).

``tgs`` is the ctypes binding; ``synth`` draws the seeded synthetic inputs.
The binding is imported lazily so that input generation works without the
built library.
"""
__all__ = ["synth", "tgs"]
