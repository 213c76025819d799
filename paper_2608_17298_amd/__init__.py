"""3DGART hot path on MI355X: ray-traced 3D Gaussian forward trace and the
primitive-centric (tile, primitive)-pair gather backward, as HIP kernels for
gfx950 behind a C ABI.

``scenes`` generates seeded synthetic inputs (numpy only).  ``gart`` is the
thin Python binding of the C ABI (``include/gart.h``); it is imported
explicitly so that importing this package never touches the GPU.
"""
__all__ = ["scenes"]
