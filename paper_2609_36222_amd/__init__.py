"""BASE decode hot path on MI355X (gfx950): hand-written HIP kernels behind a
C ABI (include/base.h), with a thin ctypes binding (``binding``)."""
