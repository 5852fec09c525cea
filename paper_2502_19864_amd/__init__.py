"""RingAda per-stage hot path for AMD Instinct MI355X (gfx950).

The compute lives in ``libringada.so`` (hand-written HIP kernels behind a
C ABI declared in ``include/ringada.h``); ``binding`` marshals arguments to it.
Importing this package does not load the library: ``binding.lib()`` does, and
fails loudly if it has not been built.
"""
