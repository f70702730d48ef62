"""MI355X-native UniSVQ inference path (2-bit affine-lattice GEMV / GEMM).

The compute lives in ``libunisvq.so`` (HIP kernels for gfx950 behind a C ABI,
declared in ``include/unisvq.h``); ``paper_2606_10520_amd.unisvq`` is the thin
ctypes binding.  Importing this package does not load the library; the first
call into the binding does, and raises if it is missing.
"""
