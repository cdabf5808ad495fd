"""MI355X-native (gfx950) training step of synchronous data-parallel SGD, after
"User-transparent Distributed TensorFlow" (arXiv 1704.04560).

The computation lives in libmtx.so (HIP kernels behind the C ABI of include/mtx.h);
``paper_1704_04560_amd.mtx`` is its ctypes binding and ``paper_1704_04560_amd.workloads`` holds
the seeded synthetic workloads.  Importing the package loads nothing; importing ``.mtx`` and
calling it loads the library and fails loudly if it is not built.
"""
