"""MI355X-native space-filling-curve, communication-avoiding bf16 GEMM.

``paper_2601_16294_amd.sfcgemm`` is the Python binding of the C-ABI library
``libsfcgemm.so`` (HIP kernels for gfx950); ``paper_2601_16294_amd.inputs``
holds the seeded synthetic workloads.  Importing this package loads neither.
"""
