"""Test infrastructure: the CPU oracle for the SFC-CA GEMM.

Only the tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import anything from here.  The product path (the HIP
library and its Python binding) never does; this package in turn imports
nothing from the product.
"""
