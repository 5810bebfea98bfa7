"""One host's share of APB prefill attention (arXiv 2502.12085) on MI355X.

The product is the gfx950 HIP library ``libapb.so`` behind the C ABI in
``include/apb.h``; ``apb`` is its Python binding and ``inputs`` the seeded
synthetic workloads.  Importing the package loads nothing: the library is
loaded on first use by ``apb.lib()``.
"""
