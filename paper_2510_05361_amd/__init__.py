"""MT-DAO optimizer hot path on MI355X (gfx950).

``mtdao`` is the ctypes binding of the C ABI declared in include/mtdao.h
(libmtdao.so, built by ``python -m paper_2510_05361_amd.build``);
``optimizer.MtdaoOptimizer`` holds torch-allocated state buffers for it.
Importing the package loads nothing; the library is loaded on first use and
its absence is an error.
"""
