"""Exact solver for the Minimum Prefix Trie with Free Permutations (MPT)
problem on MI355X (gfx950).

The solver is the O(3^m) exact algorithm of the structure theorem
(Section 3.1): a superset-zeta transform builds W(B) = w(I(B)) for every
request subset B, a popcount-layered subset-min DP over all bipartitions
keeps the argmin splits, and the per-request chunk orders are read back
top-down from the resulting hierarchy (proof of Theorem 1, the "<=" half).

Every step runs in the HIP kernels of ``libmpt.so`` behind the C ABI
declared in ``include/mpt.h``; :mod:`.mpt` is the ctypes binding. Importing
this package loads nothing: the binding loads the library on first use and
raises if it is missing.
"""
__version__ = "0.1.0"
