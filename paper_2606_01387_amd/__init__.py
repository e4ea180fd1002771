"""Claim-scoped KV materialization checking on MI355X (gfx950).

The checker lives in ``libclaimkv.so`` (HIP kernels behind a C ABI declared in
``include/claimkv.h``); :mod:`paper_2606_01387_amd.claimkv` is its Python
binding.  Importing this package loads nothing: the binding loads the library
on first use and raises if it is missing.
"""
