"""GRACE wide-beam decode attention on MI355X (gfx950).

The compute lives in the HIP library ``libgrace.so`` behind a C ABI
(``include/grace.h``); :mod:`paper_2608_00938_amd.grace` is the thin Python
binding and :mod:`paper_2608_00938_amd.workloads` the seeded input generators.
Importing this package loads nothing: the library is opened on first use and a
missing build raises an error there.
"""
