"""MI355X-native histogram gradient boosting: the per-iteration hot path of
out-of-core GPU gradient boosting (Ou, KDD 2020) as hand-written HIP kernels
for gfx950 behind a C-ABI library (``libgbt.so``).

``paper_2005_09148_amd.gbt`` is the ctypes binding of that library (it fails
loudly when the library is not built); ``paper_2005_09148_amd.datagen`` holds
the seeded synthetic workloads.  Importing the package itself loads nothing.
"""
