"""MI355X-native SSP/ESSP matrix-factorization SGD sweep (arXiv 1410.8043).

``paper_1410_8043_amd.ps_mf`` is the Python binding of the C-ABI library
``libps_mf.so`` (HIP kernels for gfx950); ``paper_1410_8043_amd.synth`` generates the
seeded synthetic workloads.
"""
