"""MI355X-native generalized Allreduce (Kolmakov & Zhang, arXiv:2004.09362).

P virtual ranks live on one GPU; the permutation-group schedule runs as HIP
kernels behind a C-ABI library (``include/ar.h``).  The Python side only
marshals arguments into that library (``paper_2004_09362_amd.ar``).
"""
