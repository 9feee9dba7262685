"""MI355X-native MoNe test-time-learning hot path (HIP kernels behind a C-ABI library).

Importing the package loads nothing native; ``paper_2608_17616_amd.mone`` binds the library.
"""
