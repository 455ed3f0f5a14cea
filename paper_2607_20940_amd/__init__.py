"""MI355X-native Multi-Scale Self-Attention (Ms. Forcing, Sec. 4.1).

``paper_2607_20940_amd.mssa`` is the ctypes binding of the C-ABI library
``libmssa.so`` (HIP kernels for gfx950).  Importing the package itself loads
nothing; importing ``.mssa`` loads the library and fails loudly if it is
missing.
"""
__all__ = ["inputs", "workloads", "mssa"]
