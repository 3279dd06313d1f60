"""ABFT-protected multi-head attention (EEC-ABFT) on AMD MI355X.

The compute path is the HIP library libattn_abft.so (include/attn_abft.h);
`paper_2410_11720_amd.abft` is its ctypes binding. Importing the binding
raises if the library has not been built.
"""
