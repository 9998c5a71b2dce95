"""LM-operator row evaluation on MI355X (gfx950): the C-ABI library and its binding.

The package's compute path is liblmop.so (HIP kernels + C ABI, built by
`python -m paper_2606_31808_amd.build`); `paper_2606_31808_amd.lmop` is the
ctypes binding.  Importing the binding without the built library raises.
"""
