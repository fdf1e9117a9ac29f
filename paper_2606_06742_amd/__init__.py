"""kmpath: cross-validated regularisation paths of RBF kernel machines on MI355X.

The compute path is the HIP library ``libkmpath.so`` (built in-tree by
``paper_2606_06742_amd.build``); ``paper_2606_06742_amd.kmpath`` is its thin
ctypes binding. Importing this package does not load the library.
"""
__all__ = ["kmpath", "build"]
