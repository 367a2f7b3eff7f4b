"""Tree-structured WY verification of the gated delta rule on MI355X (gfx950).

The compute path is the HIP library ``libtreewy.so`` (``csrc/``), reached
through the thin ctypes binding in ``treewy.py``.  Importing this package
loads nothing; ``paper_2608_20961_amd.treewy`` loads the library and raises if
it has not been built.
"""
