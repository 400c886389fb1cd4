"""Rollback-free GDN draft-tree verification on AMD Instinct MI355X (gfx950).

The compute path lives in the HIP library ``libgdntree.so`` (C ABI in
include/gdn_tree.h); ``gdn_tree`` is its Python binding and ``workloads``
generates seeded synthetic trees.  Submodules are imported explicitly so that
input generation works on machines without a GPU."""
__all__ = ["gdn_tree", "workloads"]
