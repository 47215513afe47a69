"""Forced-weight subset evaluation over attention rows on MI355X (gfx950).

The compute path is the HIP library ``libfw.so`` built from ``csrc/``; the
Python binding ``paper_2608_25230_amd.fw`` marshals arguments into it and
nothing else.  Importing this package loads nothing.
"""
__all__ = ["fw", "workloads"]
