"""Batched J-DOB policy evaluation on MI355X (gfx950).

The compute path is the C-ABI library ``libjdob.so`` built from
``csrc/jdob.hip``; ``paper_2504_14611_amd.jdob`` is its thin ctypes binding
and ``paper_2504_14611_amd.workloads`` generates seeded synthetic inputs.
Importing the package loads nothing: the binding loads the library on first
use and raises if it is missing.
"""

__all__ = ["jdob", "workloads"]
