"""STaR-KV compression stage on MI355X (gfx950).

The compute path lives in the C-ABI library ``libstarkv.so`` built from
``csrc/``; ``starkv`` is its thin ctypes binding.  ``workload`` draws the
seeded synthetic inputs.  Importing the package loads nothing native.
"""

__all__ = ["starkv", "workload"]
