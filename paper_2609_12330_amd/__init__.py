"""MI355X (gfx950) split-KV online-softmax attention.

The compute path is the HIP library ``libef_attention.so`` built from
``csrc/``; :mod:`paper_2609_12330_amd.ef_attention` is its thin ctypes
binding. Importing this package loads nothing; the binding loads the library
on first use and raises if it is missing.
"""

__all__ = ["workloads", "ef_attention"]
