"""Cached causal Conv3D for AMD Instinct MI355X (gfx950).

The compute path is the HIP library ``libc3c`` (``csrc/``), reached through
the thin ctypes binding in :mod:`paper_2609_31938_amd.c3c`.  Importing the
package itself loads nothing; importing ``c3c`` loads the built library and
fails loudly when it is missing.
"""
__all__ = ["c3c", "inputs"]
__version__ = "0.1.0"
