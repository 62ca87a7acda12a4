"""Batch-Max P&D KV-cache-compressed attention for MI355X (gfx950).

Importing the package loads nothing native; ``paper_2412_05693_amd.batchmax``
loads the HIP library ``libbatchmax.so`` and fails loudly when it is missing.
"""
__all__ = ["synth", "batchmax"]
