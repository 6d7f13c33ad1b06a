"""Miriam elastic kernels and co-scheduling runtime for AMD Instinct MI355X (gfx950).

Importing the package loads nothing; ``paper_2307_04339_amd.ops`` and
``paper_2307_04339_amd.runtime`` load ``libmiriam.so`` on first use and fail
loudly if it has not been built.
"""
__all__ = ["ops", "runtime", "models", "synth"]
