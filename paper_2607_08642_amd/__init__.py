"""MI355X-native DominoTree draft-tree builder (HIP for gfx950 behind a C-ABI).

Importing the package loads nothing native; ``paper_2607_08642_amd.binding``
loads ``libdominotree.so`` on first use and fails loudly if it is missing.
"""
__all__ = ["synth", "binding"]
