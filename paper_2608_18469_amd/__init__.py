"""MI355X-native detached-block training step (ERASE early backward).

Importing the package loads nothing native; ``paper_2608_18469_amd.erase``
loads the HIP library and raises if it has not been built.
"""
__all__ = ["erase", "synth"]
