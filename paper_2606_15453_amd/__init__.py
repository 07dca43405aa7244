"""MI355X-native decode-step MoE layer with spatio-temporal expert prefetching.

Importing the package loads nothing native; ``paper_2606_15453_amd.stmoe``
loads the HIP library and raises if it has not been built.
"""
__all__ = ["workload", "stmoe"]
