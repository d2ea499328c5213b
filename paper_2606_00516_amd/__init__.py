"""MI355X-native decoder-layer step for exclusive / mixed batching.

The compute path is the HIP library ``libeb.so`` (C ABI declared in
``include/eb_layer.h``); ``paper_2606_00516_amd.binding`` marshals torch
tensors into it.  ``paper_2606_00516_amd.inputs`` draws seeded synthetic
workloads.  Importing the package loads nothing native; the binding loads the
library on first use and raises if it is missing.
"""
__all__ = ["inputs", "binding"]
