"""MI355X-native SSD (structured state space duality) layer forward.

The product is the C-ABI library ``libssd_hip.so`` (header ``include/ssd.h``)
built from the HIP sources in ``csrc/``; :mod:`paper_2405_21060_amd.ssd` is
its Python binding and :mod:`paper_2405_21060_amd.inputs` draws the seeded
synthetic workloads.  Nothing is loaded at import time.
"""
__all__ = ["ssd", "inputs", "build"]
