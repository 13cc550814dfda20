"""MI355X-native SparCML hot path (arXiv 1802.08021).

``paper_1802_08021_amd.sparcml`` is the Python binding of the C-ABI library
``libsparcml.so`` (HIP kernels for gfx950); ``paper_1802_08021_amd.inputs``
draws the seeded synthetic workloads.
"""
