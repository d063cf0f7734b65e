"""MI355X-native interaction-network edge classifier (gfx950 HIP behind a C ABI).

Importing the package loads nothing heavy: the GPU binding lives in
``paper_2402_09633_amd.gnn`` and the seeded generators in
``paper_2402_09633_amd.inputs``.
"""
