"""libnnconv: mixed-precision 2-D convolution (forward, backward-data,
backward-weight) for MI355X / gfx950, behind a C ABI.

Importing the package loads nothing; ``paper_2102_06725_amd.nnconv`` is the
binding to the HIP library and ``paper_2102_06725_amd.inputs`` the seeded
synthetic-input generator.
"""
