"""WaveRNN sampling on MI355X (gfx950): a HIP library behind a C ABI.

``paper_1802_08435_amd.wavernn`` is the Python binding of ``libwavernn.so``;
``paper_1802_08435_amd.synth`` generates seeded synthetic weights and inputs.
Importing the package loads nothing.
"""
