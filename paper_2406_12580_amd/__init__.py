"""MI355X-native BD-LRU scan (RecBLR, arXiv 2406.12580).

The compute path is the HIP library ``librecblr.so`` built from ``csrc/`` for
gfx950; ``paper_2406_12580_amd.recblr`` is its thin ctypes binding.  Importing
the package itself loads nothing, so the seeded input generator
(``paper_2406_12580_amd.datagen``) can be used without a GPU.
"""
