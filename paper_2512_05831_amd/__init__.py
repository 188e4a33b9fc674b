"""Embedding Bag forward (arXiv 2512.05831) for AMD Instinct MI355X.

``eb``        -- binding of the C ABI in include/eb.h (libeb.so, HIP / gfx950).
``workloads`` -- seeded synthetic inputs (tables, lengths, offsets, indices).
``build``     -- compiles libeb.so in tree.
"""
