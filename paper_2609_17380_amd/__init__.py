"""canon: one replayed training step in canonical order on MI355X (gfx950).

`canon` is the binding of the HIP library (include/canon.h); `inputs` is the seeded input generator.
"""
