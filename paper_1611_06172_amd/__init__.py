"""HogBatch skip-gram negative-sampling SGD on MI355X (gfx950).

The compute path lives in the HIP library libw2v.so (C ABI declared in
include/w2v.h); `paper_1611_06172_amd.w2v` is its thin ctypes binding and
`paper_1611_06172_amd.inputs` holds the seeded synthetic-input generators.
Importing the package loads nothing; the binding loads the library on first
use and raises if it is missing.
"""
__all__ = ["w2v", "inputs"]
