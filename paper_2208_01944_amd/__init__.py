"""PalQuant inference on AMD MI355X (gfx950).

The compute path is the HIP library `libpalq.so` (C ABI in include/palq.h),
reached from Python through `paper_2208_01944_amd.palq`.  Importing this
package loads nothing; `palq` loads the library and fails loudly if it is
missing.
"""
__all__ = ["palq", "inputs"]
