"""MI355X-native hot path of memory-based TGNN training (DepTGL's per-worker step).

The compute lives in libmtgnn.so (HIP kernels for gfx950 behind a C ABI,
``include/mtgnn.h``).  ``mtgnn`` is its ctypes binding and ``step`` drives one
training step through it.  Import those submodules explicitly; importing the
package itself loads nothing.
"""
