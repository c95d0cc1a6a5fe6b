"""MI355X-native in-place KV-cache splice (Leyline hot path): HIP kernels behind a C ABI.

``paper_2606_01065_amd.leyline`` is the ctypes binding of ``libleyline.so``; importing it fails
when the library has not been built (``python -m paper_2606_01065_amd.build``).
"""
