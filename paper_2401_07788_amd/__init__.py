"""MI355X (gfx950) boundary compressors: TopK, min-max quantization, error
feedback and AQ-SGD, as a C-ABI HIP library with a thin ctypes binding."""
