"""MI355X-native tree verification for speculative decoding (Dovetail,
arXiv 2412.18934): HIP kernels behind a C ABI (include/dv.h) and a thin
ctypes binding (``dv``).  ``device`` holds the torch-side memory plumbing."""
