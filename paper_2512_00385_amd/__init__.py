"""MI355X-native EZ-SP partition step: exact kNN graph plus the parallel
merge ladder of arXiv 2512.00385, as hand-written HIP kernels for gfx950
behind a C ABI (``include/ezsp.h``).  ``ezsp`` is the thin Python binding."""
