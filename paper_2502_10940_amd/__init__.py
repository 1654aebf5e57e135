"""MI355X-native CoLA layer (arXiv 2502.10940): Y = B sigma(A X), forward and
backward, with the CoLA-M recompute mode, as hand-written HIP kernels for
gfx950 behind a C ABI (``include/cola.h``).  ``paper_2502_10940_amd.cola`` is
the thin ctypes binding; ``paper_2502_10940_amd.inputs`` the seeded synthetic
inputs."""
