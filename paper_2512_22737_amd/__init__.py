"""WeDLM streaming parallel-decode step on MI355X (gfx950).

The compute lives in libwedlm.so (hand-written HIP kernels behind a C ABI,
declared in include/wedlm.h).  `paper_2512_22737_amd.wedlm` is the thin
Python binding; importing the package itself loads nothing."""
