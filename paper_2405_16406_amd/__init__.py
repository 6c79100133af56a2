"""MI355X-native rotated W4A4 inference path of SpinQuant (arXiv 2405.16406).

The compute lives in `libsq.so` (hand-written HIP kernels for gfx950 behind a C ABI,
declared in include/sq.h).  `paper_2405_16406_amd.sq` is the thin ctypes binding: it
only marshals torch tensors into pointers and the current HIP stream.  Submodules are
imported explicitly (`from paper_2405_16406_amd import sq`), so host-only tools (input
generation, the build step) work on machines without the built library; any compute
call without the library raises.
"""
