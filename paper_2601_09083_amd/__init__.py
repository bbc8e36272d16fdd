"""SRT tree-speculative verification step on AMD Instinct MI355X (gfx950).

The work is done by hand-written HIP kernels behind the C ABI of
``include/srt.h`` (libsrt.so, built by ``paper_2601_09083_amd.build``).
``paper_2601_09083_amd.srt`` is the thin Python binding (same names as the C
entry points); ``paper_2601_09083_amd.workload`` draws the seeded synthetic
inputs.  Importing the package loads nothing: the library is loaded on the
first binding call and its absence is an error, never a fallback.
"""
__all__ = ["srt", "workload", "build"]
