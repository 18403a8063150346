"""libsfl: the ReLU-sparse FFN layer of arXiv 2603.23198 on MI355X (gfx950).

The compute lives in hand-written HIP kernels behind the C ABI in include/sfl.h
(built into libsfl.so by `paper_2603_23198_amd.build`); `paper_2603_23198_amd.binding`
is the ctypes binding with the same function names. Importing the binding fails
if the library is missing: there is no CPU fallback.
"""
