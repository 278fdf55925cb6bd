"""FOCUS scale-learning hot path for MI355X (gfx950).

The compute lives in ``libfocus.so`` (hand-written HIP kernels behind a C ABI, see
``include/focus.h``); ``paper_2608_01847_amd.focus`` is the thin ctypes binding that tests and the
benchmark call. Importing this package loads nothing: the library is opened on first use.
"""
