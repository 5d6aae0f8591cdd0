"""ZO-Act forward-only step on MI355X (gfx950): HIP kernels behind a C ABI.

`paper_2607_01125_amd.zoact` is the ctypes binding of libzoact.so (include/zoact.h);
`paper_2607_01125_amd.model` assembles decoder models from those calls.
"""
