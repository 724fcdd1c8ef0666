"""RaBitQCache decode hot path on AMD MI355X (gfx950): HIP kernels behind a C ABI.

`paper_2606_31519_amd.rbq` is the ctypes binding of librbq.so (include/rbq.h);
`paper_2606_31519_amd.pipeline` holds the device buffers of one decode workload
and runs the five calls in order; `paper_2606_31519_amd.build` compiles the
library in-tree.
"""
