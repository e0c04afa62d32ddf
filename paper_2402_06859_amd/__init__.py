"""MI355X (gfx950) Residual-DCN + QR-embedding path of LiRank (arXiv 2402.06859).

librdcn.so (HIP kernels behind the C ABI of include/rdcn.h) does the work;
`rdcn` is its ctypes binding, `synth` draws seeded synthetic inputs and `step`
sequences the calls of one training step on device buffers.
"""
