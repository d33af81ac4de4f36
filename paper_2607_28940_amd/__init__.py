"""TransX amortized serving path on MI355X (gfx950).

  paper_2607_28940_amd.transx  ctypes binding of libtransx.so (the HIP path)
  paper_2607_28940_amd.inputs  seeded synthetic inputs and weights
  paper_2607_28940_amd.build   compiles the HIP library

Submodules are imported on use so that the input generator can be used
without loading the HIP library.
"""
