"""libesb: the data-parallel hot path of elastic significant bit (ESB) quantization
on AMD MI355X (gfx950).

The product is the C-ABI shared library ``libesb.so`` (declared in
``include/esb.h``, kernels under ``csrc/``).  ``paper_2109_03513_amd.esb`` is a
thin ctypes binding with the same entry-point names; it loads the library on
first use and raises if it is missing.  ``workloads`` holds the seeded
synthetic input generators.
"""
__all__ = ["esb", "workloads"]
