"""CPU oracle for the summed-area-table box-convolution layer.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path (the HIP library and
its Python binding) may import, call or link anything in this package.  Only
the tests, the smoke check and the CPU-baseline leg of the benchmark use it.

The oracle is a plain, slow, fp64 (int64 for integer data) NumPy restatement
of what the layer computes, written from the paper's definitions (Section 3.1,
Eq. 1-4; Section 3.2) and sharing no code, table or helper with the GPU path.
"""
from .boxconv_oracle import *  # noqa: F401,F403
