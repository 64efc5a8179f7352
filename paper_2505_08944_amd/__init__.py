"""MI355X (gfx950) expert-layer hot path of Asynchronous Expert Parallelism.

mu-queue append (router), re-batch/gather, grouped SwiGLU expert FFN and
top-K combine run in libaep (HIP kernels behind a C ABI, include/aep.h);
this package only marshals torch tensors and streams into that ABI.
"""

from ._lib import AEPError, LIB_PATH  # noqa: F401
from .context import BatchView, Context, fp8_e4m3_to_bf16  # noqa: F401

__all__ = ["Context", "BatchView", "AEPError", "fp8_e4m3_to_bf16", "LIB_PATH"]
