"""MI355X (gfx950) batch-1 Llama decode megakernel: one cooperative HIP launch per token.

The compute path is libamk.so (HIP kernels + C ABI in include/amk.h); the
binding in ``amk`` only marshals arguments.  Build with
``python -m paper_2606_09682_amd.build``.
"""
from . import amk  # noqa: F401
