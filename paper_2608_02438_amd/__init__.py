"""xPress refine + verify hot path for MI355X (gfx950).

The work runs in the HIP kernels of ``libxpress.so`` (C ABI: include/xpress.h);
``xpress`` is its Python binding.  Build with ``python -m paper_2608_02438_amd.build``.
"""
from .xpress import (Refiner, RefineOut, XpError, load_library, refiner_from_arrays,  # noqa: F401
                     device_tensor, bf16_tensor, LIB_PATH, EXPORTS)
