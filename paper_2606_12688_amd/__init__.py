"""MI355X-native batched paged-KV attention with per-request segment masks.

The computation lives in ``libmstar_attn.so`` (HIP kernels for gfx950 and a
host planner behind the C-ABI in ``include/mstar_attn.h``); ``attn`` is its
Python binding.  Build with ``python -m paper_2606_12688_amd.build``.
"""

__all__ = ["attn", "build"]
