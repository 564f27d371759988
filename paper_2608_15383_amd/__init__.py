"""MI355X (gfx950) fused W4A16 routed-expert MoE layer (ExactMoE's hot path).

The compute lives in libexactmoe.so (HIP kernels + C ABI, include/exactmoe.h);
`api` is its thin Python binding.  Build with
`python -m paper_2608_15383_amd.build`.
"""
from . import api  # noqa: F401
