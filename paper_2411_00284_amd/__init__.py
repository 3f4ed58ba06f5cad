"""MI355X (gfx950) bucketed FSDP copy path of SimpleFSDP (arXiv 2411.00284).

One rank's share of the bucketed all-gather and reduce-scatter path: the
plan, the all-gather copy-in (fp32 -> bf16 cast and pack), the all-gather
copy-out, the reduce-scatter copy-in, and the rank-local fp32 average with
read-out.  The work runs in hand-written HIP kernels behind the C ABI of
``include/fsdp_bucket.h``; this package is the Python binding.  The same
library also cuts a pass's all-gathers into buckets (auto-wrapping, host
code).
"""

from .auto_wrap import auto_wrap
from .bucket import BucketPlan, FsdpError

__all__ = ["BucketPlan", "FsdpError", "auto_wrap"]
