"""ATP chunked 2D tensor-parallel shard block for AMD MI355X (gfx950).

One device's share of a transformer layer under ATP's row-first /
column-first 2D tensor parallelism (arXiv 2301.08658): sharded QKV,
out-proj, fc1 (+bias+GeLU) and fc2 bf16 MFMA GEMMs, the Partial(SUM)
reduction, and a two-stream token-chunk pipeline.  The work runs in
``libatp.so`` (hand-written HIP for gfx950, C ABI in ``include/atp.h``);
this package is its ctypes binding.  The library is loaded on first use and
there is no fallback path: without ``libatp.so`` every call raises.
"""
from .binding import *  # noqa: F401,F403
from .binding import load_library, AtpError, HipEvent, LIB_PATH, EXPORTS  # noqa: F401
from .binding import Hcm, hcm_mi355x_xgmi, model_dims  # noqa: F401

__all__ = [n for n in dir() if n.startswith(("atp_", "ATP_"))] + [
    "load_library", "AtpError", "HipEvent", "LIB_PATH", "EXPORTS", "mesh", "block_geometry",
    "attention_heads",
    "Hcm", "hcm_mi355x_xgmi", "model_dims"]
