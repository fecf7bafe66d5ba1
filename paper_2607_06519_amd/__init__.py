"""FreqDepthKV compressed-KV path on AMD MI355X (gfx950).

The product is ``libfdkv.so`` (C ABI declared in ``include/fdkv.h``) with its
hand-written HIP kernels under ``csrc/``; ``binding`` marshals torch tensors
and numpy arrays into those calls.
"""
from . import binding  # noqa: F401
from .binding import (BF16, EXACT, F32, RESIDUAL, SHARED, Dims, FdkvError, compress,  # noqa: F401
                      decode_attn, decode_workspace, dims, layout, probe, probe_workspace, route)
