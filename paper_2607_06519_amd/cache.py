"""Device-side plumbing around the C ABI: a compressed cache held in torch
device memory (buffer, segment offsets, head modes, sequence lengths) with
thin methods that queue the library calls.  All arithmetic of the method
runs in the library's kernels.
"""
from __future__ import annotations

import math
from typing import Optional, Sequence

import numpy as np

from . import binding as B


def _torch():
    import torch
    if not torch.cuda.is_available():
        raise RuntimeError("a ROCm GPU is required for the compressed-KV path")
    return torch


def torch_dtype(dtype: str):
    torch = _torch()
    # inputs, queries and outputs: FP8-coefficient caches take bf16 tensors
    return {"bf16": torch.bfloat16, "bf16_e4m3": torch.bfloat16, "f32": torch.float32}[dtype]


def to_device(x: np.ndarray, dtype: str, device="cuda"):
    """float32 numpy values (exactly representable in ``dtype``) -> device tensor."""
    torch = _torch()
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(device=device).to(torch_dtype(dtype))


class CompressedCache:
    """One compressed cache: ``batch`` sequences, modes ``[batch][n_blocks][Hkv]``."""

    def __init__(self, dims: B.Dims, seq_lens: Sequence[int], modes: np.ndarray, device="cuda"):
        torch = _torch()
        self.dims = dims
        self.seq_lens_host = [int(t) for t in seq_lens]
        self.batch = len(self.seq_lens_host)
        self.max_seq_len = max(self.seq_lens_host) if self.seq_lens_host else 0
        self.block_first, self.block_size = B.blocks(dims)
        m = np.ascontiguousarray(modes, dtype=np.uint8).reshape(self.batch, len(self.block_size), dims.n_kv_heads)
        self.modes_host = m
        self.offsets_host, self.total_bytes = B.layout(dims, self.seq_lens_host, m)
        self.buf = torch.empty(max(self.total_bytes, 256), dtype=torch.uint8, device=device)
        self.offsets = torch.from_numpy(self.offsets_host.astype(np.int64)).to(device)
        self.modes = torch.from_numpy(m).to(device)
        self.seq_lens = torch.tensor(self.seq_lens_host, dtype=torch.int32, device=device)
        self.ws = torch.empty(B.decode_workspace(dims, self.batch, self.max_seq_len) // 4 + 64,
                              dtype=torch.float32, device=device)

    def compress(self, seq: int, k_layers, v_layers, stream=None):
        """Write sequence ``seq`` from per-layer device tensors ``[Hkv][T][d]``."""
        B.compress(self.dims, self.seq_lens_host[seq], k_layers, v_layers, self.modes[seq],
                   self.offsets[seq], self.buf, stream)

    def decode(self, layer: int, q, out=None, sm_scale: Optional[float] = None, stream=None):
        """One decode step of ``layer`` for queries ``q [batch][Hq][d]``; returns ``out``."""
        torch = _torch()
        if out is None:
            out = torch.empty_like(q)
        scale = 1.0 / math.sqrt(self.dims.head_dim) if sm_scale is None else sm_scale
        B.decode_attn(self.dims, self.batch, self.seq_lens, self.max_seq_len, self.modes, self.offsets,
                      self.buf, layer, q, out, scale, self.ws, stream)
        return out

    def host_bytes(self) -> np.ndarray:
        return self.buf[: self.total_bytes].cpu().numpy()


def probe(dims: B.Dims, seq_len: int, k_layers, qp_layers, n_probe: int, stream=None):
    """Queue fdkv_probe and return the device tensor of errors ``[n_blocks][Hkv][2]``."""
    torch = _torch()
    dev = k_layers[0].device
    ws = torch.empty(B.probe_workspace(dims, seq_len, n_probe), dtype=torch.uint8, device=dev)
    err = torch.empty((len(B.blocks(dims)[0]), dims.n_kv_heads, 2), dtype=torch.float32, device=dev)
    B.probe(dims, seq_len, k_layers, qp_layers, n_probe, err, ws, stream)
    return err, ws
