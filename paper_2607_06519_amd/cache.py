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

    def compress(self, seq: int, k_layers, v_layers, stream=None, token_scores=None, k_select=None):
        """Write sequence ``seq`` from per-layer device tensors ``[Hkv][T][d]`` (``token_scores``
        from the probe when residual heads hold a token-level set; ``k_select`` the probe's K
        selections of the same keys, reused instead of selecting again)."""
        B.compress(self.dims, self.seq_lens_host[seq], k_layers, v_layers, self.modes[seq],
                   self.offsets[seq], self.buf, stream, token_scores, k_select)

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
    """Queue fdkv_probe and return the device tensor of errors ``[n_blocks][Hkv][n_err]`` and what
    compress of the same keys takes from the probe: for a token-level residual set the token
    scores ``[n_blocks][Hkv][T]``, otherwise the K selections of the pairs."""
    torch = _torch()
    dev = k_layers[0].device
    ws = torch.empty(B.probe_workspace(dims, seq_len, n_probe), dtype=torch.uint8, device=dev)
    nb = len(B.blocks(dims)[0])
    err = torch.empty((nb, dims.n_kv_heads, dims.n_err), dtype=torch.float32, device=dev)
    scores, ksel = None, None
    if dims.residual == B.RES_TOKENS:
        scores = torch.empty((nb, dims.n_kv_heads, seq_len), dtype=torch.float32, device=dev)
    else:
        ksel = torch.empty(max(B.selection_bytes(dims, seq_len), 1), dtype=torch.uint8, device=dev)
    B.probe(dims, seq_len, k_layers, qp_layers, n_probe, err, ws, stream, scores, ksel)
    return err, (scores if scores is not None else ksel)


class Generation:
    """A compressed cache being extended by decoding (the end of Section 3's
    method): compressed spans (prefill first) followed by an exact tail of
    ``tail_cap`` rows per (sequence, KV head) and layer, which ``refresh``
    compresses into a new span with freshly probed and routed modes.

    A decode step of one token, layer by layer: ``append(layer, k, v)`` puts
    the token's K / V rows at the tail's next row, ``decode(layer, q)``
    attends over every span and the tail including that row; ``advance()``
    then moves the tail position once for all layers.
    """

    def __init__(self, dims: B.Dims, prefix: "CompressedCache", tail_cap: int, device="cuda"):
        torch = _torch()
        self.dims = dims
        self.batch = prefix.batch
        self.spans = [prefix]
        self.cap = int(tail_cap)
        tdt = torch_dtype({B.F32: "f32", B.BF16: "bf16", B.BF16_E4M3: "bf16_e4m3"}[dims.dtype])
        shape = (self.batch, dims.n_kv_heads, self.cap, dims.head_dim)
        self.tail_k = [torch.zeros(shape, dtype=tdt, device=device) for _ in range(dims.n_layers)]
        self.tail_v = [torch.zeros(shape, dtype=tdt, device=device) for _ in range(dims.n_layers)]
        self.n_tail = 0                                     # rows held before the current step
        self.pos = torch.zeros(self.batch, dtype=torch.int32, device=device)      # row the step writes
        self.lens = torch.zeros(self.batch, dtype=torch.int32, device=device)     # rows the step attends
        self._ws = None
        self._refresh_ws()
        self._begin_step()

    def _refresh_ws(self):
        torch = _torch()
        n = B.decode_spans_workspace(self.dims, self.batch, [s.max_seq_len for s in self.spans], self.cap)
        self._ws = torch.empty(n // 4 + 64, dtype=torch.float32, device=self.pos.device)
        self._span_desc = [B.Span(int(s.seq_lens.data_ptr()), s.max_seq_len, int(s.modes.data_ptr()),
                                  int(s.offsets.data_ptr()), int(s.buf.data_ptr())) for s in self.spans]

    def _begin_step(self):
        self.pos.fill_(self.n_tail)
        self.lens.fill_(self.n_tail + 1)

    @property
    def full(self) -> bool:
        return self.n_tail >= self.cap

    def append(self, layer: int, k_new, v_new, stream=None):
        """This step's K / V rows ``[batch][Hkv][d]`` of ``layer`` into the tail."""
        if self.full:
            raise RuntimeError("the tail is full: refresh before appending")
        B.append(self.dims, self.batch, self.pos, self.cap, k_new, v_new, self.tail_k[layer], self.tail_v[layer],
                 stream)

    def decode(self, layer: int, q, out=None, sm_scale: Optional[float] = None, stream=None):
        torch = _torch()
        if out is None:
            out = torch.empty_like(q)
        scale = 1.0 / math.sqrt(self.dims.head_dim) if sm_scale is None else sm_scale
        tail = B.Tail(int(self.lens.data_ptr()), self.cap, int(self.tail_k[layer].data_ptr()),
                      int(self.tail_v[layer].data_ptr()))
        B.decode_spans(self.dims, self.batch, self._span_desc, tail, layer, q, out, scale, self._ws, stream)
        return out

    def advance(self):
        """End of a decode step: the appended rows become part of the tail."""
        self.n_tail += 1
        if not self.full:
            self._begin_step()

    def refresh(self, probe_rows, n_probe: int, lam: float = 0.0, budget_bytes: int = 0):
        """Compress the full tail into a new span.  ``probe_rows[l]`` holds the most
        recent decode queries of layer ``l`` as ``[batch][Hq][n_probe][d]``; each
        sequence's span is probed on its own tail keys and routed with ``lam`` (or
        ``budget_bytes`` per sequence).  Returns the new span's modes."""
        torch = _torch()
        nb = len(B.blocks(self.dims)[0])
        T = self.n_tail
        modes = np.zeros((self.batch, nb, self.dims.n_kv_heads), dtype=np.uint8)
        scores = []
        for s in range(self.batch):
            kl = [self.tail_k[l][s, :, :T] if T < self.cap else self.tail_k[l][s] for l in range(self.dims.n_layers)]
            kl = [t.contiguous() for t in kl]
            ql = [probe_rows[l][s].contiguous() for l in range(self.dims.n_layers)]
            err, extra = probe(self.dims, T, kl, ql, n_probe)
            scores.append(extra)
            modes[s], _, _ = B.route(self.dims, T, err.cpu().numpy(), lam=lam, budget_bytes=budget_bytes,
                                     allow_infeasible=True)
        span = CompressedCache(self.dims, [T] * self.batch, modes, device=self.pos.device)
        for s in range(self.batch):
            kl = [self.tail_k[l][s, :, :T].contiguous() for l in range(self.dims.n_layers)]
            vl = [self.tail_v[l][s, :, :T].contiguous() for l in range(self.dims.n_layers)]
            if self.dims.residual == B.RES_TOKENS:
                span.compress(s, kl, vl, token_scores=scores[s])
            else:
                span.compress(s, kl, vl, k_select=scores[s])
        torch.cuda.synchronize()
        self.spans.append(span)
        self.n_tail = 0
        self._refresh_ws()
        self._begin_step()
        return modes
