"""ctypes binding of libfdkv (argument marshalling only).

Each function mirrors one entry point of ``include/fdkv.h`` and takes torch
tensors for device buffers (their ``data_ptr()`` is passed) and numpy arrays
for host buffers.  Work is queued on the current torch stream.  Nothing here
computes any part of the method; a missing library raises ``RuntimeError``.
"""
from __future__ import annotations

import ctypes
import os
from typing import Sequence

import numpy as np

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libfdkv.so")
_lib = None

SHARED, RESIDUAL, EXACT = 0, 1, 2
F32, BF16, BF16_E4M3 = 0, 1, 2   # cache types (fdkv_dtype)

STATUS = {0: "FDKV_OK", -1: "FDKV_E_INVALID_ARG", -2: "FDKV_E_UNSUPPORTED", -3: "FDKV_E_WORKSPACE",
          -4: "FDKV_E_BUDGET", -5: "FDKV_E_HIP"}

SYMBOLS = ("fdkv_status_string", "fdkv_last_error", "fdkv_blocks", "fdkv_layout", "fdkv_route",
           "fdkv_probe_workspace", "fdkv_probe", "fdkv_compress", "fdkv_decode_workspace", "fdkv_decode_attn",
           "fdkv_append", "fdkv_decode_spans_workspace", "fdkv_decode_spans", "fdkv_decode_static_scratch_bytes",
           "fdkv_decode_attn_static", "fdkv_decode_partial", "fdkv_decode_combine", "fdkv_selection_bytes",
           "fdkv_check_conversions")
PAIRS, MIXED, QUADS = 0, 1, 2    # block schedules (fdkv_schedule)
RES_CHANNELS, RES_TOKENS = 0, 1  # residual kinds (fdkv_residual)


class FdkvError(RuntimeError):
    def __init__(self, status: int, where: str):
        lib = load()
        msg = lib.fdkv_status_string(status).decode()
        if status == -5 or (status == -3 and "static" in where):
            msg += ": " + lib.fdkv_last_error().decode()
        super().__init__(f"{where}: {STATUS.get(status, status)} ({msg})")
        self.status = status


class Dims(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("topk", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("schedule", ctypes.c_int32), ("residual", ctypes.c_int32), ("res_ppm", ctypes.c_int32),
                ("n_rates", ctypes.c_int32), ("rates_ppm", ctypes.c_int32 * 8)]

    @property
    def n_err(self) -> int:
        """Columns of the probe's loss array: E_S, then E_R at each candidate fraction."""
        return 1 + (self.n_rates if self.residual == RES_TOKENS and self.n_rates else 1)


class Span(ctypes.Structure):
    _fields_ = [("seq_lens", ctypes.c_void_p), ("max_seq_len", ctypes.c_int32), ("modes", ctypes.c_void_p),
                ("seg_offsets", ctypes.c_void_p), ("cache", ctypes.c_void_p)]


class Tail(ctypes.Structure):
    _fields_ = [("lens", ctypes.c_void_p), ("cap", ctypes.c_int32), ("k", ctypes.c_void_p), ("v", ctypes.c_void_p)]


def dims(n_layers, n_kv_heads, n_q_heads, head_dim, topk, dtype, schedule=PAIRS, residual=RES_CHANNELS,
         res_ppm=0, res_rates=()) -> Dims:
    """``res_rates``: routed candidate fractions (ppm) of token-level sets, at most 8."""
    dt = {"f32": F32, "bf16": BF16, "bf16_e4m3": BF16_E4M3}.get(dtype, dtype)
    rates = list(res_rates) + [0] * (8 - len(res_rates))
    return Dims(n_layers, n_kv_heads, n_q_heads, head_dim, topk, dt, schedule, residual, res_ppm, len(res_rates),
                (ctypes.c_int32 * 8)(*rates))


def load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise RuntimeError(f"{_LIB_PATH} is not built; run __graft_entry__.build() first")
    lib = ctypes.CDLL(_LIB_PATH)
    P, I32, U64, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_uint64, ctypes.c_size_t
    DP = ctypes.POINTER(Dims)
    lib.fdkv_status_string.restype = ctypes.c_char_p
    lib.fdkv_status_string.argtypes = [I32]
    lib.fdkv_last_error.restype = ctypes.c_char_p
    lib.fdkv_last_error.argtypes = []
    lib.fdkv_blocks.restype = I32
    lib.fdkv_blocks.argtypes = [DP, P, P, P]
    lib.fdkv_layout.restype = I32
    lib.fdkv_layout.argtypes = [DP, I32, P, P, P, P]
    lib.fdkv_route.restype = I32
    lib.fdkv_route.argtypes = [DP, I32, P, ctypes.c_double, U64, P, P]
    lib.fdkv_probe_workspace.restype = I32
    lib.fdkv_probe_workspace.argtypes = [DP, I32, I32, P]
    lib.fdkv_probe.restype = I32
    lib.fdkv_probe.argtypes = [DP, I32, P, P, I32, P, P, P, SZ, P, P]
    lib.fdkv_compress.restype = I32
    lib.fdkv_compress.argtypes = [DP, I32, P, P, P, P, P, P, P, P]
    lib.fdkv_selection_bytes.restype = I32
    lib.fdkv_selection_bytes.argtypes = [DP, I32, P]
    lib.fdkv_check_conversions.restype = I32
    lib.fdkv_check_conversions.argtypes = [P, P]
    lib.fdkv_decode_workspace.restype = I32
    lib.fdkv_decode_workspace.argtypes = [DP, I32, I32, P]
    lib.fdkv_decode_attn.restype = I32
    lib.fdkv_decode_attn.argtypes = [DP, I32, P, I32, P, P, P, I32, P, P, ctypes.c_float, P, SZ, P]
    lib.fdkv_decode_static_scratch_bytes.restype = SZ
    lib.fdkv_decode_static_scratch_bytes.argtypes = []
    lib.fdkv_decode_attn_static.restype = I32
    lib.fdkv_decode_attn_static.argtypes = [DP, I32, P, I32, P, P, P, I32, P, P, ctypes.c_float, P]
    lib.fdkv_decode_partial.restype = I32
    lib.fdkv_decode_partial.argtypes = [DP, I32, P, I32, P, P, P, I32, P, ctypes.c_float, P, SZ, P]
    lib.fdkv_decode_combine.restype = I32
    lib.fdkv_decode_combine.argtypes = [DP, I32, I32, P, P, SZ, P]
    lib.fdkv_append.restype = I32
    lib.fdkv_append.argtypes = [DP, I32, P, I32, P, P, P, P, P]
    lib.fdkv_decode_spans_workspace.restype = I32
    lib.fdkv_decode_spans_workspace.argtypes = [DP, I32, I32, P, I32, P]
    lib.fdkv_decode_spans.restype = I32
    lib.fdkv_decode_spans.argtypes = [DP, I32, I32, P, P, I32, P, P, ctypes.c_float, P, SZ, P]
    _lib = lib
    return lib


def _check(st: int, where: str):
    if st != 0:
        raise FdkvError(st, where)


def _np_ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _dev(t) -> int:
    return 0 if t is None else int(t.data_ptr())


def _stream(stream=None):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(int(s.cuda_stream))


def _ptr_array(tensors: Sequence) -> ctypes.Array:
    arr = (ctypes.c_void_p * len(tensors))()
    for i, t in enumerate(tensors):
        arr[i] = _dev(t)
    return arr


# ----------------------------------------------------------------- host entry points
def blocks(d: Dims):
    """``(first_layer [n_blocks] int32, block_size [n_blocks] int32)`` of the schedule."""
    lib = load()
    n = ctypes.c_int32(0)
    _check(lib.fdkv_blocks(ctypes.byref(d), ctypes.byref(n), None, None), "fdkv_blocks")
    first = np.zeros(n.value, dtype=np.int32)
    size = np.zeros(n.value, dtype=np.int32)
    _check(lib.fdkv_blocks(ctypes.byref(d), ctypes.byref(n), _np_ptr(first), _np_ptr(size)), "fdkv_blocks")
    return first, size


def layout(d: Dims, seq_lens, modes):
    """``(seg_offsets [batch][n_blocks][Hkv] uint64, total_bytes)`` for host ``modes``."""
    lib = load()
    sl = np.ascontiguousarray(seq_lens, dtype=np.int32)
    m = np.ascontiguousarray(modes, dtype=np.uint8)
    off = np.zeros(m.shape, dtype=np.uint64)
    total = ctypes.c_uint64(0)
    _check(lib.fdkv_layout(ctypes.byref(d), int(sl.size), _np_ptr(sl), _np_ptr(m), _np_ptr(off),
                           ctypes.byref(total)), "fdkv_layout")
    return off, int(total.value)


def route(d: Dims, seq_len: int, errors, lam: float = 0.0, budget_bytes: int = 0, allow_infeasible=False):
    """``(modes [n_blocks][Hkv] uint8, lambda_used, status)`` from host ``errors [n_blocks][Hkv][n_err]``
    (the mode bytes carry the routed fraction index of residual units in bits 2-4)."""
    lib = load()
    e = np.ascontiguousarray(errors, dtype=np.float32)
    modes = np.zeros(e.shape[:-1], dtype=np.uint8)
    lam_out = ctypes.c_double(0.0)
    st = lib.fdkv_route(ctypes.byref(d), int(seq_len), _np_ptr(e), float(lam), int(budget_bytes),
                        _np_ptr(modes), ctypes.byref(lam_out))
    if not (st == 0 or (st == -4 and allow_infeasible)):
        _check(st, "fdkv_route")
    return modes, float(lam_out.value), st


def probe_workspace(d: Dims, seq_len: int, n_probe: int) -> int:
    n = ctypes.c_size_t(0)
    _check(load().fdkv_probe_workspace(ctypes.byref(d), int(seq_len), int(n_probe), ctypes.byref(n)),
           "fdkv_probe_workspace")
    return int(n.value)


def selection_bytes(d: Dims, seq_len: int) -> int:
    n = ctypes.c_size_t(0)
    _check(load().fdkv_selection_bytes(ctypes.byref(d), int(seq_len), ctypes.byref(n)), "fdkv_selection_bytes")
    return int(n.value)


def check_conversions(stream=None) -> tuple:
    """Mismatches of the device E4M3 encoder and bf16 rounding against their integer
    definitions over every non-NaN fp32 bit pattern (fdkv_check_conversions)."""
    out = (ctypes.c_uint64 * 2)()
    _check(load().fdkv_check_conversions(out, _stream(stream)), "fdkv_check_conversions")
    return int(out[0]), int(out[1])


def decode_workspace(d: Dims, batch: int, max_seq_len: int) -> int:
    n = ctypes.c_size_t(0)
    _check(load().fdkv_decode_workspace(ctypes.byref(d), int(batch), int(max_seq_len), ctypes.byref(n)),
           "fdkv_decode_workspace")
    return int(n.value)


# ----------------------------------------------------------------- device entry points
def probe(d: Dims, seq_len: int, k_layers: Sequence, qp_layers: Sequence, n_probe: int, errors_out, ws,
          stream=None, token_scores=None, k_select=None):
    """Queue fdkv_probe; ``k_layers``/``qp_layers`` are per-layer device tensors;
    ``token_scores`` (token-level residual set) receives s_t ``[n_blocks][Hkv][T]``;
    ``k_select`` (``selection_bytes`` bytes) the K selections for compress to reuse."""
    _check(load().fdkv_probe(ctypes.byref(d), int(seq_len), _ptr_array(k_layers), _ptr_array(qp_layers),
                             int(n_probe), _dev(errors_out), _dev(token_scores), _dev(ws),
                             int(ws.numel() * ws.element_size()), _dev(k_select), _stream(stream)), "fdkv_probe")


def compress(d: Dims, seq_len: int, k_layers: Sequence, v_layers: Sequence, modes, seg_offsets, cache,
             stream=None, token_scores=None, k_select=None):
    """Queue fdkv_compress for one sequence (``modes``/``seg_offsets`` device tensors; ``token_scores``
    from the probe when residual heads hold a token-level set; ``k_select`` the probe's K selections
    of the same keys, or None to select in the pass)."""
    _check(load().fdkv_compress(ctypes.byref(d), int(seq_len), _ptr_array(k_layers), _ptr_array(v_layers),
                                _dev(modes), _dev(seg_offsets), _dev(token_scores), _dev(k_select), _dev(cache),
                                _stream(stream)), "fdkv_compress")


def decode_attn(d: Dims, batch: int, seq_lens, max_seq_len: int, modes, seg_offsets, cache, layer: int, q, out,
                sm_scale: float, ws, stream=None):
    """Queue fdkv_decode_attn for one layer."""
    _check(load().fdkv_decode_attn(ctypes.byref(d), int(batch), _dev(seq_lens), int(max_seq_len), _dev(modes),
                                   _dev(seg_offsets), _dev(cache), int(layer), _dev(q), _dev(out),
                                   ctypes.c_float(sm_scale), _dev(ws), int(ws.numel() * ws.element_size()),
                                   _stream(stream)), "fdkv_decode_attn")


def decode_partial(d: Dims, batch: int, seq_lens, max_seq_len: int, modes, seg_offsets, cache, layer: int, q,
                   sm_scale: float, ws, stream=None):
    """Queue fdkv_decode_partial: the split-K records of one layer into ``ws``."""
    _check(load().fdkv_decode_partial(ctypes.byref(d), int(batch), _dev(seq_lens), int(max_seq_len), _dev(modes),
                                      _dev(seg_offsets), _dev(cache), int(layer), _dev(q), ctypes.c_float(sm_scale),
                                      _dev(ws), int(ws.numel() * ws.element_size()), _stream(stream)),
           "fdkv_decode_partial")


def decode_combine(d: Dims, batch: int, n_chunks: int, out, ws, stream=None):
    """Queue fdkv_decode_combine: merge ``n_chunks`` records per (sequence, query head) of ``ws`` into ``out``."""
    _check(load().fdkv_decode_combine(ctypes.byref(d), int(batch), int(n_chunks), _dev(out), _dev(ws),
                                      int(ws.numel() * ws.element_size()), _stream(stream)), "fdkv_decode_combine")


def decode_static_scratch_bytes() -> int:
    """Bytes of the static device scratch behind fdkv_decode_attn_static."""
    return int(load().fdkv_decode_static_scratch_bytes())


def decode_attn_static(d: Dims, batch: int, seq_lens, max_seq_len: int, modes, seg_offsets, cache, layer: int, q,
                       out, sm_scale: float, stream=None):
    """Queue fdkv_decode_attn_static for one layer (no workspace: the library's static scratch)."""
    _check(load().fdkv_decode_attn_static(ctypes.byref(d), int(batch), _dev(seq_lens), int(max_seq_len), _dev(modes),
                                          _dev(seg_offsets), _dev(cache), int(layer), _dev(q), _dev(out),
                                          ctypes.c_float(sm_scale), _stream(stream)), "fdkv_decode_attn_static")


def decode_attn_raw(d: Dims, batch: int, seq_lens_ptr: int, max_seq_len: int, modes_ptr: int, offs_ptr: int,
                    cache_ptr: int, layer: int, q_ptr: int, out_ptr: int, sm_scale: float, ws_ptr: int,
                    ws_bytes: int, stream_ptr: int) -> int:
    """Same call with raw integer pointers (for tight timing loops); returns the status."""
    return load().fdkv_decode_attn(ctypes.byref(d), batch, seq_lens_ptr, max_seq_len, modes_ptr, offs_ptr,
                                   cache_ptr, layer, q_ptr, out_ptr, ctypes.c_float(sm_scale), ws_ptr, ws_bytes,
                                   ctypes.c_void_p(stream_ptr))


# ----------------------------------------------------------------- generation: spans and the exact tail
def append(d: Dims, batch: int, pos, cap: int, k_new, v_new, tail_k, tail_v, stream=None):
    """Queue fdkv_append: row ``pos[s]`` of the layer's tail gets the new K / V rows."""
    _check(load().fdkv_append(ctypes.byref(d), int(batch), _dev(pos), int(cap), _dev(k_new), _dev(v_new),
                              _dev(tail_k), _dev(tail_v), _stream(stream)), "fdkv_append")


def decode_spans_workspace(d: Dims, batch: int, max_seq_lens, tail_cap: int) -> int:
    m = np.ascontiguousarray(max_seq_lens, dtype=np.int32)
    n = ctypes.c_size_t(0)
    _check(load().fdkv_decode_spans_workspace(ctypes.byref(d), int(batch), int(m.size), _np_ptr(m),
                                              int(tail_cap), ctypes.byref(n)), "fdkv_decode_spans_workspace")
    return int(n.value)


def decode_spans(d: Dims, batch: int, spans: Sequence[Span], tail, layer: int, q, out, sm_scale: float, ws,
                 stream=None):
    """Queue fdkv_decode_spans; ``spans`` are ``Span`` descriptors, ``tail`` a ``Tail`` or None."""
    arr = (Span * max(len(spans), 1))(*spans)
    _check(load().fdkv_decode_spans(ctypes.byref(d), int(batch), len(spans), ctypes.cast(arr, ctypes.c_void_p),
                                    None if tail is None else ctypes.byref(tail), int(layer), _dev(q), _dev(out),
                                    ctypes.c_float(sm_scale), _dev(ws), int(ws.numel() * ws.element_size()),
                                    _stream(stream)), "fdkv_decode_spans")
