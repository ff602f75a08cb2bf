"""Python binding of ``libavq.so``: argument marshalling only.

Every step of the forward pass runs in the HIP kernels behind the C ABI
declared in ``include/avq.h``; this module checks tensor shapes, dtypes and
devices, passes raw device pointers and the current HIP stream, and turns a
non-OK status into an exception. There is no fallback: if the library is not
built, every call raises.
"""
from __future__ import annotations

import ctypes
import os
from pathlib import Path
from typing import Optional

import torch

# AVQ_LIB names another build of the same library (a sanitizer build of the
# host code, for instance); by default the in-tree build is loaded
_LIB_PATH = Path(os.environ.get("AVQ_LIB") or Path(__file__).resolve().parent / "libavq.so")
_lib = None

AVQ_OK, AVQ_ERR_INVALID_ARG, AVQ_ERR_UNSUPPORTED, AVQ_ERR_DEVICE = 0, 1, 2, 3
AVQ_F32, AVQ_BF16 = 0, 1
_DTYPES = {torch.float32: AVQ_F32, torch.bfloat16: AVQ_BF16}
SYMBOLS = ("avq_version", "avq_last_error", "avq_packed_bytes", "avq_assign",
           "avq_aggregate", "avq_attention_fwd", "avq_attention_fwd_tiled",
           "avq_codebook_update", "avq_attention_fwd_ordered", "avq_gilbert_order",
           "avq_pack_aggregates", "avq_assign_aggregate")
IMPORTANCE_TILE = 64  # parents per codeword tile of attention_fwd(tiled_importance=True)


class AvqError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"status {status}: {message}")
        self.status = status


def library_path() -> Path:
    return _LIB_PATH


def lib():
    """The loaded C library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not _LIB_PATH.exists():
            raise RuntimeError(f"{_LIB_PATH} is missing: build it with "
                               "`python -m paper_2607_12789_amd.build`")
        L = ctypes.CDLL(str(_LIB_PATH))
        i32, vp = ctypes.c_int32, ctypes.c_void_p
        L.avq_version.restype = ctypes.c_int
        L.avq_last_error.restype = ctypes.c_char_p
        L.avq_packed_bytes.argtypes = [ctypes.c_int, i32, i32, i32]
        L.avq_packed_bytes.restype = ctypes.c_int64
        L.avq_assign.argtypes = [ctypes.c_int, i32, i32, i32, i32, i32, i32, vp, vp, vp, vp, vp, vp]
        L.avq_aggregate.argtypes = [ctypes.c_int, i32, i32, i32, i32, i32, i32,
                                    vp, vp, vp, vp, vp, vp]
        for name in ("avq_attention_fwd", "avq_attention_fwd_tiled"):
            getattr(L, name).argtypes = [ctypes.c_int, i32, i32, i32, i32, i32, i32, i32, i32,
                                         vp, vp, vp, vp, vp, vp, vp, vp]
        L.avq_attention_fwd_ordered.argtypes = [ctypes.c_int, i32, i32, i32, i32, i32, i32, i32,
                                                i32, vp, i32, vp, vp, vp, vp, vp, vp, vp, vp]
        L.avq_gilbert_order.argtypes = [i32, i32, vp, vp]
        L.avq_codebook_update.argtypes = [ctypes.c_int, i32, i32, i32, i32, i32, ctypes.c_float,
                                          vp, vp, vp, vp, vp, vp, vp]
        L.avq_pack_aggregates.argtypes = [ctypes.c_int, i32, i32, i32, i32, i32, vp, vp, vp, vp]
        L.avq_assign_aggregate.argtypes = [ctypes.c_int, i32, i32, i32, i32, i32, i32,
                                           vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
        for name in ("avq_assign", "avq_aggregate", "avq_attention_fwd", "avq_pack_aggregates",
                     "avq_assign_aggregate",
                     "avq_attention_fwd_tiled", "avq_codebook_update",
                     "avq_attention_fwd_ordered", "avq_gilbert_order"):
            getattr(L, name).restype = ctypes.c_int
        _lib = L
    return _lib


def _check(status: int) -> None:
    if status != AVQ_OK:
        raise AvqError(status, lib().avq_last_error().decode())


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _dev(t: torch.Tensor, name: str, dtype=None, shape=None):
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise ValueError(f"{name} must be a tensor on the GPU")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    return t


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype not in _DTYPES:
        raise ValueError(f"unsupported dtype {t.dtype}: use float32 or bfloat16")
    return _DTYPES[t.dtype]


def assign(K, Cp, Cc, parent_idx=None, code_idx=None, stream=None):
    """Tree assignment of the keys (``avq_assign``). Returns (parent_idx, code_idx)."""
    B, H, N, d = K.shape
    M0, Ch = Cc.shape[1], Cc.shape[2]
    _dev(K, "K")
    _dev(Cp, "Cp", K.dtype, (H, M0, d))
    _dev(Cc, "Cc", K.dtype, (H, M0, Ch, d))
    if parent_idx is None:
        parent_idx = torch.empty((B, H, N), dtype=torch.int32, device=K.device)
    if code_idx is None:
        code_idx = torch.empty((B, H, N), dtype=torch.int32, device=K.device)
    _dev(parent_idx, "parent_idx", torch.int32, (B, H, N))
    _dev(code_idx, "code_idx", torch.int32, (B, H, N))
    _check(lib().avq_assign(_dtype_code(K), B, H, N, d, M0, Ch, _ptr(K), _ptr(Cp), _ptr(Cc),
                            _ptr(parent_idx), _ptr(code_idx), _stream(stream)))
    return parent_idx, code_idx


def packed_bytes(dtype: torch.dtype, M0: int, Ch: int, d: int) -> int:
    """Bytes of the packed aggregates of one (batch, head)."""
    if dtype not in _DTYPES:
        raise ValueError(f"unsupported dtype {dtype}: use float32 or bfloat16")
    n = lib().avq_packed_bytes(_DTYPES[dtype], M0, Ch, d)
    if n < 0:
        raise ValueError(f"invalid sizes M0={M0} Ch={Ch} d={d}")
    return n


def aggregate(V, code_idx, M0: int, Ch: int, packed=None, counts=None, Vbar=None,
              sums: bool = False, stream=None):
    """Per-codeword counts, packed aggregates and optionally fp32 sums (``avq_aggregate``).

    Returns (packed, counts, Vbar); Vbar is None unless ``sums`` is set or a
    buffer is given. ``packed`` is a uint8 tensor [B, H, packed_bytes(...)]
    that ``attention_fwd`` takes.
    """
    B, H, N, d = V.shape
    Mtot = M0 * (1 + Ch)
    _dev(V, "V")
    _dev(code_idx, "code_idx", torch.int32, (B, H, N))
    E = packed_bytes(V.dtype, M0, Ch, d)
    if packed is None:
        packed = torch.empty((B, H, E), dtype=torch.uint8, device=V.device)
    if counts is None:
        counts = torch.empty((B, H, Mtot), dtype=torch.int32, device=V.device)
    if Vbar is None and sums:
        Vbar = torch.empty((B, H, Mtot, d), dtype=torch.float32, device=V.device)
    _dev(packed, "packed", torch.uint8, (B, H, E))
    _dev(counts, "counts", torch.int32, (B, H, Mtot))
    if Vbar is not None:
        _dev(Vbar, "Vbar", torch.float32, (B, H, Mtot, d))
    _check(lib().avq_aggregate(_dtype_code(V), B, H, N, d, M0, Ch, _ptr(V), _ptr(code_idx),
                               _ptr(Vbar), _ptr(counts), _ptr(packed), _stream(stream)))
    return packed, counts, Vbar


def assign_aggregate(K, V, Cp, Cc, parent_idx=None, code_idx=None, packed=None, counts=None,
                     Vbar=None, sums: bool = False, stream=None):
    """Alg. 1 as one precompute (``avq_assign_aggregate``): the codes of
    ``assign`` and the aggregates of ``aggregate``, with the child compare and
    the value sums in one pass. Returns (parent_idx, code_idx, packed, counts,
    Vbar); Vbar is None unless ``sums`` is set or a buffer is given."""
    B, H, N, d = K.shape
    M0, Ch = Cc.shape[1], Cc.shape[2]
    Mtot = M0 * (1 + Ch)
    _dev(K, "K")
    _dev(V, "V", K.dtype, (B, H, N, d))
    _dev(Cp, "Cp", K.dtype, (H, M0, d))
    _dev(Cc, "Cc", K.dtype, (H, M0, Ch, d))
    dev = K.device
    if parent_idx is None:
        parent_idx = torch.empty((B, H, N), dtype=torch.int32, device=dev)
    if code_idx is None:
        code_idx = torch.empty((B, H, N), dtype=torch.int32, device=dev)
    E = packed_bytes(K.dtype, M0, Ch, d)
    if packed is None:
        packed = torch.empty((B, H, E), dtype=torch.uint8, device=dev)
    if counts is None:
        counts = torch.empty((B, H, Mtot), dtype=torch.int32, device=dev)
    if Vbar is None and sums:
        Vbar = torch.empty((B, H, Mtot, d), dtype=torch.float32, device=dev)
    _dev(parent_idx, "parent_idx", torch.int32, (B, H, N))
    _dev(code_idx, "code_idx", torch.int32, (B, H, N))
    _dev(packed, "packed", torch.uint8, (B, H, E))
    _dev(counts, "counts", torch.int32, (B, H, Mtot))
    if Vbar is not None:
        _dev(Vbar, "Vbar", torch.float32, (B, H, Mtot, d))
    _check(lib().avq_assign_aggregate(_dtype_code(K), B, H, N, d, M0, Ch, _ptr(K), _ptr(V),
                                      _ptr(Cp), _ptr(Cc), _ptr(parent_idx), _ptr(code_idx),
                                      _ptr(Vbar), _ptr(counts), _ptr(packed), _stream(stream)))
    return parent_idx, code_idx, packed, counts, Vbar


def pack_aggregates(Vbar, counts, M0: int, Ch: int, dtype, packed=None, stream=None):
    """The paper's aggregates (Vbar fp32 [B, H, Mtot, d], counts int32
    [B, H, Mtot]) in the operand layout ``attention_fwd`` reads
    (``avq_pack_aggregates``). Returns packed (uint8 [B, H, packed_bytes])."""
    B, H, Mtot, d = Vbar.shape
    if Mtot != M0 * (1 + Ch):
        raise ValueError(f"Vbar holds {Mtot} codes, expected M0 * (1 + Ch) = {M0 * (1 + Ch)}")
    _dev(Vbar, "Vbar", torch.float32)
    _dev(counts, "counts", torch.int32, (B, H, Mtot))
    E = packed_bytes(dtype, M0, Ch, d)
    if packed is None:
        packed = torch.empty((B, H, E), dtype=torch.uint8, device=Vbar.device)
    _dev(packed, "packed", torch.uint8, (B, H, E))
    _check(lib().avq_pack_aggregates(_DTYPES[dtype], B, H, d, M0, Ch, _ptr(Vbar), _ptr(counts),
                                     _ptr(packed), _stream(stream)))
    return packed


def attention_fwd(Q, Cp, Cc, packed, P: int, block_q: int, Y=None, topp_idx=None,
                  importance=None, debug: bool = False, tiled_importance: bool = False,
                  query_order=None, stream=None):
    """Refined-codebook attention (``avq_attention_fwd``, or
    ``avq_attention_fwd_tiled`` with ``tiled_importance``: the importance of
    App. B over tiles of IMPORTANCE_TILE parents).

    query_order (int32 [N] on the GPU): take the queries in this order
    (``avq_attention_fwd_ordered``); Y rows still land on their tokens.

    Returns Y, or (Y, topp_idx, importance) when ``debug`` is set (the two
    debug outputs are then allocated if not given).
    """
    B, H, N, d = Q.shape
    M0, Ch = Cc.shape[1], Cc.shape[2]
    T = (N + block_q - 1) // block_q if block_q > 0 else 0
    _dev(Q, "Q")
    _dev(Cp, "Cp", Q.dtype, (H, M0, d))
    _dev(Cc, "Cc", Q.dtype, (H, M0, Ch, d))
    _dev(packed, "packed", torch.uint8, (B, H, packed_bytes(Q.dtype, M0, Ch, d)))
    if Y is None:
        Y = torch.empty_like(Q)
    _dev(Y, "Y", Q.dtype, Q.shape)
    if debug:
        if topp_idx is None:
            topp_idx = torch.empty((B, H, T, max(P, 0)), dtype=torch.int32, device=Q.device)
        if importance is None:
            importance = torch.empty((B, H, T, M0), dtype=torch.float32, device=Q.device)
    if topp_idx is not None:
        _dev(topp_idx, "topp_idx", torch.int32, (B, H, T, P))
    if importance is not None:
        _dev(importance, "importance", torch.float32, (B, H, T, M0))
    if query_order is not None:
        _dev(query_order, "query_order", torch.int32, (N,))
        _check(lib().avq_attention_fwd_ordered(
            _dtype_code(Q), B, H, N, d, M0, Ch, P, block_q, _ptr(query_order),
            int(bool(tiled_importance)), _ptr(Q), _ptr(Cp), _ptr(Cc), _ptr(packed), _ptr(Y),
            _ptr(topp_idx), _ptr(importance), _stream(stream)))
    else:
        fn = lib().avq_attention_fwd_tiled if tiled_importance else lib().avq_attention_fwd
        _check(fn(_dtype_code(Q), B, H, N, d, M0, Ch, P, block_q, _ptr(Q), _ptr(Cp), _ptr(Cc),
                  _ptr(packed), _ptr(Y), _ptr(topp_idx), _ptr(importance), _stream(stream)))
    if debug:
        return Y, topp_idx, importance
    return Y


def forward(Q, K, V, Cp, Cc, P: int, block_q: int, stream=None):
    """The whole forward pass: assign, aggregate, attention. Returns Y."""
    M0, Ch = Cc.shape[1], Cc.shape[2]
    _, code_idx = assign(K, Cp, Cc, stream=stream)
    packed, _, _ = aggregate(V, code_idx, M0, Ch, stream=stream)
    return attention_fwd(Q, Cp, Cc, packed, P, block_q, stream=stream)


def codebook_update(sums, counts, S, Nema, M0: int, Ch: int, lam: float, Cp_out=None,
                    Cc_out=None, dtype=None, stream=None):
    """EMA codebook step with the constrained child projection
    (``avq_codebook_update``). sums [B, H, Mtot, d] fp32 and counts
    [B, H, Mtot] int32 are the aggregates of the keys; S [H, Mtot, d] and
    Nema [H, Mtot] (fp32) are updated in place. Returns (Cp, Cc) in ``dtype``
    (default bfloat16 unless Cp_out is given)."""
    B, H, Mtot, d = sums.shape
    if Mtot != M0 * (1 + Ch):
        raise ValueError(f"sums hold {Mtot} codes, expected M0 * (1 + Ch) = {M0 * (1 + Ch)}")
    _dev(sums, "sums", torch.float32)
    _dev(counts, "counts", torch.int32, (B, H, Mtot))
    _dev(S, "S", torch.float32, (H, Mtot, d))
    _dev(Nema, "Nema", torch.float32, (H, Mtot))
    if dtype is None:
        dtype = Cp_out.dtype if Cp_out is not None else torch.bfloat16
    if Cp_out is None:
        Cp_out = torch.empty((H, M0, d), dtype=dtype, device=sums.device)
    if Cc_out is None:
        Cc_out = torch.empty((H, M0, Ch, d), dtype=dtype, device=sums.device)
    _dev(Cp_out, "Cp_out", dtype, (H, M0, d))
    _dev(Cc_out, "Cc_out", dtype, (H, M0, Ch, d))
    _check(lib().avq_codebook_update(_dtype_code(Cp_out), B, H, d, M0, Ch, float(lam), _ptr(sums),
                                     _ptr(counts), _ptr(S), _ptr(Nema), _ptr(Cp_out),
                                     _ptr(Cc_out), _stream(stream)))
    return Cp_out, Cc_out


def gilbert_order(width: int, height: int):
    """Tokens of a width x height grid (token y*width + x) in the order of a
    generalized Hilbert curve (``avq_gilbert_order``, host only). Returns
    (order, rank) as int32 CPU tensors, rank[order[k]] = k."""
    n = int(width) * int(height)
    order = torch.empty(max(n, 0), dtype=torch.int32)
    rank = torch.empty(max(n, 0), dtype=torch.int32)
    _check(lib().avq_gilbert_order(int(width), int(height), _ptr(order), _ptr(rank)))
    return order, rank

