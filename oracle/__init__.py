"""fp64 CPU oracle for the AVQ-Attention forward pass (test infrastructure).

Only the tests, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package. The product path (the HIP library and
its binding) never imports it, and the two share no code: this package widens
the stored inputs to fp64, calls the plain C loops in ``avq_oracle.c`` and
returns NumPy arrays.

Each function names the passage of the paper it follows; the C file carries
the definitions term by term.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from pathlib import Path

import numpy as np

_DIR = Path(__file__).resolve().parent
_SRC = _DIR / "avq_oracle.c"
_LIB = _DIR / "libavq_oracle.so"
# AVQ_ORACLE_LIB: an already built copy to load instead (the sanitizer build)
_LIB_OVERRIDE = os.environ.get("AVQ_ORACLE_LIB")
_lib = None

_f64p = ctypes.POINTER(ctypes.c_double)
_i32p = ctypes.POINTER(ctypes.c_int32)
_i64p = ctypes.POINTER(ctypes.c_int64)
_u8p = ctypes.POINTER(ctypes.c_uint8)


def build(force: bool = True) -> Path:
    """Compile the oracle with gcc (plain -O2, OpenMP) into ``libavq_oracle.so``."""
    if force or not _LIB.exists() or _LIB.stat().st_mtime < _SRC.stat().st_mtime:
        tmp = _LIB.with_suffix(".so.tmp")
        subprocess.run(["gcc", "-O2", "-std=c99", "-fopenmp", "-fPIC", "-shared",
                        str(_SRC), "-o", str(tmp), "-lm"], check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if _LIB_OVERRIDE:
            _lib = open_library(_LIB_OVERRIDE)
            return _lib
        if not _LIB.exists() or _LIB.stat().st_mtime < _SRC.stat().st_mtime:
            build(force=True)
        _lib = open_library(_LIB)
    return _lib


def open_library(path):
    """Open a compiled oracle and declare its C signatures."""
    lib = ctypes.CDLL(str(path))
    i = ctypes.c_int
    lib.avqo_assign.argtypes = [i, i, i, i, i, i, _f64p, _f64p, _f64p, _i32p, _i32p,
                                _f64p, _f64p, _f64p, _f64p]
    lib.avqo_aggregate.argtypes = [i, i, i, i, i, _f64p, _i32p, _i32p, _f64p, _i64p]
    lib.avqo_importance.argtypes = [i, i, i, i, i, i, i, _f64p, _f64p, _i64p, _u8p, _f64p]
    lib.avqo_importance_tiled.argtypes = [i, i, i, i, i, i, i, i, _f64p, _f64p, _i64p, _u8p,
                                          _f64p]
    lib.avqo_codebook_update.argtypes = [i, i, i, i, i, ctypes.c_double, _f64p, _i64p, _f64p,
                                         _f64p, _f64p, _f64p]
    lib.avqo_topp.argtypes = [ctypes.c_longlong, i, i, _f64p, _u8p, _i32p]
    lib.avqo_output.argtypes = [i, i, i, i, i, i, i, i, _f64p, _f64p, _f64p, _f64p,
                                _i64p, _i32p, i, _u8p, _f64p, _f64p]
    lib.avqo_num_threads.restype = ctypes.c_int
    lib.avqo_set_num_threads.argtypes = [i]
    return lib


def num_threads() -> int:
    return _load().avqo_num_threads()


def set_num_threads(n: int) -> None:
    _load().avqo_set_num_threads(int(n))


def f64(x) -> np.ndarray:
    """Exact widening of a stored bf16/fp32 tensor (torch or NumPy) to fp64."""
    if hasattr(x, "detach"):
        x = x.detach().cpu().double().numpy()
    return np.ascontiguousarray(x, dtype=np.float64)


def _p(a: np.ndarray, t):
    return a.ctypes.data_as(t) if a is not None else ctypes.cast(None, t)


def _mask(mask, n):
    if mask is None:
        return None
    m = np.ascontiguousarray(np.asarray(mask, dtype=np.uint8).reshape(-1))
    if m.size != n:
        raise ValueError(f"mask has {m.size} entries, expected {n}")
    return m


def assign(K, Cp, Cc) -> dict:
    """Tree assignment (Sec. 3.2; Alg. 1): parent argmin, then child argmin.

    K: [B, H, N, d]; Cp: [H, M0, d]; Cc: [H, M0, Ch, d].
    Returns parent_idx, code_idx (int32 [B, H, N]) and the fp64 certification
    distances d_parent, d_parent2, d_child, d_child2 ([B, H, N]).
    """
    K, Cp, Cc = f64(K), f64(Cp), f64(Cc)
    B, H, N, d = K.shape
    M0, Ch = Cc.shape[1], Cc.shape[2]
    out = {k: np.empty((B, H, N), np.int32) for k in ("parent_idx", "code_idx")}
    for k in ("d_parent", "d_parent2", "d_child", "d_child2"):
        out[k] = np.empty((B, H, N), np.float64)
    _load().avqo_assign(B * H, H, N, d, M0, Ch, _p(K, _f64p), _p(Cp, _f64p), _p(Cc, _f64p),
                        _p(out["parent_idx"], _i32p), _p(out["code_idx"], _i32p),
                        _p(out["d_parent"], _f64p), _p(out["d_parent2"], _f64p),
                        _p(out["d_child"], _f64p), _p(out["d_child2"], _f64p))
    return out


def aggregate(V, parent_idx, code_idx, M0: int, Ch: int):
    """Eq. (aggregates): (Vbar [B,H,Mtot,d] fp64, counts [B,H,Mtot] int64)."""
    V = f64(V)
    B, H, N, d = V.shape
    pi = np.ascontiguousarray(parent_idx, dtype=np.int32)
    ci = np.ascontiguousarray(code_idx, dtype=np.int32)
    Mtot = M0 * (1 + Ch)
    Vbar = np.empty((B, H, Mtot, d), np.float64)
    counts = np.empty((B, H, Mtot), np.int64)
    _load().avqo_aggregate(B * H, N, d, M0, Ch, _p(V, _f64p), _p(pi, _i32p), _p(ci, _i32p),
                           _p(Vbar, _f64p), _p(counts, _i64p))
    return Vbar, counts


def importance(Q, Cp, counts, Ch: int, block_q: int, tile_mask=None) -> np.ndarray:
    """Eq. (importance) per query tile: w [B, H, T, M0] (rows outside tile_mask: 0)."""
    Q, Cp = f64(Q), f64(Cp)
    B, H, N, d = Q.shape
    M0 = Cp.shape[1]
    n = np.ascontiguousarray(counts, dtype=np.int64)
    T = (N + block_q - 1) // block_q
    w = np.zeros((B, H, T, M0), np.float64)
    m = _mask(tile_mask, B * H * T)
    _load().avqo_importance(B * H, H, N, d, M0, Ch, block_q, _p(Q, _f64p), _p(Cp, _f64p),
                            _p(n, _i64p), _p(m, _u8p), _p(w, _f64p))
    return w


def importance_tiled(Q, Cp, counts, Ch: int, block_q: int, tile_c: int,
                     tile_mask=None) -> np.ndarray:
    """App. B importance (count-extrapolated denominator, parents in tiles of
    tile_c): w [B, H, T, M0] (rows outside tile_mask: 0)."""
    Q, Cp = f64(Q), f64(Cp)
    B, H, N, d = Q.shape
    M0 = Cp.shape[1]
    if tile_c < 1:
        raise ValueError("tile_c must be positive")
    n = np.ascontiguousarray(counts, dtype=np.int64)
    T = (N + block_q - 1) // block_q
    w = np.zeros((B, H, T, M0), np.float64)
    m = _mask(tile_mask, B * H * T)
    _load().avqo_importance_tiled(B * H, H, N, d, M0, Ch, block_q, tile_c, _p(Q, _f64p),
                                  _p(Cp, _f64p), _p(n, _i64p), _p(m, _u8p), _p(w, _f64p))
    return w


def capture(Q, K, parent_idx, sel, block_q: int, tile_mask=None) -> dict:
    """Top-P capture (App. B, tab. tiled_capture): the fraction of the exact
    softmax attention mass of each query (over the original keys, Eq.
    (standardattention)) that falls on keys whose parent is in its tile's
    selection sel [B, H, T, P]. Also the capture of the best possible
    selection: per tile, the P parents whose keys receive the most mass.

    Returns mean capture over the queries of the evaluated tiles for the
    given selection ("selected") and the best one ("exact")."""
    Q, K = f64(Q), f64(K)
    B, H, N, d = Q.shape
    T = (N + block_q - 1) // block_q
    par = np.asarray(parent_idx)
    sel = np.asarray(sel)
    P = sel.shape[-1]
    M0 = int(par.max()) + 1 if P == 0 else max(int(par.max()), int(sel.max())) + 1
    got, best, count = 0.0, 0.0, 0
    for b in range(B):
        for h in range(H):
            nk = K.shape[2]  # one row per key (the keys need not number N)
            onehot = np.zeros((nk, M0))
            onehot[np.arange(nk), par[b, h]] = 1.0
            for t in range(T):
                if tile_mask is not None and not tile_mask[b, h, t]:
                    continue
                i0, i1 = t * block_q, min(N, (t + 1) * block_q)
                S = Q[b, h, i0:i1] @ K[b, h].T
                A = np.exp(S - S.max(axis=1, keepdims=True))
                A /= A.sum(axis=1, keepdims=True)
                mass = A @ onehot  # [queries, M0]: attention mass per parent
                got += mass[:, sel[b, h, t]].sum()
                top = np.argsort(-mass.sum(axis=0), kind="stable")[:P]
                best += mass[:, top].sum()
                count += i1 - i0
    return {"selected": got / count, "exact": best / count}


def codebook_update(sums, counts, S, Nema, M0: int, Ch: int, lam: float):
    """App. A codebook update (EMA statistics, constrained child projection).

    sums [B, H, Mtot, d] key sums and counts [B, H, Mtot] of one batch (the
    aggregates of the keys); S [H, Mtot, d] and Nema [H, Mtot] the EMA state.
    Returns (S', Nema', Cp [H, M0, d], Cc [H, M0, Ch, d]) as fp64 arrays; the
    inputs are not modified."""
    sums = f64(sums)
    B, H, Mtot, d = sums.shape
    if Mtot != M0 * (1 + Ch):
        raise ValueError("sums do not hold M0 * (1 + Ch) codes")
    n = np.ascontiguousarray(counts, dtype=np.int64)
    S2 = np.array(f64(S), dtype=np.float64, copy=True)
    N2 = np.array(f64(Nema), dtype=np.float64, copy=True)
    Cp = np.zeros((H, M0, d))
    Cc = np.zeros((H, M0, Ch, d))
    _load().avqo_codebook_update(B, H, d, M0, Ch, float(lam), _p(sums, _f64p), _p(n, _i64p),
                                 _p(S2, _f64p), _p(N2, _f64p), _p(Cp, _f64p), _p(Cc, _f64p))
    return S2, N2, Cp, Cc


def topp(w, P: int, row_mask=None) -> np.ndarray:
    """Top-P parents per row of w, canonical order (w desc, index asc): int32 [..., P]."""
    w = np.ascontiguousarray(w, dtype=np.float64)
    M0 = w.shape[-1]
    if not 0 <= P <= M0:
        raise ValueError("P must lie in [0, M0]")
    rows = int(np.prod(w.shape[:-1]))
    sel = np.zeros(w.shape[:-1] + (P,), np.int32)
    m = _mask(row_mask, rows)
    if P > 0:
        _load().avqo_topp(rows, M0, P, _p(w, _f64p), _p(m, _u8p), _p(sel, _i32p))
    return sel


def output(Q, Cp, Cc, Vbar, counts, sel, block_q: int, recovered: bool = True,
           tile_mask=None):
    """Refined output (Eq. (vqflashattention) + Eq. (correcting_attention)).

    Returns (Y [B,H,N,d] fp64, zratio [B,H,N]) where zratio is the refined
    denominator over the parent-only denominator. Rows of tiles outside
    tile_mask are NaN.
    """
    Q, Cp, Cc, Vbar = f64(Q), f64(Cp), f64(Cc), f64(Vbar)
    B, H, N, d = Q.shape
    M0, Ch = Cc.shape[1], Cc.shape[2]
    n = np.ascontiguousarray(counts, dtype=np.int64)
    sel = np.ascontiguousarray(sel, dtype=np.int32)
    P = sel.shape[-1]
    T = (N + block_q - 1) // block_q
    if sel.shape != (B, H, T, P):
        raise ValueError(f"selection shape {sel.shape} != {(B, H, T, P)}")
    Y = np.full((B, H, N, d), np.nan)
    zr = np.full((B, H, N), np.nan)
    m = _mask(tile_mask, B * H * T)
    _load().avqo_output(B * H, H, N, d, M0, Ch, P, block_q, _p(Q, _f64p), _p(Cp, _f64p),
                        _p(Cc, _f64p), _p(Vbar, _f64p), _p(n, _i64p), _p(sel, _i32p),
                        int(bool(recovered)), _p(m, _u8p), _p(Y, _f64p), _p(zr, _f64p))
    return Y, zr


def forward(Q, K, V, Cp, Cc, P: int, block_q: int, recovered: bool = True,
            tile_mask=None, importance_tile=None) -> dict:
    """The whole forward pass (Fig. pipeline): assign, aggregate, importance,
    top-P, refined output. Returns every intermediate as NumPy arrays.
    importance_tile: None for Eq. (importance), or the codeword tile size of
    the App. B approximation."""
    Cc64 = f64(Cc)
    M0, Ch = Cc64.shape[1], Cc64.shape[2]
    a = assign(K, Cp, Cc64)
    Vbar, counts = aggregate(V, a["parent_idx"], a["code_idx"], M0, Ch)
    if importance_tile is None:
        w = importance(Q, Cp, counts, Ch, block_q, tile_mask)
    else:
        w = importance_tiled(Q, Cp, counts, Ch, block_q, importance_tile, tile_mask)
    sel = topp(w, P, tile_mask)
    Y, zr = output(Q, Cp, Cc64, Vbar, counts, sel, block_q, recovered, tile_mask)
    a.update(Vbar=Vbar, counts=counts, importance=w, selection=sel, Y=Y, zratio=zr)
    return a
