"""Host-side checks of the C ABI (no GPU needed).

The library must load, export every function that ``include/avq.h``
declares, and reject invalid arguments on the host before anything is
launched (these calls pass null device pointers and never reach the GPU).
"""
import ctypes
import re
from pathlib import Path

import pytest

from paper_2607_12789_amd import avq

ROOT = Path(__file__).resolve().parents[1]
HEADER = ROOT / "include" / "avq.h"
OK, INVALID, UNSUPPORTED = avq.AVQ_OK, avq.AVQ_ERR_INVALID_ARG, avq.AVQ_ERR_UNSUPPORTED
F32, BF16 = avq.AVQ_F32, avq.AVQ_BF16


def declared_functions():
    text = HEADER.read_text()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+[\s\*]+(avq_\w+)\s*\(", text, re.M)))


@pytest.fixture(scope="module")
def L():
    if not avq.library_path().exists():
        pytest.fail("libavq.so is not built (python -m paper_2607_12789_amd.build)")
    return avq.lib()


def test_header_declares_the_entry_points():
    assert declared_functions() == sorted(avq.SYMBOLS)


def test_library_exports_every_declared_symbol(L):
    for name in declared_functions():
        assert hasattr(L, name), name
    assert L.avq_version() == 202


NULL = None
FAKE = ctypes.c_void_p(16)  # never dereferenced: validation fails first


def assign(L, dtype=BF16, B=1, H=1, N=8, d=64, M0=4, Ch=2, ptrs=(FAKE,) * 5):
    return L.avq_assign(dtype, B, H, N, d, M0, Ch, *ptrs, NULL)


def aggregate(L, dtype=BF16, B=1, H=1, N=8, d=64, M0=4, Ch=2, ptrs=(FAKE,) * 5):
    return L.avq_aggregate(dtype, B, H, N, d, M0, Ch, *ptrs, NULL)


def attn(L, dtype=BF16, B=1, H=1, N=8, d=64, M0=4, Ch=2, P=1, bq=64, ptrs=(FAKE,) * 5):
    return L.avq_attention_fwd(dtype, B, H, N, d, M0, Ch, P, bq, *ptrs, NULL, NULL, NULL)


def attn_tiled(L, dtype=BF16, B=1, H=1, N=8, d=64, M0=4, Ch=2, P=1, bq=64, ptrs=(FAKE,) * 5):
    return L.avq_attention_fwd_tiled(dtype, B, H, N, d, M0, Ch, P, bq, *ptrs, NULL, NULL, NULL)


@pytest.mark.parametrize("kw,status", [
    (dict(dtype=7), INVALID),
    (dict(B=0), INVALID), (dict(H=-1), INVALID), (dict(N=0), INVALID), (dict(M0=0), INVALID),
    (dict(Ch=-1), INVALID),
    (dict(d=96), UNSUPPORTED), (dict(d=32), UNSUPPORTED), (dict(Ch=3), UNSUPPORTED),
    (dict(Ch=32), UNSUPPORTED), (dict(M0=513), UNSUPPORTED),
    (dict(B=1 << 14, H=1 << 10, N=1 << 10, d=128), UNSUPPORTED),
])
def test_shape_validation(L, kw, status):
    for fn in (assign, aggregate, attn, attn_tiled):
        assert fn(L, **kw) == status, (fn.__name__, kw)
        assert L.avq_last_error().decode() != ""


def test_null_pointers_are_rejected(L):
    for i in range(5):
        ptrs = [FAKE] * 5
        ptrs[i] = NULL
        assert assign(L, ptrs=ptrs) == INVALID
    # V, code_idx, counts are required; of Vbar and packed at least one
    for i in (0, 1, 3):
        ptrs = [FAKE] * 5
        ptrs[i] = NULL
        assert aggregate(L, ptrs=ptrs) == INVALID
    assert aggregate(L, ptrs=(FAKE, FAKE, NULL, FAKE, NULL)) == INVALID
    for fn in (attn, attn_tiled):
        for i in range(5):
            ptrs = [FAKE] * 5
            ptrs[i] = NULL
            assert fn(L, ptrs=ptrs) == INVALID
        assert "null" in L.avq_last_error().decode()


def test_packed_size(L):
    # octets of 8 codes: parents padded to a multiple of 64, ceil(Ch/8) child
    # octets per parent, one empty octet; each octet is 8 d values plus 64
    # bytes of count info
    def expect(M0, Ch, d, esz):
        n_oct = -(-M0 // 64) * 8 + M0 * -(-Ch // 8) + 1
        return n_oct * (8 * d * esz + 64)
    assert L.avq_packed_bytes(BF16, 256, 8, 128) == expect(256, 8, 128, 2)
    assert L.avq_packed_bytes(BF16, 256, 8, 128) == (32 + 256 + 1) * (2048 + 64)
    assert L.avq_packed_bytes(F32, 37, 16, 64) == expect(37, 16, 64, 4)
    assert L.avq_packed_bytes(BF16, 5, 2, 64) == expect(5, 2, 64, 2)
    assert L.avq_packed_bytes(BF16, 100, 0, 64) == expect(100, 0, 64, 2)  # flat codebook
    assert L.avq_packed_bytes(BF16, 4, -1, 64) == -1
    assert L.avq_packed_bytes(BF16, 0, 2, 64) == -1
    assert L.avq_packed_bytes(BF16, 4, 2, -1) == -1
    assert L.avq_packed_bytes(7, 4, 2, 64) == -1


def test_misaligned_pointers_are_rejected(L):
    odd = ctypes.c_void_p(24)
    assert assign(L, ptrs=(odd,) + (FAKE,) * 4) == INVALID
    assert aggregate(L, ptrs=(FAKE, FAKE, FAKE, FAKE, odd)) == INVALID
    assert attn(L, ptrs=(FAKE,) * 3 + (odd,) + (FAKE,)) == INVALID
    assert "aligned" in L.avq_last_error().decode()


@pytest.mark.parametrize("P,bq,status", [(-1, 64, INVALID), (5, 64, INVALID), (1, 0, INVALID),
                                         (1, 257, UNSUPPORTED)])
def test_attention_argument_validation(L, P, bq, status):
    assert attn(L, P=P, bq=bq) == status
    assert attn_tiled(L, P=P, bq=bq) == status


def test_flat_codebook_arguments(L):
    # Ch = 0: no children to select, so P must be 0
    assert attn(L, Ch=0, P=1) == INVALID
    assert "flat" in L.avq_last_error().decode()
    assert attn_tiled(L, Ch=0, P=1) == INVALID
    # Cc may be NULL: validation goes on to the next problem (here a
    # misaligned output), which also proves nothing was launched
    odd = ctypes.c_void_p(24)
    assert assign(L, Ch=0, ptrs=(FAKE, FAKE, NULL, odd, FAKE)) == INVALID
    assert "aligned" in L.avq_last_error().decode()
    assert attn(L, Ch=0, P=0, ptrs=(FAKE, FAKE, NULL, FAKE, odd)) == INVALID
    assert "aligned" in L.avq_last_error().decode()
    # with children, Cc is required
    assert assign(L, Ch=2, ptrs=(FAKE, FAKE, NULL, FAKE, FAKE)) == INVALID
    assert "null" in L.avq_last_error().decode()


def test_binding_refuses_cpu_tensors():
    import torch
    K = torch.zeros(1, 1, 8, 64, dtype=torch.bfloat16)
    Cp = torch.zeros(1, 4, 64, dtype=torch.bfloat16)
    Cc = torch.zeros(1, 4, 2, 64, dtype=torch.bfloat16)
    with pytest.raises(ValueError):
        avq.assign(K, Cp, Cc)


def update(L, dtype=BF16, B=1, H=1, d=64, M0=4, Ch=2, lam=0.9, ptrs=(FAKE,) * 6):
    return L.avq_codebook_update(dtype, B, H, d, M0, Ch, lam, *ptrs, NULL)


def test_codebook_update_validation(L):
    for lam in (0.0, -0.5, 1.5, float("nan")):
        assert update(L, lam=lam) == INVALID
        assert "lambda" in L.avq_last_error().decode()
    assert update(L, lam=1.0, ptrs=(FAKE,) * 5 + (ctypes.c_void_p(24),)) == INVALID  # lambda 1 ok
    assert "aligned" in L.avq_last_error().decode()
    for i in range(6):
        ptrs = [FAKE] * 6
        ptrs[i] = NULL
        assert update(L, ptrs=ptrs) == INVALID
        assert "null" in L.avq_last_error().decode()
    # Ch = 0: no children to write
    assert update(L, Ch=0, ptrs=(FAKE,) * 4 + (ctypes.c_void_p(24), NULL)) == INVALID
    assert "aligned" in L.avq_last_error().decode()
    assert update(L, d=96) == UNSUPPORTED
    assert update(L, Ch=3) == UNSUPPORTED
    assert update(L, M0=0) == INVALID


def test_ordered_attention_validation(L):
    def ordered(order=FAKE, tiled=0, **kw):
        args = dict(dtype=BF16, B=1, H=1, N=8, d=64, M0=4, Ch=2, P=1, bq=64)
        args.update(kw)
        return L.avq_attention_fwd_ordered(args["dtype"], args["B"], args["H"], args["N"],
                                           args["d"], args["M0"], args["Ch"], args["P"],
                                           args["bq"], order, tiled, *(FAKE,) * 5, NULL, NULL,
                                           NULL)
    assert ordered(order=NULL) == INVALID
    assert "query_order" in L.avq_last_error().decode()
    assert ordered(tiled=2) == INVALID
    assert ordered(order=ctypes.c_void_p(24)) == INVALID
    assert "aligned" in L.avq_last_error().decode()
    assert ordered(d=96) == UNSUPPORTED
    assert ordered(P=9) == INVALID



def pack(L, dtype=BF16, B=1, H=1, d=64, M0=4, Ch=2, ptrs=(FAKE,) * 3):
    return L.avq_pack_aggregates(dtype, B, H, d, M0, Ch, *ptrs, NULL)


def test_pack_aggregates_validation(L):
    for i in range(3):
        ptrs = [FAKE] * 3
        ptrs[i] = NULL
        assert pack(L, ptrs=ptrs) == INVALID
        assert "null" in L.avq_last_error().decode()
    assert pack(L, ptrs=(FAKE, ctypes.c_void_p(24), FAKE)) == INVALID
    assert "aligned" in L.avq_last_error().decode()
    assert pack(L, dtype=7) == INVALID
    assert pack(L, B=0) == INVALID
    assert pack(L, M0=0) == INVALID
    assert pack(L, d=96) == UNSUPPORTED
    assert pack(L, Ch=3) == UNSUPPORTED
    assert pack(L, M0=513) == UNSUPPORTED


def assign_aggregate(L, dtype=BF16, B=1, H=1, N=8, d=64, M0=4, Ch=2, ptrs=(FAKE,) * 9):
    return L.avq_assign_aggregate(dtype, B, H, N, d, M0, Ch, *ptrs, NULL)


def test_assign_aggregate_validation(L):
    # K, V, Cp, Cc, parent_idx, code_idx, Vbar, counts, packed: each required
    # one null at a time (Vbar and packed may each be null, not both; Cc only
    # when Ch = 0)
    # (a call that passes validation would launch: every call here fails it)
    names = ["K", "V", "Cp", "Cc", "parent_idx", "code_idx", "Vbar", "counts", "packed"]
    for i, name in enumerate(names):
        if name in ("Vbar", "packed"):
            continue
        ptrs = [FAKE] * 9
        ptrs[i] = NULL
        assert assign_aggregate(L, ptrs=ptrs) == INVALID, name
        assert "null" in L.avq_last_error().decode()
    ptrs = [FAKE] * 9
    ptrs[6] = ptrs[8] = NULL
    assert assign_aggregate(L, ptrs=ptrs) == INVALID
    assert "both null" in L.avq_last_error().decode()
    ptrs = [FAKE] * 9
    ptrs[1] = ctypes.c_void_p(24)
    assert assign_aggregate(L, ptrs=ptrs) == INVALID
    assert "aligned" in L.avq_last_error().decode()
    assert assign_aggregate(L, dtype=7) == INVALID
    assert assign_aggregate(L, N=0) == INVALID
    assert assign_aggregate(L, d=96) == UNSUPPORTED
    assert assign_aggregate(L, Ch=3) == UNSUPPORTED
    assert assign_aggregate(L, M0=513) == UNSUPPORTED
