"""Host-side tests of the C ABI: the library loads, exports every function the
header declares, and rejects invalid arguments before any device work.

Fake pointers are used only for calls that must fail validation (or, with no
GPU present, the device check), so nothing here ever reaches a kernel.
"""
import ctypes
import os
import re

import pytest
import torch

from paper_2608_01528_amd import gramspace as gsm

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "gramspace.h")

P = ctypes.c_void_p
A1 = P(0x10000)       # distinct, well-aligned fake addresses
A2 = P(0x20000000)
A3 = P(0x40000000)
A4 = P(0x60000000)
WS = P(0x80000000)
NULL = None


def header_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(gs_\w+)\s*\(", src, flags=re.M)))


@pytest.fixture(scope="module")
def L():
    return gsm.lib()


def err(L):
    return L.gs_last_error().decode()


def test_exports_every_declared_function(L):
    names = header_functions()
    assert set(names) >= {"gs_compress", "gs_project", "gs_prob2vec", "gs_similarity",
                          "gs_attention", "gs_reconstruct", "gs_last_error", "gs_abi_version",
                          "gs_compress_workspace"}
    for n in names:
        assert hasattr(L, n), n


def test_abi_version_matches_header(L):
    v = int(re.search(r"#define GS_ABI_VERSION (\d+)", open(HEADER).read()).group(1))
    assert L.gs_abi_version() == v


def test_workspace_size(L):
    assert L.gs_compress_workspace(0, 10) == 0
    assert L.gs_compress_workspace(11, 10) == 0          # D < M unsupported
    a = L.gs_compress_workspace(10, 1024)
    b = L.gs_compress_workspace(2048, 16384)
    assert 0 < a < b
    assert b >= 2048 * 16384 * 8                          # fp64 master basis


def compress(L, C=A1, ct=gsm.GS_F32, M=10, D=64, ldc=64, tol=1e-10, Q=A2, qt=gsm.GS_F64, ldq=64,
             R=A3, rt=gsm.GS_F64, ldr=10, kept=NULL, cnorm=NULL, rank=True, ws=WS, wsb=None):
    rk = ctypes.c_int32(0)
    if wsb is None:
        wsb = L.gs_compress_workspace(M, D) if 1 <= M <= D else 1 << 20
    return L.gs_compress(C, ct, M, D, ldc, tol, Q, qt, ldq, R, rt, ldr, kept, cnorm,
                         ctypes.byref(rk) if rank else None, ws, wsb, None)


def test_compress_validation(L):
    assert compress(L, ct=7) == gsm.GS_ERR_DTYPE
    assert compress(L, rank=False) == gsm.GS_ERR_ARG
    assert compress(L, M=0) == gsm.GS_ERR_SHAPE
    assert compress(L, M=65, ldr=65) == gsm.GS_ERR_SHAPE and "gs_compress_partitioned" in err(L)
    assert compress(L, tol=1.5) == gsm.GS_ERR_ARG
    assert compress(L, tol=float("nan")) == gsm.GS_ERR_ARG
    assert compress(L, C=NULL) == gsm.GS_ERR_ARG and "C" in err(L)
    assert compress(L, ldc=63) == gsm.GS_ERR_SHAPE
    assert compress(L, ldr=9) == gsm.GS_ERR_SHAPE and "R" in err(L)
    assert compress(L, Q=P(0x20000004)) == gsm.GS_ERR_ALIGN            # f64 needs 8 bytes
    assert compress(L, ws=NULL) == gsm.GS_ERR_WORKSPACE
    assert compress(L, ws=P(0x80000010)) == gsm.GS_ERR_ALIGN
    assert compress(L, wsb=100) == gsm.GS_ERR_WORKSPACE and "needed" in err(L)
    assert compress(L, Q=A1) == gsm.GS_ERR_ARG and "overlaps" in err(L)   # output aliases input
    assert compress(L, kept=P(0x20000000 + 8)) == gsm.GS_ERR_ARG            # kept inside Q


def test_compress_partitioned_validation(L):
    ranks = (ctypes.c_int32 * 8)()
    rk = ctypes.c_int32(0)

    def call(M=100, D=32, subset=32, ct=gsm.GS_F32, ldc=32, Q=A2, ldq=32, R=A3, ldr=100, ws=WS, wsb=1 << 30,
             rank=True, rks=True):
        return L.gs_compress_partitioned(A1, ct, M, D, ldc, 1e-10, subset, Q, gsm.GS_F64, ldq, R, gsm.GS_F64, ldr,
                                         NULL, NULL, ranks if rks else None, ctypes.byref(rk) if rank else None,
                                         ws, wsb, None)
    assert call(ct=9) == gsm.GS_ERR_DTYPE
    assert call(rank=False) == gsm.GS_ERR_ARG and call(rks=False) == gsm.GS_ERR_ARG
    assert call(subset=0) == gsm.GS_ERR_SHAPE and call(subset=33) == gsm.GS_ERR_SHAPE
    assert call(ldr=99) == gsm.GS_ERR_SHAPE                              # R holds M x M
    assert call(ws=NULL) == gsm.GS_ERR_WORKSPACE
    assert call(wsb=16) == gsm.GS_ERR_WORKSPACE and "needed" in err(L)
    assert call(Q=A1) == gsm.GS_ERR_ARG                                   # Q over C
    # the workspace is sized by one subset, not by the whole codebook
    assert L.gs_compress_workspace(32, 32) < L.gs_compress_workspace(32, 32) * 2
    assert call(wsb=L.gs_compress_workspace(32, 32)) == gsm.GS_ERR_DEVICE  # valid: only the device is missing


def test_compress_padded_validation(L):
    rk = ctypes.c_int32(0)

    def call(M=10, D=64, k=20, ct=gsm.GS_F32, H=NULL, ldh=20, ldq=64, ldr=20, ws=WS, wsb=1 << 30, Q=A2, R=A3):
        return L.gs_compress_padded(A1, ct, M, D, 64, 1e-10, k, H, ldh, Q, gsm.GS_F64, ldq, R, gsm.GS_F64, ldr,
                                    NULL, NULL, ctypes.byref(rk), ws, wsb, None)
    assert call(ct=7) == gsm.GS_ERR_DTYPE
    assert call(k=9) == gsm.GS_ERR_SHAPE                     # k < M
    assert call(k=55) == gsm.GS_ERR_SHAPE                    # M + k > D
    assert call(ldr=19) == gsm.GS_ERR_SHAPE                  # R is M x k
    assert call(H=P(0x60000004)) == gsm.GS_ERR_ALIGN         # fp64 H
    assert call(ldh=19, H=A4) == gsm.GS_ERR_SHAPE
    assert call(wsb=100) == gsm.GS_ERR_WORKSPACE
    assert call(Q=A1) == gsm.GS_ERR_ARG
    assert L.gs_compress_padded_workspace(10, 64, 9) == 0 and L.gs_compress_padded_workspace(10, 64, 20) > 0
    assert call() == gsm.GS_ERR_DEVICE                       # valid: only the device is missing


def compress_noalloc(L, C=A1, ct=gsm.GS_F32, M=10, D=64, ldc=64, tol=1e-10, Q=A2, qt=gsm.GS_F64, ldq=64,
                     R=A3, rt=gsm.GS_F64, ldr=10, kept=NULL, cnorm=NULL, rank=True):
    rk = ctypes.c_int32(0)
    return L.gs_compress_noalloc(C, ct, M, D, ldc, tol, Q, qt, ldq, R, rt, ldr, kept, cnorm,
                                 ctypes.byref(rk) if rank else None, None)


def test_compress_noalloc_validation(L):
    # the same argument checks as gs_compress ...
    assert compress_noalloc(L, ct=7) == gsm.GS_ERR_DTYPE
    assert compress_noalloc(L, rank=False) == gsm.GS_ERR_ARG
    assert compress_noalloc(L, M=65, ldr=65) == gsm.GS_ERR_SHAPE
    assert compress_noalloc(L, ldc=63) == gsm.GS_ERR_SHAPE
    assert compress_noalloc(L, Q=A1) == gsm.GS_ERR_ARG and "overlaps" in err(L)
    # ... and codebooks whose workspace exceeds the static array are refused
    # before any device work
    big = L.gs_compress_workspace(2048, 16384)
    assert big > (64 << 20)
    assert compress_noalloc(L, M=2048, D=16384, ldc=16384, ldq=16384, ldr=2048, Q=P(0x100000000),
                            R=P(0x200000000)) == gsm.GS_ERR_WORKSPACE
    assert "scratch" in err(L)
    assert L.gs_compress_workspace(1000, 4096) <= (64 << 20)        # the binary workload's codebook fits


def test_prob2vec_sparse_validation(L):
    f = L.gs_prob2vec_sparse
    # rowptr, cols, vals, vt, B, M, nnz, R, rt, r, ldr, T, tt, ldt, stream
    ok = [A1, A2, A3, gsm.GS_F32, 4, 10, 6, A4, gsm.GS_F32, 10, 10, WS, gsm.GS_F32, 10, NULL]

    def call(**kw):
        a = list(ok)
        names = ["rowptr", "cols", "vals", "vt", "B", "M", "nnz", "R", "rt", "r", "ldr", "T", "tt", "ldt", "s"]
        for k, v in kw.items():
            a[names.index(k)] = v
        return f(*a)

    assert call(vt=gsm.GS_F64, rt=gsm.GS_F64) == gsm.GS_ERR_DTYPE
    assert call(rt=gsm.GS_BF16) == gsm.GS_ERR_DTYPE
    assert call(r=0) == gsm.GS_ERR_SHAPE
    assert call(M=0) == gsm.GS_ERR_SHAPE
    assert call(nnz=-1) == gsm.GS_ERR_SHAPE
    assert call(rowptr=NULL) == gsm.GS_ERR_ARG
    assert call(cols=NULL) == gsm.GS_ERR_ARG
    assert call(rowptr=P(0x10004)) == gsm.GS_ERR_ALIGN                  # int64 pointers
    assert call(ldt=9) == gsm.GS_ERR_SHAPE
    assert call(T=P(0x20000000 + 8)) == gsm.GS_ERR_ARG and "overlaps" in err(L)   # T on cols
    assert call(B=0, rowptr=NULL, T=NULL) == gsm.GS_OK                  # empty batch
    assert call(nnz=0, cols=NULL, vals=NULL, B=0) == gsm.GS_OK


def test_project_validation(L):
    f = L.gs_project
    # dtype mismatch X f32 / Q bf16
    assert f(A1, gsm.GS_F32, 4, 8, 8, A2, gsm.GS_BF16, 2, 8, A3, gsm.GS_F32, 2, NULL, NULL) == gsm.GS_ERR_DTYPE
    assert f(A1, gsm.GS_F64, 4, 8, 8, A2, gsm.GS_F64, 2, 8, A3, gsm.GS_F32, 2, NULL, NULL) == gsm.GS_ERR_DTYPE
    assert f(A1, gsm.GS_F32, 4, 8, 8, A2, gsm.GS_F32, 0, 8, A3, gsm.GS_F32, 2, NULL, NULL) == gsm.GS_ERR_SHAPE
    assert f(A1, gsm.GS_F32, 4, 8, 7, A2, gsm.GS_F32, 2, 8, A3, gsm.GS_F32, 2, NULL, NULL) == gsm.GS_ERR_SHAPE
    assert f(NULL, gsm.GS_F32, 4, 8, 8, A2, gsm.GS_F32, 2, 8, A3, gsm.GS_F32, 2, NULL, NULL) == gsm.GS_ERR_ARG
    assert f(A1, gsm.GS_F32, 4, 8, 8, A2, gsm.GS_F32, 2, 8, P(0x10004), gsm.GS_F32, 2, NULL, NULL) == gsm.GS_ERR_ARG
    assert f(A1, gsm.GS_F32, 4, 8, 8, A2, gsm.GS_F32, 2, 8, A3, gsm.GS_F32, 2, P(0x40000002), NULL) == gsm.GS_ERR_ALIGN
    # xnorm2 overlapping T
    assert f(A1, gsm.GS_F32, 4, 8, 8, A2, gsm.GS_F32, 2, 8, A3, gsm.GS_F32, 2, P(0x40000008), NULL) == gsm.GS_ERR_ARG
    # empty batch is a valid no-op that touches nothing
    assert f(A1, gsm.GS_F32, 0, 8, 8, A2, gsm.GS_F32, 2, 8, A3, gsm.GS_F32, 2, NULL, NULL) == gsm.GS_OK
    assert err(L) == ""


def test_prob2vec_validation(L):
    f = L.gs_prob2vec
    assert f(A1, gsm.GS_F32, 4, 5, 5, A2, gsm.GS_F32, 0, 6, A3, gsm.GS_F32, 6, NULL) == gsm.GS_ERR_SHAPE  # r = 0
    # r > M is a padded basis: valid (only the device is missing here)
    assert f(A1, gsm.GS_F32, 4, 5, 5, A2, gsm.GS_F32, 6, 6, A3, gsm.GS_F32, 6, NULL) == gsm.GS_ERR_DEVICE
    assert f(A1, gsm.GS_BF16, 4, 5, 5, A2, gsm.GS_F32, 5, 5, A3, gsm.GS_F32, 5, NULL) == gsm.GS_ERR_DTYPE
    assert f(A1, gsm.GS_F32, 4, 5, 4, A2, gsm.GS_F32, 5, 5, A3, gsm.GS_F32, 5, NULL) == gsm.GS_ERR_SHAPE
    assert f(A1, gsm.GS_F32, -1, 5, 5, A2, gsm.GS_F32, 5, 5, A3, gsm.GS_F32, 5, NULL) == gsm.GS_ERR_SHAPE
    assert f(A1, gsm.GS_F32, 0, 5, 5, A2, gsm.GS_F32, 5, 5, A3, gsm.GS_F32, 5, NULL) == gsm.GS_OK


def test_similarity_validation(L):
    f = L.gs_similarity
    ok = dict(T=A1, tt=gsm.GS_F32, B=4, r=5, ldt=5, R=A2, rt=gsm.GS_F32, M=5, ldr=5, qn=NULL, cn=NULL,
              mode=gsm.GS_SIM_COSINE, scale=1.0, S=A3, lds=5, am=A4)

    def call(**kw):
        a = dict(ok)
        a.update(kw)
        return f(a["T"], a["tt"], a["B"], a["r"], a["ldt"], a["R"], a["rt"], a["M"], a["ldr"], a["qn"],
                 a["cn"], a["mode"], a["scale"], a["S"], a["lds"], a["am"], NULL)

    assert call(mode=3) == gsm.GS_ERR_ARG
    assert call(S=NULL, am=NULL) == gsm.GS_ERR_ARG
    assert call(lds=4) == gsm.GS_ERR_SHAPE
    assert call(am=P(0x60000001)) == gsm.GS_ERR_ALIGN
    assert call(am=P(0x40000004)) == gsm.GS_ERR_ARG          # argmax inside S
    assert call(S=A1) == gsm.GS_ERR_ARG                      # S aliases T
    assert call(r=6) == gsm.GS_ERR_SHAPE                     # ldt < r
    assert call(r=0) == gsm.GS_ERR_SHAPE
    assert call(B=0) == gsm.GS_OK
    # r above M is the dense form of the lookup (D-space rows, uncompressed codebook)
    assert call(B=0, r=6, ldt=6, ldr=6) == gsm.GS_OK


def test_attention_and_reconstruct_validation(L):
    f = L.gs_attention
    base = [A1, gsm.GS_F32, 4, 5, 5, A2, gsm.GS_F32, 5, 5, NULL, NULL, gsm.GS_SIM_DOT, 1.0, 2.0]
    assert f(*base, NULL, 5, NULL, gsm.GS_F32, 5, NULL) == gsm.GS_ERR_ARG           # A required
    assert f(*base, A3, 5, A4, gsm.GS_F64, 5, NULL) == gsm.GS_ERR_DTYPE            # O f64
    assert f(*base, A3, 5, A4, gsm.GS_F32, 4, NULL) == gsm.GS_ERR_SHAPE            # ldo < r
    assert f(*base, A3, 5, A3, gsm.GS_F32, 5, NULL) == gsm.GS_ERR_ARG              # O aliases A
    g = L.gs_reconstruct
    assert g(A1, gsm.GS_F32, 4, 5, 5, NULL, 5, gsm.GS_BIND_MUL, A2, gsm.GS_F32, 16, 16, A3, gsm.GS_F32, 16,
             NULL) == gsm.GS_ERR_ARG                                               # T2 missing
    assert g(A1, gsm.GS_F32, 4, 5, 5, A4, 5, gsm.GS_BIND_NONE, A2, gsm.GS_F32, 16, 16, A3, gsm.GS_F32, 16,
             NULL) == gsm.GS_ERR_ARG                                               # T2 without bind
    assert g(A1, gsm.GS_F32, 4, 5, 5, NULL, 5, 9, A2, gsm.GS_F32, 16, 16, A3, gsm.GS_F32, 16,
             NULL) == gsm.GS_ERR_ARG
    assert g(A1, gsm.GS_F32, 4, 5, 5, NULL, 5, gsm.GS_BIND_NONE, A2, gsm.GS_BF16, 16, 16, A3, gsm.GS_F32, 16,
             NULL) == gsm.GS_ERR_DTYPE
    assert g(A1, gsm.GS_F32, 4, 5, 5, NULL, 5, gsm.GS_BIND_NONE, A2, gsm.GS_F32, 16, 16, A3, gsm.GS_F32, 15,
             NULL) == gsm.GS_ERR_SHAPE


def test_similarity_attention_validation(L):
    f = L.gs_similarity_attention
    base = [A1, gsm.GS_F32, 4, 5, 5, A2, gsm.GS_F32, 5, 5, NULL, NULL, gsm.GS_SIM_DOT, 1.0]
    assert f(*base, NULL, 5, NULL, 2.0, NULL, 5, NULL) == gsm.GS_ERR_ARG              # nothing asked for
    assert "all null" in err(L)
    assert f(*base, A3, 5, NULL, 2.0, A3, 5, NULL) == gsm.GS_ERR_ARG                  # A aliases S
    assert f(*base, A1, 5, NULL, 2.0, NULL, 5, NULL) == gsm.GS_ERR_ARG                # S aliases T
    assert f(*base, NULL, 5, NULL, 2.0, A2, 5, NULL) == gsm.GS_ERR_ARG                # A aliases R
    assert f(*base, A3, 4, NULL, 2.0, NULL, 5, NULL) == gsm.GS_ERR_SHAPE              # lds < M
    assert f(*base, NULL, 5, NULL, 2.0, A3, 4, NULL) == gsm.GS_ERR_SHAPE              # lda < M
    assert f(A1, gsm.GS_F32, 4, 5, 5, A2, gsm.GS_BF16, 5, 5, NULL, NULL, gsm.GS_SIM_DOT, 1.0,
             A3, 5, NULL, 2.0, NULL, 5, NULL) == gsm.GS_ERR_DTYPE                     # T/R types differ
    assert f(A1, gsm.GS_F32, 4, 5, 5, A2, gsm.GS_F32, 5, 5, NULL, NULL, 7, 1.0,
             A3, 5, NULL, 2.0, NULL, 5, NULL) == gsm.GS_ERR_ARG                       # unknown mode
    assert f(NULL, gsm.GS_F32, 0, 5, 5, A2, gsm.GS_F32, 5, 5, NULL, NULL, gsm.GS_SIM_DOT, 1.0,
             NULL, 5, NULL, 2.0, NULL, 5, NULL) == gsm.GS_OK                          # empty batch


def test_bind_coords_validation(L):
    f = L.gs_bind_coords
    # T (4 x 5), T2, Q (5 x 8), Z (4 x 5)
    ok = [A1, gsm.GS_F32, 4, 5, 5, A2, 5, A3, gsm.GS_F32, 8, 8, A4, gsm.GS_F32, 5, NULL]
    bad = list(ok); bad[1] = gsm.GS_BF16
    assert f(*bad) == gsm.GS_ERR_DTYPE and "f32" in err(L)                            # bf16 T
    bad = list(ok); bad[12] = gsm.GS_BF16
    assert f(*bad) == gsm.GS_ERR_DTYPE                                                # bf16 Z
    bad = list(ok); bad[3] = 257; bad[4] = 257; bad[6] = 257; bad[13] = 257
    assert f(*bad) == gsm.GS_ERR_SHAPE and "256" in err(L)                            # r > 256
    bad = list(ok); bad[4] = 4
    assert f(*bad) == gsm.GS_ERR_SHAPE                                                # ldt < r
    bad = list(ok); bad[10] = 7
    assert f(*bad) == gsm.GS_ERR_SHAPE                                                # ldq < D
    bad = list(ok); bad[11] = A1
    assert f(*bad) == gsm.GS_ERR_ARG                                                  # Z aliases T
    bad = list(ok); bad[5] = NULL
    assert f(*bad) == gsm.GS_ERR_ARG                                                  # no T2
    empty = list(ok); empty[0] = NULL; empty[2] = 0; empty[5] = NULL; empty[11] = NULL
    assert f(*empty) == gsm.GS_OK                                                     # empty batch


def test_wrappers_reject_mismatched_shapes():
    # operands whose shapes disagree with the sizes the wrapper passes would
    # be read or written past their ends: rejected before any call
    f = lambda *s: torch.zeros(*s)
    cases = [
        lambda: gsm.gs_project(f(4, 8), f(3, 7)),                              # Q columns != D
        lambda: gsm.gs_project(f(4, 8), f(3, 8), out=f(4, 2)),                 # out columns != r
        lambda: gsm.gs_prob2vec(f(4, 5), f(6, 3)),                             # R rows != M
        lambda: gsm.gs_similarity(f(4, 3), f(5, 2)),                           # R columns != r
        lambda: gsm.gs_similarity(f(4, 3), f(5, 3), qnorm2=f(3)),              # qnorm2 too short
        lambda: gsm.gs_attention(f(4, 3), f(5, 3), out=f(4, 4)),              # A columns != M
        lambda: gsm.gs_similarity_attention(f(4, 3), f(5, 3), a_out=f(3, 5)),  # A rows != B
        lambda: gsm.gs_reconstruct(f(4, 3), f(2, 8)),                          # Q rows != r
        lambda: gsm.gs_reconstruct(f(4, 3), f(3, 8), T2=f(4, 2), bind="mul"),  # T2 shape
        lambda: gsm.gs_bind_coords(f(4, 3), f(4, 3), f(2, 8)),                 # Q rows != r
        lambda: gsm.gs_bind_coords(f(4, 3), f(5, 3), f(3, 8)),                 # T2 shape
        lambda: gsm.gs_bind_restored(f(4, 8), f(4, 7)),                        # Y shape
    ]
    for c in cases:
        with pytest.raises(ValueError, match="must be|needs at least"):
            c()


def test_errors_are_per_thread(L):
    import threading
    assert compress(L, ct=7) == gsm.GS_ERR_DTYPE
    seen = []

    def other():
        seen.append(err(L))

    t = threading.Thread(target=other)
    t.start()
    t.join()
    assert seen == [""] and "element type" in err(L)


@pytest.mark.skipif(torch.cuda.device_count() > 0, reason="a GPU is present: valid fake pointers would reach a kernel")
def test_no_device_is_reported(L):
    # every argument valid: the only thing missing is a GPU
    assert L.gs_project(A1, gsm.GS_F32, 4, 8, 8, A2, gsm.GS_F32, 2, 8, A3, gsm.GS_F32, 2, NULL, NULL) == gsm.GS_ERR_DEVICE
    assert "device" in err(L)
    assert compress(L) == gsm.GS_ERR_DEVICE


def test_python_wrapper_raises_with_status():
    e = gsm.GramSpaceError(gsm.GS_ERR_SHAPE, "boom")
    assert e.status == gsm.GS_ERR_SHAPE and "GS_ERR_SHAPE" in str(e)


def test_empty_batch_accepts_null_buffers(L):
    # B == 0: batch-sized buffers may be null (torch gives empty tensors no storage)
    assert L.gs_similarity(NULL, gsm.GS_F32, 0, 4, 4, A2, gsm.GS_F32, 4, 4, NULL, NULL, gsm.GS_SIM_COSINE,
                           1.0, NULL, 4, NULL, NULL) == gsm.GS_OK
    assert L.gs_prob2vec(NULL, gsm.GS_F32, 0, 4, 4, A2, gsm.GS_F32, 4, 4, NULL, gsm.GS_F32, 4, NULL) == gsm.GS_OK
    assert L.gs_attention(NULL, gsm.GS_F32, 0, 4, 4, A2, gsm.GS_F32, 4, 4, NULL, NULL, gsm.GS_SIM_DOT, 1.0, 1.0,
                          NULL, 4, NULL, gsm.GS_F32, 4, NULL) == gsm.GS_OK
    assert L.gs_reconstruct(NULL, gsm.GS_F32, 0, 4, 4, NULL, 4, gsm.GS_BIND_NONE, A2, gsm.GS_F32, 8, 8, NULL,
                            gsm.GS_F32, 8, NULL) == gsm.GS_OK
    assert L.gs_project(NULL, gsm.GS_F32, 0, 8, 8, A2, gsm.GS_F32, 2, 8, NULL, gsm.GS_F32, 2, NULL, NULL) == gsm.GS_OK
    # ... but not the codebook
    assert L.gs_prob2vec(NULL, gsm.GS_F32, 0, 4, 4, NULL, gsm.GS_F32, 4, 4, NULL, gsm.GS_F32, 4, NULL) == gsm.GS_ERR_ARG


def soft(L, groups, ngroups=None, pt=gsm.GS_F32, tt=gsm.GS_F32, mode=gsm.GS_SIM_COSINE, form=gsm.GS_SOFT_AUTO):
    arr = (gsm.SoftGroup * max(1, len(groups)))()
    for i, g in enumerate(groups):
        for k, v in g.items():
            setattr(arr[i], k, v)
    n = len(groups) if ngroups is None else ngroups
    return L.gs_soft_select(arr, n, pt, tt, mode, 1.0, 1.0, form, None)


def group(**kw):
    g = dict(P=0x10000, ldp=10, R=0x200000, ldr=10, cnorm=None, B=5, M=10, r=10, T=None, ldt=10,
             S=0x400000, lds=10, argmax=None, A=None, lda=10)
    g.update(kw)
    return g


def test_soft_select_validation(L):
    assert L.gs_soft_select(None, 1, gsm.GS_F32, gsm.GS_F32, 1, 1.0, 1.0, gsm.GS_SOFT_AUTO, None) == gsm.GS_ERR_ARG
    assert soft(L, [group()], form=3) == gsm.GS_ERR_ARG                  # unknown form
    assert soft(L, [group(T=0x800000)], form=gsm.GS_SOFT_GRAM) == gsm.GS_ERR_ARG   # Gram form writes no T
    assert soft(L, [group()], ngroups=0) == gsm.GS_ERR_ARG
    assert soft(L, [group()] * 9) == gsm.GS_ERR_ARG                      # more than 8 groups
    assert soft(L, [group()], pt=gsm.GS_F64) == gsm.GS_ERR_DTYPE
    assert soft(L, [group()], mode=5) == gsm.GS_ERR_ARG
    assert soft(L, [group(M=33, ldp=33, r=33, ldr=33, lds=33)]) == gsm.GS_ERR_SHAPE  # beyond small codebooks
    assert soft(L, [group(r=11, ldr=11)]) == gsm.GS_ERR_SHAPE            # r > M
    assert soft(L, [group(ldp=9)]) == gsm.GS_ERR_SHAPE
    assert soft(L, [group(P=None)]) == gsm.GS_ERR_ARG
    assert soft(L, [group(A=0x400000 + 16)]) == gsm.GS_ERR_ARG           # A overlaps S
    assert soft(L, [group(), group(S=0x10000 + 40)]) == gsm.GS_ERR_ARG   # S of group 1 inside P of group 0
    assert soft(L, [group(argmax=0x600002)]) == gsm.GS_ERR_ALIGN
    assert soft(L, [group(B=0, P=None, S=None)]) == gsm.GS_OK            # empty: nothing to do
    assert "gs_" in err(L) or err(L) == ""


def test_bind_restored_validation(L):
    f = L.gs_bind_restored
    ok = dict(X=A1, xt=gsm.GS_F32, B=4, D=16, ldx=16, Y=A2, ldy=16, op=gsm.GS_BINDOP_CONV, Lb=8, Z=A3,
              zt=gsm.GS_F32, ldz=16)

    def call(**kw):
        a = dict(ok)
        a.update(kw)
        return f(a["X"], a["xt"], a["B"], a["D"], a["ldx"], a["Y"], a["ldy"], a["op"], a["Lb"], a["Z"], a["zt"],
                 a["ldz"], NULL)

    assert call(op=7) == gsm.GS_ERR_ARG
    assert call(xt=gsm.GS_F64) == gsm.GS_ERR_DTYPE
    assert call(Lb=6) == gsm.GS_ERR_SHAPE                     # not a power of two
    assert call(Lb=32) == gsm.GS_ERR_SHAPE                    # does not divide D
    assert call(Lb=1) == gsm.GS_ERR_SHAPE
    assert call(D=16384, ldx=16384, ldy=16384, ldz=16384, Lb=16384) == gsm.GS_ERR_SHAPE   # above 8192
    assert call(ldz=15) == gsm.GS_ERR_SHAPE
    assert call(Z=A1) == gsm.GS_ERR_ARG                       # Z aliases X
    assert call(B=0) == gsm.GS_OK
    assert call(B=0, op=gsm.GS_BINDOP_XOR, Lb=6) == gsm.GS_OK    # L is ignored by the element-wise operators
    assert err(L) == ""


def test_echelon_flag_validation(L):
    # GS_ECHELON is accepted on R of prob2vec, similarity and attention and
    # stripped before the type checks; other bits, or the flag elsewhere, are not
    e32, e16 = gsm.GS_F32 | gsm.GS_ECHELON, gsm.GS_BF16 | gsm.GS_ECHELON
    p = L.gs_prob2vec
    assert p(A1, gsm.GS_F32, 0, 5, 5, A2, e32, 5, 5, A3, gsm.GS_F32, 5, NULL) == gsm.GS_OK
    assert p(A1, gsm.GS_BF16, 0, 5, 8, A2, e16, 5, 8, A3, gsm.GS_BF16, 8, NULL) == gsm.GS_OK
    assert p(A1, gsm.GS_BF16, 4, 5, 5, A2, e32, 5, 5, A3, gsm.GS_F32, 5, NULL) == gsm.GS_ERR_DTYPE
    assert p(A1, gsm.GS_F32, 4, 5, 5, A2, gsm.GS_F32 | 0x200, 5, 5, A3, gsm.GS_F32, 5, NULL) == gsm.GS_ERR_DTYPE
    assert p(A1, e32, 4, 5, 5, A2, e32, 5, 5, A3, gsm.GS_F32, 5, NULL) == gsm.GS_ERR_DTYPE   # flag on P
    s = L.gs_similarity
    assert s(A1, gsm.GS_F32, 0, 5, 5, A2, e32, 5, 5, NULL, NULL, gsm.GS_SIM_COSINE, 1.0, A3, 5, A4,
             NULL) == gsm.GS_OK
    assert s(A1, gsm.GS_BF16, 4, 5, 5, A2, e32, 5, 5, NULL, NULL, gsm.GS_SIM_COSINE, 1.0, A3, 5, A4,
             NULL) == gsm.GS_ERR_DTYPE
    a = L.gs_attention
    assert a(A1, gsm.GS_F32, 0, 5, 5, A2, e32, 5, 5, NULL, NULL, gsm.GS_SIM_DOT, 1.0, 2.0, A3, 5, A4,
             gsm.GS_F32, 5, NULL) == gsm.GS_OK
    assert a(A1, gsm.GS_F32, 4, 5, 5, A2, gsm.GS_F64 | gsm.GS_ECHELON, 5, 5, NULL, NULL, gsm.GS_SIM_DOT, 1.0,
             2.0, A3, 5, A4, gsm.GS_F32, 5, NULL) == gsm.GS_ERR_DTYPE
    # not a coordinate argument of these calls
    assert L.gs_project(A1, gsm.GS_F32, 4, 8, 8, A2, e32, 2, 8, A3, gsm.GS_F32, 2, NULL,
                        NULL) == gsm.GS_ERR_DTYPE


def test_log_lines_for_rejected_calls():
    # GS_LOG is read once per process: run a rejected call in a child process
    import subprocess
    import sys
    code = ("import ctypes\nfrom paper_2608_01528_amd import gramspace as gsm\n"
            "L = gsm.lib()\n"
            "print(L.gs_prob2vec(None, gsm.GS_F32, 4, 4, 4, None, gsm.GS_F32, 4, 4, None, gsm.GS_F32, 4, None))\n")
    env = dict(os.environ, GS_LOG="1")
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, env=env, cwd=ROOT, timeout=120)
    assert r.returncode == 0, r.stderr
    assert r.stdout.strip() == str(gsm.GS_ERR_ARG)
    assert "[gramspace] status %d:" % gsm.GS_ERR_ARG in r.stderr
    env["GS_LOG"] = "0"
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, env=env, cwd=ROOT, timeout=120)
    assert "[gramspace]" not in r.stderr
