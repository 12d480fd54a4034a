"""Thin ctypes binding of the Gram-Space C ABI (include/gramspace.h).

Two layers with the C names:

* `lib()` returns the loaded shared library; its `gs_*` functions take raw
  pointers exactly as declared in the header.
* `gs_compress`, `gs_compress_padded`, `gs_compress_partitioned`, `gs_compress_noalloc`, `gs_project`, `gs_prob2vec`, `gs_prob2vec_sparse`,
  `gs_similarity`,
  `gs_attention`, `gs_similarity_attention`, `gs_reconstruct`, `gs_bind_coords`, `gs_soft_select` and `gs_bind_restored`
  below take torch tensors on the current
  GPU, allocate the outputs with torch, and pass pointers, sizes and the
  current stream to the library.  They only marshal arguments: every step of
  the computation runs in the library's HIP kernels.

Loading fails loudly (GramSpaceError) when libgramspace.so has not been
built; there is no fallback.
"""
from __future__ import annotations

import ctypes
import os

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libgramspace.so")

GS_OK, GS_ERR_ARG, GS_ERR_SHAPE, GS_ERR_DTYPE, GS_ERR_ALIGN, GS_ERR_WORKSPACE, \
    GS_ERR_NUMERIC, GS_ERR_DEVICE = range(8)
STATUS_NAMES = ["GS_OK", "GS_ERR_ARG", "GS_ERR_SHAPE", "GS_ERR_DTYPE", "GS_ERR_ALIGN",
                "GS_ERR_WORKSPACE", "GS_ERR_NUMERIC", "GS_ERR_DEVICE"]
GS_F32, GS_BF16, GS_F64 = 0, 1, 2
GS_SIM_DOT, GS_SIM_COSINE = 0, 1
GS_BIND_NONE, GS_BIND_MUL = 0, 1
GS_BINDOP_MUL, GS_BINDOP_XOR, GS_BINDOP_CONV, GS_BINDOP_CORR = 0, 1, 2, 3
GS_ECHELON = 0x100   # OR'ed into R's type: R[j, k] == 0 for k > j (as gs_compress returns it)
GS_SOFT_AUTO, GS_SOFT_GRAM, GS_SOFT_COORDS = 0, 1, 2

_DT = {torch.float32: GS_F32, torch.bfloat16: GS_BF16, torch.float64: GS_F64}


class GramSpaceError(RuntimeError):
    def __init__(self, status: int, msg: str):
        self.status = status
        name = STATUS_NAMES[status] if 0 <= status < len(STATUS_NAMES) else str(status)
        super().__init__("%s: %s" % (name, msg))


_lib = None

_vp, _i64, _i32p, _fp = ctypes.c_void_p, ctypes.c_int64, ctypes.POINTER(ctypes.c_int32), ctypes.c_void_p
_SIGS = {
    "gs_abi_version": ([], ctypes.c_int),
    "gs_last_error": ([], ctypes.c_char_p),
    "gs_compress_workspace": ([_i64, _i64], ctypes.c_size_t),
    "gs_compress": ([_vp, ctypes.c_int, _i64, _i64, _i64, ctypes.c_double,
                     _vp, ctypes.c_int, _i64, _vp, ctypes.c_int, _i64,
                     _vp, _vp, _i32p, _vp, ctypes.c_size_t, _vp], ctypes.c_int),
    "gs_compress_padded_workspace": ([_i64, _i64, _i64], ctypes.c_size_t),
    "gs_compress_padded": ([_vp, ctypes.c_int, _i64, _i64, _i64, ctypes.c_double, _i64, _vp, _i64,
                            _vp, ctypes.c_int, _i64, _vp, ctypes.c_int, _i64,
                            _vp, _vp, _i32p, _vp, ctypes.c_size_t, _vp], ctypes.c_int),
    "gs_compress_partitioned": ([_vp, ctypes.c_int, _i64, _i64, _i64, ctypes.c_double, _i64,
                                 _vp, ctypes.c_int, _i64, _vp, ctypes.c_int, _i64,
                                 _vp, _vp, _i32p, _i32p, _vp, ctypes.c_size_t, _vp], ctypes.c_int),
    "gs_compress_noalloc": ([_vp, ctypes.c_int, _i64, _i64, _i64, ctypes.c_double,
                             _vp, ctypes.c_int, _i64, _vp, ctypes.c_int, _i64,
                             _vp, _vp, _i32p, _vp], ctypes.c_int),
    "gs_project": ([_vp, ctypes.c_int, _i64, _i64, _i64, _vp, ctypes.c_int, _i64, _i64,
                    _vp, ctypes.c_int, _i64, _vp, _vp], ctypes.c_int),
    "gs_prob2vec": ([_vp, ctypes.c_int, _i64, _i64, _i64, _vp, ctypes.c_int, _i64, _i64,
                     _vp, ctypes.c_int, _i64, _vp], ctypes.c_int),
    "gs_similarity": ([_vp, ctypes.c_int, _i64, _i64, _i64, _vp, ctypes.c_int, _i64, _i64,
                       _vp, _vp, ctypes.c_int, ctypes.c_float, _vp, _i64, _vp, _vp], ctypes.c_int),
    "gs_attention": ([_vp, ctypes.c_int, _i64, _i64, _i64, _vp, ctypes.c_int, _i64, _i64,
                      _vp, _vp, ctypes.c_int, ctypes.c_float, ctypes.c_float, _vp, _i64,
                      _vp, ctypes.c_int, _i64, _vp], ctypes.c_int),
    "gs_similarity_attention": ([_vp, ctypes.c_int, _i64, _i64, _i64, _vp, ctypes.c_int, _i64, _i64,
                                 _vp, _vp, ctypes.c_int, ctypes.c_float, _vp, _i64, _vp,
                                 ctypes.c_float, _vp, _i64, _vp], ctypes.c_int),
    "gs_reconstruct": ([_vp, ctypes.c_int, _i64, _i64, _i64, _vp, _i64, ctypes.c_int,
                        _vp, ctypes.c_int, _i64, _i64, _vp, ctypes.c_int, _i64, _vp], ctypes.c_int),
}


class SoftGroup(ctypes.Structure):
    """Mirror of gs_soft_group."""
    _fields_ = [("P", _vp), ("ldp", _i64), ("R", _vp), ("ldr", _i64), ("cnorm", _vp),
                ("B", _i64), ("M", _i64), ("r", _i64), ("T", _vp), ("ldt", _i64),
                ("S", _vp), ("lds", _i64), ("argmax", _vp), ("A", _vp), ("lda", _i64)]


_SIGS["gs_prob2vec_sparse"] = ([_vp, _vp, _vp, ctypes.c_int, _i64, _i64, _i64, _vp, ctypes.c_int, _i64, _i64,
                                _vp, ctypes.c_int, _i64, _vp], ctypes.c_int)

_SIGS["gs_bind_restored"] = ([_vp, ctypes.c_int, _i64, _i64, _i64, _vp, _i64, ctypes.c_int, _i64,
                     _vp, ctypes.c_int, _i64, _vp], ctypes.c_int)

_SIGS["gs_bind_coords"] = ([_vp, ctypes.c_int, _i64, _i64, _i64, _vp, _i64, _vp, ctypes.c_int, _i64, _i64,
                           _vp, ctypes.c_int, _i64, _vp], ctypes.c_int)

_SIGS["gs_soft_select"] = ([ctypes.POINTER(SoftGroup), ctypes.c_int, ctypes.c_int, ctypes.c_int,
                            ctypes.c_int, ctypes.c_float, ctypes.c_float, ctypes.c_int, _vp], ctypes.c_int)


def lib():
    """The loaded libgramspace.so (raises GramSpaceError if it is not built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise GramSpaceError(GS_ERR_DEVICE, "libgramspace.so is not built (run "
                                 "paper_2608_01528_amd/build.py or __graft_entry__.build())")
        L = ctypes.CDLL(LIB_PATH)
        for name, (args, res) in _SIGS.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = res
        _lib = L
    return _lib


def _check(status: int):
    if status != GS_OK:
        raise GramSpaceError(status, lib().gs_last_error().decode())


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _mat(t: torch.Tensor, name: str):
    # an empty matrix has no layout to check (its strides are arbitrary)
    if t.dim() != 2 or (t.numel() > 0 and t.size(1) > 1 and t.stride(1) != 1):
        raise ValueError("%s must be a 2-D row-major tensor (unit column stride)" % name)
    if not t.is_cuda:
        raise ValueError("%s must be on the GPU" % name)
    if t.dtype not in _DT:
        raise ValueError("%s: unsupported dtype %s" % (name, t.dtype))
    if t.numel() == 0:
        return _DT[t.dtype], max(t.size(1), 1)
    return _DT[t.dtype], max(t.stride(0), t.size(1))


def _shape(t, name: str, rows=None, cols=None):
    """The library reads and writes the sizes it is given: an operand whose
    shape disagrees with them would be read or written past its end."""
    if t is None:
        return
    if t.dim() != 2 or (rows is not None and t.shape[0] != rows) or (cols is not None and t.shape[1] != cols):
        raise ValueError("%s must be %s x %s, got %s" % (name, "?" if rows is None else rows,
                                                         "?" if cols is None else cols, tuple(t.shape)))


def _vec(t, name: str, n: int):
    if t is not None and t.numel() < n:
        raise ValueError("%s needs at least %d entries, has %d" % (name, n, t.numel()))


def alloc_rows(rows: int, cols: int, dtype, device) -> torch.Tensor:
    """rows x cols matrix whose rows start on 16-byte boundaries (leading
    dimension rounded up to a multiple of 16 bytes).  bf16 operands laid out
    this way take the kernels' direct global-to-LDS load path."""
    per = 16 // torch.empty((), dtype=dtype).element_size()
    ld = max(1, (cols + per - 1) // per * per)
    return torch.empty((rows, ld), dtype=dtype, device=device)[:, :cols]


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _mode(mode):
    if mode in ("cosine", GS_SIM_COSINE):
        return GS_SIM_COSINE
    if mode in ("dot", GS_SIM_DOT):
        return GS_SIM_DOT
    raise ValueError("mode must be 'cosine' or 'dot'")


def compress_workspace_bytes(M: int, D: int) -> int:
    return int(lib().gs_compress_workspace(M, D))


def gs_compress(C: torch.Tensor, tol: float = 1e-10, q_dtype=torch.float64, r_dtype=torch.float64,
                workspace: torch.Tensor | None = None):
    """Compress codebook C (M x D).  Returns (Q, R, rank, kept, cnorm) with
    Q rank x D, R M x rank, kept int32[rank], cnorm float32[M] (all views of
    full-capacity buffers)."""
    ct, ldc = _mat(C, "C")
    M, D = C.shape
    dev = C.device
    Q = alloc_rows(M, D, q_dtype, dev)
    R = alloc_rows(M, M, r_dtype, dev)
    kept = torch.empty(M, dtype=torch.int32, device=dev)
    cnorm = torch.empty(M, dtype=torch.float32, device=dev)
    need = compress_workspace_bytes(M, D)
    if workspace is None:
        workspace = torch.empty(max(need, 1) + 256, dtype=torch.uint8, device=dev)
    base = workspace.data_ptr()
    off = (-base) % 256
    rank = ctypes.c_int32(0)
    _check(lib().gs_compress(_ptr(C), ct, M, D, ldc, float(tol), _ptr(Q), _DT[q_dtype], Q.stride(0),
                             _ptr(R), _DT[r_dtype], R.stride(0), _ptr(kept), _ptr(cnorm), ctypes.byref(rank),
                             ctypes.c_void_p(base + off), workspace.numel() - off, _stream()))
    r = rank.value
    return Q[:r], R[:, :r], r, kept[:r], cnorm


def gs_compress_partitioned(C: torch.Tensor, subset: int | None = None, tol: float = 1e-10,
                            q_dtype=torch.float64, r_dtype=torch.float64, workspace: torch.Tensor | None = None):
    """Compress codebook C (M x D, any M) in consecutive subsets of `subset`
    rows (default D).  Returns (Q, R, rank, ranks, kept, cnorm): Q the stacked
    bases (rank x D), R (M x rank) block diagonal, ranks the subsets' ranks."""
    ct, ldc = _mat(C, "C")
    M, D = C.shape
    subset = D if subset is None else int(subset)
    dev = C.device
    Q = alloc_rows(M, D, q_dtype, dev)
    R = alloc_rows(M, M, r_dtype, dev)
    kept = torch.empty(M, dtype=torch.int32, device=dev)
    cnorm = torch.empty(M, dtype=torch.float32, device=dev)
    need = compress_workspace_bytes(min(subset, M), D)
    if workspace is None:
        workspace = torch.empty(max(need, 1) + 256, dtype=torch.uint8, device=dev)
    base = workspace.data_ptr()
    off = (-base) % 256
    nsub = (M + subset - 1) // subset
    ranks = (ctypes.c_int32 * nsub)()
    rank = ctypes.c_int32(0)
    _check(lib().gs_compress_partitioned(_ptr(C), ct, M, D, ldc, float(tol), subset, _ptr(Q), _DT[q_dtype],
                                         Q.stride(0), _ptr(R), _DT[r_dtype], R.stride(0), _ptr(kept), _ptr(cnorm),
                                         ranks, ctypes.byref(rank), ctypes.c_void_p(base + off),
                                         workspace.numel() - off, _stream()))
    r = rank.value
    return Q[:r], R[:, :r], r, list(ranks), kept[:r], cnorm


def gs_compress_padded(C: torch.Tensor, k: int, H: torch.Tensor | None = None, tol: float = 1e-10,
                       q_dtype=torch.float64, r_dtype=torch.float64, workspace: torch.Tensor | None = None):
    """Basis of k >= M vectors (the codebook's, completed by unit vectors),
    optionally transformed by an orthogonal k x k fp64 matrix H.  Returns
    (Q k x D, R M x k, rank, kept, cnorm)."""
    ct, ldc = _mat(C, "C")
    M, D = C.shape
    dev = C.device
    Q = alloc_rows(k, D, q_dtype, dev)
    R = alloc_rows(M, k, r_dtype, dev)
    kept = torch.empty(M, dtype=torch.int32, device=dev)
    cnorm = torch.empty(M, dtype=torch.float32, device=dev)
    ldh = k
    if H is not None:
        if H.dtype != torch.float64:
            raise ValueError("H must be float64")
        _, ldh = _mat(H, "H")
    need = int(lib().gs_compress_padded_workspace(M, D, k))
    if workspace is None:
        workspace = torch.empty(max(need, 1) + 256, dtype=torch.uint8, device=dev)
    base = workspace.data_ptr()
    off = (-base) % 256
    rank = ctypes.c_int32(0)
    _check(lib().gs_compress_padded(_ptr(C), ct, M, D, ldc, float(tol), int(k), _ptr(H), ldh, _ptr(Q), _DT[q_dtype],
                                    Q.stride(0), _ptr(R), _DT[r_dtype], R.stride(0), _ptr(kept), _ptr(cnorm),
                                    ctypes.byref(rank), ctypes.c_void_p(base + off), workspace.numel() - off,
                                    _stream()))
    return Q, R, rank.value, kept, cnorm


def gs_compress_noalloc(C: torch.Tensor, tol: float = 1e-10, q_dtype=torch.float64, r_dtype=torch.float64,
                        out=None):
    """gs_compress without a workspace (the library's static scratch array).
    `out` = (Q, R, kept, cnorm) full-capacity buffers (Q M x D, R M x M) to
    write into; allocated here when None.  Returns (Q, R, rank, kept, cnorm)
    as gs_compress does."""
    ct, ldc = _mat(C, "C")
    M, D = C.shape
    dev = C.device
    if out is None:
        out = (alloc_rows(M, D, q_dtype, dev), alloc_rows(M, M, r_dtype, dev),
               torch.empty(M, dtype=torch.int32, device=dev), torch.empty(M, dtype=torch.float32, device=dev))
    Q, R, kept, cnorm = out
    qt, ldq = _mat(Q, "Q")
    rt, ldr = _mat(R, "R")
    rank = ctypes.c_int32(0)
    _check(lib().gs_compress_noalloc(_ptr(C), ct, M, D, ldc, float(tol), _ptr(Q), qt, ldq, _ptr(R), rt, ldr,
                                     _ptr(kept), _ptr(cnorm), ctypes.byref(rank), _stream()))
    r = rank.value
    return Q[:r], R[:, :r], r, kept[:r], cnorm


def gs_project(X: torch.Tensor, Q: torch.Tensor, out_dtype=None, xnorm2: bool = False,
               out: torch.Tensor | None = None, xnorm2_out: torch.Tensor | None = None):
    """T = X Q^T (and ||x_b||^2 if xnorm2)."""
    _shape(X, "X")
    _shape(Q, "Q", cols=X.shape[1])
    _shape(out, "out", X.shape[0], Q.shape[0])
    _vec(xnorm2_out, "xnorm2_out", X.shape[0])
    xt, ldx = _mat(X, "X")
    qt, ldq = _mat(Q, "Q")
    B, D = X.shape
    r = Q.shape[0]
    if out is None:
        out = alloc_rows(B, r, out_dtype or X.dtype, X.device)
    tt, ldt = _mat(out, "T")
    xn = None
    if xnorm2:
        xn = xnorm2_out if xnorm2_out is not None else torch.empty(B, dtype=torch.float32, device=X.device)
    _check(lib().gs_project(_ptr(X), xt, B, D, ldx, _ptr(Q), qt, r, ldq, _ptr(out), tt, ldt,
                            _ptr(xn), _stream()))
    return (out, xn) if xnorm2 else out


def gs_prob2vec(P: torch.Tensor, R: torch.Tensor, out_dtype=None, out: torch.Tensor | None = None,
                echelon: bool = False):
    """T = P R: Gram-loc of sum_j P[b, j] c_j.  echelon: R is lower echelon
    (as gs_compress returns it), so its zero blocks may be skipped."""
    _shape(P, "P")
    _shape(R, "R", rows=P.shape[1])
    _shape(out, "out", P.shape[0], R.shape[1])
    pt, ldp = _mat(P, "P")
    rt, ldr = _mat(R, "R")
    rt |= GS_ECHELON if echelon else 0
    B, M = P.shape
    r = R.shape[1]
    if out is None:
        out = alloc_rows(B, r, out_dtype or P.dtype, P.device)
    tt, ldt = _mat(out, "T")
    _check(lib().gs_prob2vec(_ptr(P), pt, B, M, ldp, _ptr(R), rt, r, ldr, _ptr(out), tt, ldt, _stream()))
    return out


def gs_prob2vec_sparse(rowptr: torch.Tensor, cols: torch.Tensor, vals: torch.Tensor, R: torch.Tensor,
                       out_dtype=None, out: torch.Tensor | None = None):
    """T = P R for P in compressed sparse row form: rowptr (int64, B + 1),
    cols (int32, nnz), vals (nnz, the type of R)."""
    if rowptr.dtype != torch.int64 or cols.dtype != torch.int32:
        raise ValueError("rowptr must be int64 and cols int32")
    if vals.numel() != cols.numel():
        raise ValueError("vals and cols must have the same length")
    _shape(R, "R")
    _shape(out, "out", rowptr.numel() - 1, R.shape[1])
    rt, ldr = _mat(R, "R")
    M, r = R.shape
    B = rowptr.numel() - 1
    if out is None:
        out = alloc_rows(B, r, out_dtype or R.dtype, R.device)
    tt, ldt = _mat(out, "T")
    _check(lib().gs_prob2vec_sparse(_ptr(rowptr), _ptr(cols), _ptr(vals), _DT[vals.dtype], B, M, cols.numel(),
                                    _ptr(R), rt, r, ldr, _ptr(out), tt, ldt, _stream()))
    return out


def gs_similarity(T: torch.Tensor, R: torch.Tensor, qnorm2=None, cnorm=None, mode="cosine",
                  scale: float = 1.0, scores: bool = True, argmax: bool = True,
                  out: torch.Tensor | None = None, argmax_out: torch.Tensor | None = None,
                  echelon: bool = False):
    """Scores S (B x M, fp32) and row argmax (int32) of T against R
    (echelon: as in gs_prob2vec)."""
    _shape(T, "T")
    _shape(R, "R", cols=T.shape[1])
    _shape(out if scores else None, "out", T.shape[0], R.shape[0])
    _vec(argmax_out if argmax else None, "argmax_out", T.shape[0])
    _vec(qnorm2, "qnorm2", T.shape[0])
    _vec(cnorm, "cnorm", R.shape[0])
    tt, ldt = _mat(T, "T")
    rt, ldr = _mat(R, "R")
    rt |= GS_ECHELON if echelon else 0
    B, r = T.shape
    M = R.shape[0]
    S = None
    if scores:
        S = out if out is not None else torch.empty((B, M), dtype=torch.float32, device=T.device)
    idx = None
    if argmax:
        idx = argmax_out if argmax_out is not None else torch.empty(B, dtype=torch.int32, device=T.device)
    lds = _mat(S, "S")[1] if S is not None else M
    _check(lib().gs_similarity(_ptr(T), tt, B, r, ldt, _ptr(R), rt, M, ldr, _ptr(qnorm2), _ptr(cnorm),
                               _mode(mode), float(scale), _ptr(S), lds, _ptr(idx), _stream()))
    return S, idx


def gs_attention(T: torch.Tensor, R: torch.Tensor, qnorm2=None, cnorm=None, mode="cosine",
                 scale: float = 1.0, beta: float = 1.0, weighted_sum: bool = False, out_dtype=None,
                 out: torch.Tensor | None = None, o_out: torch.Tensor | None = None,
                 echelon: bool = False):
    """Attention weights A = softmax(beta * S) (B x M, fp32) and optionally the
    weighted sum O = A R (B x r) (echelon: as in gs_prob2vec)."""
    _shape(T, "T")
    _shape(R, "R", cols=T.shape[1])
    _shape(out, "out", T.shape[0], R.shape[0])
    _shape(o_out if weighted_sum else None, "o_out", T.shape[0], T.shape[1])
    _vec(qnorm2, "qnorm2", T.shape[0])
    _vec(cnorm, "cnorm", R.shape[0])
    tt, ldt = _mat(T, "T")
    rt, ldr = _mat(R, "R")
    rt |= GS_ECHELON if echelon else 0
    B, r = T.shape
    M = R.shape[0]
    A = out if out is not None else torch.empty((B, M), dtype=torch.float32, device=T.device)
    _, lda = _mat(A, "A")
    O, ot, ldo = None, GS_F32, r
    if weighted_sum:
        O = o_out if o_out is not None else alloc_rows(B, r, out_dtype or T.dtype, T.device)
        ot, ldo = _mat(O, "O")
    _check(lib().gs_attention(_ptr(T), tt, B, r, ldt, _ptr(R), rt, M, ldr, _ptr(qnorm2), _ptr(cnorm),
                              _mode(mode), float(scale), float(beta), _ptr(A), lda, _ptr(O), ot, ldo,
                              _stream()))
    return A, O


def gs_similarity_attention(T: torch.Tensor, R: torch.Tensor, qnorm2=None, cnorm=None, mode="cosine",
                            scale: float = 1.0, beta: float = 1.0, scores: bool = True, argmax: bool = True,
                            attention: bool = True, out: torch.Tensor | None = None,
                            argmax_out: torch.Tensor | None = None, a_out: torch.Tensor | None = None,
                            echelon: bool = False):
    """Scores S, row argmax and attention weights A = softmax(beta * S) from
    one evaluation of the scores; each of the three may be switched off
    (None is returned in its place)."""
    _shape(T, "T")
    _shape(R, "R", cols=T.shape[1])
    _shape(out if scores else None, "out", T.shape[0], R.shape[0])
    _shape(a_out if attention else None, "a_out", T.shape[0], R.shape[0])
    _vec(argmax_out if argmax else None, "argmax_out", T.shape[0])
    _vec(qnorm2, "qnorm2", T.shape[0])
    _vec(cnorm, "cnorm", R.shape[0])
    tt, ldt = _mat(T, "T")
    rt, ldr = _mat(R, "R")
    rt |= GS_ECHELON if echelon else 0
    B, r = T.shape
    M = R.shape[0]
    S = idx = A = None
    if scores:
        S = out if out is not None else torch.empty((B, M), dtype=torch.float32, device=T.device)
    if argmax:
        idx = argmax_out if argmax_out is not None else torch.empty(B, dtype=torch.int32, device=T.device)
    if attention:
        A = a_out if a_out is not None else torch.empty((B, M), dtype=torch.float32, device=T.device)
    lds = _mat(S, "S")[1] if S is not None else M
    lda = _mat(A, "A")[1] if A is not None else M
    _check(lib().gs_similarity_attention(_ptr(T), tt, B, r, ldt, _ptr(R), rt, M, ldr, _ptr(qnorm2),
                                         _ptr(cnorm), _mode(mode), float(scale), _ptr(S), lds, _ptr(idx),
                                         float(beta), _ptr(A), lda, _stream()))
    return S, idx, A


def gs_reconstruct(T: torch.Tensor, Q: torch.Tensor, T2: torch.Tensor | None = None, bind=None,
                   out_dtype=None, out: torch.Tensor | None = None):
    """X = T Q, or (T Q) .* (T2 Q) with bind='mul'."""
    _shape(T, "T")
    _shape(Q, "Q", rows=T.shape[1])
    _shape(T2, "T2", T.shape[0], T.shape[1])
    _shape(out, "out", T.shape[0], Q.shape[1])
    tt, ldt = _mat(T, "T")
    qt, ldq = _mat(Q, "Q")
    B, r = T.shape
    D = Q.shape[1]
    b = GS_BIND_NONE
    ldt2 = r
    if bind in ("mul", GS_BIND_MUL):
        b = GS_BIND_MUL
        _, ldt2 = _mat(T2, "T2")
    elif bind not in (None, "none", GS_BIND_NONE):
        raise ValueError("bind must be None or 'mul'")
    if out is None:
        out = alloc_rows(B, D, out_dtype or T.dtype, T.device)
    xt, ldx = _mat(out, "X")
    _check(lib().gs_reconstruct(_ptr(T), tt, B, r, ldt, _ptr(T2), ldt2, b, _ptr(Q), qt, D, ldq,
                                _ptr(out), xt, ldx, _stream()))
    return out


def gs_bind_coords(T: torch.Tensor, T2: torch.Tensor, Q: torch.Tensor, out: torch.Tensor | None = None):
    """Z = ((T Q) .* (T2 Q)) Q^T in one pass (fp32, r <= 256)."""
    _shape(T, "T")
    _shape(T2, "T2", T.shape[0], T.shape[1])
    _shape(Q, "Q", rows=T.shape[1])
    _shape(out, "out", T.shape[0], T.shape[1])
    tt, ldt = _mat(T, "T")
    _, ldt2 = _mat(T2, "T2")
    qt, ldq = _mat(Q, "Q")
    B, r = T.shape
    D = Q.shape[1]
    if out is None:
        out = alloc_rows(B, r, T.dtype, T.device)
    zt, ldz = _mat(out, "Z")
    _check(lib().gs_bind_coords(_ptr(T), tt, B, r, ldt, _ptr(T2), ldt2, _ptr(Q), qt, D, ldq,
                                _ptr(out), zt, ldz, _stream()))
    return out


_BINDOPS = {"mul": GS_BINDOP_MUL, "xor": GS_BINDOP_XOR, "conv": GS_BINDOP_CONV, "corr": GS_BINDOP_CORR}


def gs_bind_restored(X: torch.Tensor, Y: torch.Tensor, op: str = "conv", L: int | None = None, out_dtype=None,
            out: torch.Tensor | None = None):
    """Binding of restored vectors row by row: 'mul' (element-wise product),
    'xor' (binary vectors), 'conv' / 'corr' (blockwise circular convolution /
    correlation over blocks of L values, L = D by default)."""
    _shape(X, "X")
    _shape(Y, "Y", X.shape[0], X.shape[1])
    _shape(out, "out", X.shape[0], X.shape[1])
    xt, ldx = _mat(X, "X")
    _, ldy = _mat(Y, "Y")
    B, D = X.shape
    if out is None:
        out = alloc_rows(B, D, out_dtype or X.dtype, X.device)
    zt, ldz = _mat(out, "Z")
    _check(lib().gs_bind_restored(_ptr(X), xt, B, D, ldx, _ptr(Y), ldy, _BINDOPS[op], int(L or D), _ptr(out), zt, ldz,
                         _stream()))
    return out


def soft_groups(groups):
    """Build the gs_soft_group array for gs_soft_select from dicts with keys
    P, R and optionally cnorm, T, S, argmax, A (torch tensors).  Returns the
    ctypes array and the element types (pt, tt)."""
    arr = (SoftGroup * len(groups))()
    pt = tt = None
    for i, g in enumerate(groups):
        P, R = g["P"], g["R"]
        p_t, ldp = _mat(P, "P")
        _, ldr = _mat(R, "R")
        pt = p_t
        d = arr[i]
        d.P, d.ldp, d.R, d.ldr = P.data_ptr(), ldp, R.data_ptr(), ldr
        d.cnorm = g["cnorm"].data_ptr() if g.get("cnorm") is not None else None
        d.B, d.M, d.r = P.shape[0], P.shape[1], R.shape[1]
        if g.get("T") is not None:
            t_t, d.ldt = _mat(g["T"], "T")
            d.T, tt = g["T"].data_ptr(), t_t
        else:
            d.T, d.ldt = None, R.shape[1]
        for key, ld in (("S", "lds"), ("A", "lda")):
            if g.get(key) is not None:
                _, l = _mat(g[key], key)
                setattr(d, key, g[key].data_ptr())
                setattr(d, ld, l)
            else:
                setattr(d, key, None)
                setattr(d, ld, P.shape[1])
        d.argmax = g["argmax"].data_ptr() if g.get("argmax") is not None else None
    return arr, pt, (tt if tt is not None else GS_F32)


_SOFT_FORMS = {"auto": GS_SOFT_AUTO, "gram": GS_SOFT_GRAM, "coords": GS_SOFT_COORDS}


def gs_soft_select(groups, mode="cosine", scale: float = 1.0, beta: float = 1.0, prepared=None, form="auto"):
    """Fused prob2vec -> similarity/argmax -> attention over several small
    codebooks in one launch.  `groups` is a list of dicts (see soft_groups);
    outputs named in the dicts are written in place.  form: 'coords' (t = p R
    per row), 'gram' (scores through R R^T, no coordinates) or 'auto'."""
    arr, pt, tt = prepared if prepared is not None else soft_groups(groups)
    _check(lib().gs_soft_select(arr, len(arr), pt, tt, _mode(mode), float(scale), float(beta),
                                _SOFT_FORMS[form], _stream()))
