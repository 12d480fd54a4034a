"""Gram-Space oracle: a plain fp64 CPU reference of the method's operators.

TEST INFRASTRUCTURE ONLY.  Only the test-suite, the package's smoke check and
the CPU-baseline leg of the benchmark may import this package.  It shares no
code with the HIP library (no headers, kernels, helpers or constants) and never
imports it.

What each function computes, in the paper's terms (codebook C holds the
paper's W transposed: row j is codebook vector c_j; Q = U^T; R = T^T):

* compress     -- Sec. 3.1 Eq. 1 and Sec. 3.2: orthonormal basis of the span of
                  the codebook, rank = algebraic rank, built by Householder QR
                  (the paper's finite-precision construction) with column
                  skipping; C = R Q, R lower-echelon with positive pivots.
* compress_padded -- Sec. 3.1 (k > M): the basis completed by unit vectors,
                  coordinates zero-padded, then an optional orthogonal
                  transformation H of both.
* prob2vec     -- Sec. 2.2: v = sum_j p_j c_j, dense in D-space.
* similarity   -- Sec. 2.2, Sec. 3.2 Eq. 2-3: scaled dot product or cosine of
                  a query with every codebook vector, dense in D-space.
* argmax       -- lowest index on an exact tie.
* softmax      -- Sec. 2.2 attention score: softmax over the M scores.
* project      -- Sec. 3.1: t = U^T x.
* reconstruct  -- Sec. 3.1 and 3.3: x = U t ("decompose").
* bind         -- Sec. 2.2 / Table 1: element-wise product in D-space.
* circular     -- Sec. 2.2, Sec. 3.3: blockwise circular convolution (bind)
                  and circular correlation (unbind) of restored vectors, the
                  modulo-style component-wise operators, by their sums.
* xor          -- exclusive-or binding of binary vectors (bits value >= 0.5).
* memory_model -- Sec. 3.1: storage O(MD) against O(Dk + Mk), ratio D/k.

The C part (gs_oracle.c) is compiled with gcc -O2 for the baseline x86-64
target: no FMA contraction, every sum in index order.  Parallelism is over
independent rows only, so results do not depend on the thread count.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "gs_oracle.c")
_LIB = os.path.join(_HERE, "_liboracle.so")
_lib = None

DOT = 0
COSINE = 1


def build(force: bool = True) -> str:
    """Compile the C oracle into oracle/_liboracle.so with gcc."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(
            ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp",
             "-ffp-contract=off", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB):
        build(force=False)
    _lib = _bind(ctypes.CDLL(_LIB))
    return _lib


def use_native_build() -> str:
    """For timing only: compile the same source on the running machine with
    gcc -O3 -march=native (still no FMA contraction and no reassociation, so
    every sum keeps its order), check on a small case that it returns bit for
    bit what the tested build returns, and use it from then on.  Falls back to
    the tested build if compilation or the check fails.  Returns the flags of
    the build in use."""
    global _lib
    import tempfile
    base = "gcc -O2 -fopenmp -ffp-contract=off"
    ref = _load()
    try:
        d = tempfile.mkdtemp(prefix="gs_oracle_")
        path = os.path.join(d, "liboracle_native.so")
        subprocess.check_call(["gcc", "-O3", "-march=native", "-std=c11", "-fPIC", "-shared", "-fopenmp",
                               "-ffp-contract=off", _SRC, "-o", path, "-lm"],
                              stdout=subprocess.DEVNULL, stderr=subprocess.DEVNULL)
        native = _bind(ctypes.CDLL(path))
    except (OSError, subprocess.CalledProcessError):
        return base
    g = np.random.default_rng(0)
    X, C, P = g.standard_normal((3, 257)), g.standard_normal((5, 257)), g.random((3, 5))
    outs = []
    for lib in (ref, native):
        _lib = lib
        S = similarity(X, C, COSINE)
        outs.append((S, softmax(S, 3.0), prob2vec(P, C), project(X, C), reconstruct(P, C)))
    same = all(np.array_equal(a, b) for a, b in zip(*outs))
    _lib = native if same else ref
    return "gcc -O3 -march=native -fopenmp -ffp-contract=off" if same else base


def _bind(lib):
    dp = ctypes.POINTER(ctypes.c_double)
    ip = ctypes.POINTER(ctypes.c_int)
    L = ctypes.c_long
    lib.gso_threads.restype = ctypes.c_int
    lib.gso_set_threads.argtypes = [ctypes.c_int]
    lib.gso_compress.argtypes = [dp, L, L, ctypes.c_double, dp, dp, ip, ip]
    lib.gso_compress.restype = ctypes.c_int
    lib.gso_prob2vec.argtypes = [dp, L, L, dp, L, dp]
    lib.gso_row_norms.argtypes = [dp, L, L, dp]
    lib.gso_similarity.argtypes = [dp, L, L, dp, L, ctypes.c_int, ctypes.c_double, dp]
    lib.gso_argmax.argtypes = [dp, L, L, ip]
    lib.gso_softmax.argtypes = [dp, L, L, ctypes.c_double, dp]
    lib.gso_project.argtypes = [dp, L, L, dp, L, dp]
    lib.gso_reconstruct.argtypes = [dp, L, L, dp, L, dp]
    lib.gso_bind.argtypes = [dp, dp, L, dp]
    lib.gso_circular.argtypes = [dp, dp, L, L, L, ctypes.c_int, dp]
    lib.gso_xor.argtypes = [dp, dp, L, dp]
    return lib


def _f64(a) -> np.ndarray:
    a = np.asarray(a)
    if a.dtype != np.float64:
        a = a.astype(np.float64)  # exact for fp32 and bf16-valued inputs
    return np.ascontiguousarray(a)


def _dp(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def threads() -> int:
    return _load().gso_threads()


def set_threads(n: int) -> None:
    _load().gso_set_threads(int(n))


def compress(C, tau: float = 1e-10):
    """Householder compress of the M x D codebook C.

    Returns (Q, R, kept, rank): Q is rank x D with orthonormal rows, R is
    M x rank with C = R Q, kept lists the codebook rows that produced each
    basis vector (first occurrence wins, index order)."""
    C = _f64(C)
    M, D = C.shape
    Q = np.zeros((max(M, 1), D), np.float64)
    R = np.zeros((max(M, 1), max(M, 1)), np.float64)
    kept = np.zeros(max(M, 1), np.int32)
    rank = ctypes.c_int(0)
    rc = _load().gso_compress(_dp(C), M, D, float(tau), _dp(Q), _dp(R),
                              kept.ctypes.data_as(ctypes.POINTER(ctypes.c_int)),
                              ctypes.byref(rank))
    if rc != 0:
        raise MemoryError("oracle compress: allocation failed")
    r = rank.value
    return Q[:r].copy(), R[:M, :r].copy(), kept[:r].copy(), r


def compress_padded(C, k: int, H=None, tau: float = 1e-10):
    """Basis of k vectors (Sec. 3.1, k > M): the codebook's basis completed by
    the unit vectors e_0, e_1, ... in index order (each kept when it leaves the
    span built so far), the codebook's coordinates zero-padded; then, with an
    orthogonal k x k matrix H, Q' = H Q and R' = R H^T.  The completion is
    the Householder compression of the codebook followed by the unit rows.
    Returns (Q' k x D, R' M x k, kept, rank) with kept / rank those of the
    codebook itself."""
    C = _f64(C)
    M, D = C.shape
    aug = np.vstack([C, np.eye(D)[:k]])
    Qa, Ra, kept_a, ra = compress(aug, tau)
    if ra < k:
        raise ValueError("the unit rows did not complete the basis to k vectors")
    Qk = Qa[:k]
    Rk = Ra[:M, :k]
    r = int(np.sum(kept_a < M))
    if H is not None:
        H = _f64(H)
        Qk = H @ Qk
        Rk = Rk @ H.T
    return Qk, Rk, kept_a[:r].copy(), r


def prob2vec(P, C) -> np.ndarray:
    """Dense v_b = sum_j P[b, j] c_j (B x D)."""
    P, C = _f64(P), _f64(C)
    B, M = P.shape
    M2, D = C.shape
    assert M == M2
    V = np.empty((B, D), np.float64)
    _load().gso_prob2vec(_dp(P), B, M, _dp(C), D, _dp(V))
    return V


def row_norms(X) -> np.ndarray:
    X = _f64(X)
    B, D = X.shape
    out = np.empty(B, np.float64)
    _load().gso_row_norms(_dp(X), B, D, _dp(out))
    return out


def similarity(X, C, mode: int = COSINE, scale: float = 1.0) -> np.ndarray:
    """Dense similarity of each query row of X with each codebook row of C."""
    X, C = _f64(X), _f64(C)
    B, D = X.shape
    M, D2 = C.shape
    assert D == D2
    S = np.empty((B, M), np.float64)
    _load().gso_similarity(_dp(X), B, D, _dp(C), M, int(mode), float(scale), _dp(S))
    return S


def argmax(S) -> np.ndarray:
    S = _f64(S)
    B, M = S.shape
    idx = np.empty(B, np.int32)
    _load().gso_argmax(_dp(S), B, M, idx.ctypes.data_as(ctypes.POINTER(ctypes.c_int)))
    return idx


def softmax(S, beta: float = 1.0) -> np.ndarray:
    S = _f64(S)
    B, M = S.shape
    A = np.empty((B, M), np.float64)
    _load().gso_softmax(_dp(S), B, M, float(beta), _dp(A))
    return A


def project(X, Q) -> np.ndarray:
    """T[b, k] = <x_b, q_k>."""
    X, Q = _f64(X), _f64(Q)
    B, D = X.shape
    r, D2 = Q.shape
    assert D == D2
    T = np.empty((B, r), np.float64)
    _load().gso_project(_dp(X), B, D, _dp(Q), r, _dp(T))
    return T


def reconstruct(T, Q) -> np.ndarray:
    """X[b] = sum_k T[b, k] q_k."""
    T, Q = _f64(T), _f64(Q)
    B, r = T.shape
    r2, D = Q.shape
    assert r == r2
    X = np.empty((B, D), np.float64)
    _load().gso_reconstruct(_dp(T), B, r, _dp(Q), D, _dp(X))
    return X


def bind(X, Y) -> np.ndarray:
    """Element-wise product."""
    X, Y = _f64(X), _f64(Y)
    assert X.shape == Y.shape
    Z = np.empty_like(X)
    _load().gso_bind(_dp(X), _dp(Y), X.size, _dp(Z))
    return Z


def circular(X, Y, L: int, corr: bool = False) -> np.ndarray:
    """Blockwise circular convolution (corr=False) or correlation (corr=True)
    of the rows of X and Y over consecutive blocks of length L."""
    X, Y = _f64(X), _f64(Y)
    assert X.shape == Y.shape and X.ndim == 2
    B, D = X.shape
    assert L >= 1 and D % L == 0
    Z = np.empty_like(X)
    _load().gso_circular(_dp(X), _dp(Y), B, D, int(L), int(bool(corr)), _dp(Z))
    return Z


def xor(X, Y) -> np.ndarray:
    """Exclusive or of the bits (value >= 0.5) of X and Y, as 0.0 / 1.0."""
    X, Y = _f64(X), _f64(Y)
    assert X.shape == Y.shape
    Z = np.empty_like(X)
    _load().gso_xor(_dp(X), _dp(Y), X.size, _dp(Z))
    return Z


def memory_model(M: int, D: int, k: int, elem_bytes: int = 4) -> dict:
    """Storage of the dense codebook against basis + Gram-loc (Sec. 3.1).

    dense = M*D elements; compressed = D*k + M*k elements; per-vector ratio
    D/k (one dense vector against its Gram-loc)."""
    dense = M * D * elem_bytes
    comp = (D * k + M * k) * elem_bytes
    return {"dense_bytes": dense, "compressed_bytes": comp,
            "total_ratio": dense / comp, "per_vector_ratio": D / k}
