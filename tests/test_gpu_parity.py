"""GPU parity of every C-ABI call against the fp64 oracle.

Inputs are seeded and synthetic; the oracle's own outputs (Q, R) are fed to
the GPU calls that need a basis, so each call is checked on its own, and the
chained cases check the GPU's compress output end to end.  Sizes span several
128-wide tiles with ragged tails, strided leading dimensions, leading
dimensions that force the scalar load path, r = 1, B = 1, and B = 0.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2608_01528_amd import gramspace as gsm
from paper_2608_01528_amd import workloads as wl
from tests.gpu_util import (TOL_BF16, TOL_F32, U32, check_argmax_bound, dev, exact_scores_bound, gamma, host,
                            rowrel, score_bound, cosine_factor)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    gsm.lib()


def padded(a, pad, dtype=torch.float32):
    """Device copy of a with `pad` extra columns of leading dimension (a view)."""
    a = np.asarray(a)
    full = np.zeros((a.shape[0], a.shape[1] + pad), a.dtype)
    full[:, : a.shape[1]] = a
    return dev(full, dtype)[:, : a.shape[1]]


def rq_codebook(kind, M, D, seed, dup=0.0):
    C = (wl.bipolar_codebook if kind == "bipolar" else wl.binary_codebook)(M, D, seed)
    if dup:
        C, _, _ = wl.duplicate_rows(C, dup, seed)
    return C


def _name_early(dt):
    return "bf16" if dt == torch.bfloat16 else "f32"


def argmax_exact(idx, T, R, qnorm2=None, cnorm=None, mode="cosine", scale=1.0):
    """The argmax against the oracle's exact scores of the values the kernel
    read: T and R (upcast exactly), and the norms passed to it (None: summed
    by the kernel from T or R).  Bit-exact outside twice the a-priori bound of
    the fp32 evaluation; returns the near-tie count."""
    cos = mode == "cosine"
    given = (qnorm2 is not None and cnorm is not None) or not cos
    Se, E = exact_scores_bound(T, R, qnorm2, cnorm, cosine=cos, scale=scale, norms_given=given)
    return check_argmax_bound(host(idx) if torch.is_tensor(idx) else idx, Se, E)


def soft_exact(P, R, cnorm=None, mode="cosine", scale=1.0):
    """The oracle's exact scores of the fused soft selection's inputs P and R
    (t = p R, s_j = scale * sim(t, R_j) with ||t|| from t), and the per-row
    bound of the kernel's fp32 evaluation.  Both of the kernel's forms (t
    formed, or scores through R R^T) sum p_k and R entries in fp32; their
    error is at most (gamma_M + gamma_r) times ((|P| |R|) |R|^T) for the
    inner products, and the norm of t carries (2 gamma_M + gamma_r) rho^2 +
    gamma_M rho + gamma_r with rho = || |p| |R| || / ||t||."""
    P = np.asarray(P, np.float64)
    R = np.asarray(R, np.float64)
    M, r = R.shape
    T = oracle.prob2vec(P, R)
    dot = oracle.similarity(T, R, oracle.DOT)
    absT = oracle.prob2vec(np.abs(P), np.abs(R))
    absdot = oracle.similarity(absT, np.abs(R), oracle.DOT)
    gam = gamma(M) + gamma(r)
    if mode == "cosine":
        tn2 = (T * T).sum(1)
        cn = np.sqrt((R * R).sum(1)) if cnorm is None else np.asarray(cnorm, np.float64)
        factor = cosine_factor(tn2, cn, scale)
        rho = np.sqrt((absT * absT).sum(1)) / np.maximum(np.sqrt(tn2), 1e-300)
        rel = ((2 * gamma(M) + gamma(r)) * rho ** 2 + gamma(M) * rho + gamma(r) + 10 * U32)[:, None]
    else:
        factor = np.full(dot.shape, float(scale))
        rel = 8 * U32
    S = factor * dot
    return S, score_bound(S, absdot, factor, gam, rel)


def soft_argmax_exact(idx, P, R, cnorm=None, mode="cosine", scale=1.0):
    """The fused soft selection's argmax against the oracle's exact scores of
    its inputs (soft_exact): bit-exact outside the near-tie band."""
    S, E = soft_exact(P, R, cnorm, mode, scale)
    return check_argmax_bound(host(idx) if torch.is_tensor(idx) else idx, S, E)


# ---------------------------------------------------------------- compress

COMPRESS = [
    ("tiny", lambda: rq_codebook("bipolar", 10, 1024, 1)),
    ("vsa22", lambda: wl.codebook(wl.WORKLOADS["vsa"], 3)),
    ("bipolar64x2048", lambda: rq_codebook("bipolar", 64, 2048, 3)),
    ("binary120x1000", lambda: rq_codebook("binary", 120, 1000, 4)),
    ("dup100x700", lambda: rq_codebook("bipolar", 100, 700, 5, dup=0.1)),
    ("hadamard64", lambda: wl.hadamard_codebook(64)),
    ("single", lambda: rq_codebook("bipolar", 1, 100, 6)),
]


def special_rows():
    C = rq_codebook("binary", 40, 256, 7).astype(np.float32)
    C[3] = 0
    C[10] = C[2]
    C[20] = C[5] + C[6]
    C[33] = C[1]
    return C


COMPRESS.append(("special_rows", special_rows))


@pytest.mark.parametrize("name,make", COMPRESS, ids=[c[0] for c in COMPRESS])
def test_compress_matches_oracle(name, make):
    C = np.ascontiguousarray(make(), dtype=np.float32)
    print("compress case", name, C.shape, flush=True)
    Qo, Ro, kept_o, ro = oracle.compress(C)
    Q, R, r, kept, cnorm = gsm.gs_compress(dev(C))
    torch.cuda.synchronize()
    assert r == ro
    assert list(host(kept).astype(int)) == list(kept_o)
    Qg, Rg = host(Q), host(R)
    assert np.abs(Qg - Qo).max() <= 1e-12
    assert np.abs(Rg - Ro).max() <= 1e-12 * max(1.0, np.abs(Ro).max())
    # invariants on the GPU's own output: Q Q^T = I, C = R Q
    assert np.abs(Qg @ Qg.T - np.eye(r)).max() <= 1e-12
    assert np.abs(Rg @ Qg - C).max() <= 1e-12 * np.abs(C).max()
    np.testing.assert_allclose(host(cnorm), oracle.row_norms(C), rtol=1e-6)


@pytest.mark.parametrize("qt,rt", [(torch.float32, torch.float32), (torch.bfloat16, torch.bfloat16),
                                   (torch.float32, torch.float64)])
def test_compress_output_types(qt, rt):
    C = rq_codebook("binary", 50, 600, 8)
    Qo, Ro, kept_o, ro = oracle.compress(C)
    Q, R, r, kept, cnorm = gsm.gs_compress(dev(C), q_dtype=qt, r_dtype=rt)
    torch.cuda.synchronize()
    assert r == ro
    tq = 1e-6 if qt == torch.float32 else 4e-3
    tr = 1e-6 if rt != torch.bfloat16 else 4e-3
    assert rowrel(host(Q), Qo) <= tq
    assert rowrel(host(R), Ro) <= tr


def test_compress_capacity_is_zero_filled():
    C = rq_codebook("bipolar", 20, 128, 9)
    C[5] = C[4]
    Cd = dev(C)
    Q, R, r, kept, cnorm = gsm.gs_compress(Cd)
    torch.cuda.synchronize()
    assert r == 19
    # the wrapper returns views of full M-row / M-column buffers
    Qb = torch.as_strided(Q, (20, 128), (128, 1))
    Rb = torch.as_strided(R, (20, 20), (20, 1))
    assert float(Qb[19:].abs().max()) == 0.0
    assert float(Rb[:, 19:].abs().max()) == 0.0


def near_dependent_codebook():
    """Rows 40 and 41 almost in the span of earlier rows (residuals about 1e-9
    and 0 relative to the row), row 41 a combination in the same panel, a
    duplicate and a negation across panels, D not a multiple of the chunk
    sizes, several levels of the panel factor (D = 5000: 20 leaves)."""
    g = np.random.default_rng(3)
    C = g.standard_normal((100, 5000))
    C[40] = C[3] + 1e-9 * g.standard_normal(5000)
    C[41] = C[40] + C[7]
    C[70] = C[33]
    C[95] = -C[64]
    return C


@pytest.mark.parametrize("tol", [1e-12, 1e-10, 1e-8, 1e-3])
def test_compress_rank_threshold(tol):
    # the rank decisions follow the relative threshold as the oracle does:
    # row 40 (residual ~1e-9) is kept below tol 1e-9 and dropped above
    C = near_dependent_codebook()
    Qo, Ro, kept_o, ro = oracle.compress(C, tol)
    Q, R, r, kept, cnorm = gsm.gs_compress(dev(C, torch.float64), tol=tol)
    torch.cuda.synchronize()
    print("rank threshold", tol, r, ro, flush=True)
    assert r == ro == (97 if tol < 1e-9 else 96)
    assert list(host(kept).astype(int)) == list(kept_o)
    Qg, Rg = host(Q), host(R)
    assert np.abs(Qg @ Qg.T - np.eye(r)).max() <= 1e-12
    # C = R Q where every row is kept or exactly dependent; a dropped
    # near-dependent row keeps its own residual, as in the oracle
    assert np.abs(Rg @ Qg - Ro @ Qo).max() <= 1e-11 * np.abs(C).max()
    if tol > 1e-9:
        # with the near-dependent row dropped every basis vector is well determined
        assert np.abs(Qg - Qo).max() <= 1e-12
        assert np.abs(Rg - Ro).max() <= 1e-12 * np.abs(Ro).max()


def test_compress_rank_one_codebook():
    # every row a multiple of one bipolar vector: the panels' triangular
    # factors hold only rounding residue past the first column, decaying by
    # about 1e-16 per reflection towards the underflow range
    rng = np.random.default_rng(21)
    base = rng.choice([-1.0, 1.0], 700)
    coef = rng.integers(1, 4, 45) * rng.choice([-1.0, 1.0], 45)
    C = np.outer(coef, base).astype(np.float32)
    Qo, Ro, kept_o, ro = oracle.compress(C)
    Q, R, r, kept, _ = gsm.gs_compress(dev(C))
    torch.cuda.synchronize()
    assert r == ro == 1 and list(host(kept).astype(int)) == list(kept_o) == [0]
    assert np.isfinite(host(R)).all() and np.isfinite(host(Q)).all()
    assert np.abs(host(Q) - Qo).max() <= 1e-12
    assert np.abs(host(R) - Ro).max() <= 1e-12 * np.abs(Ro).max()


def test_compress_rejects_nonfinite():
    C = rq_codebook("bipolar", 8, 64, 1)
    C[3, 7] = np.nan
    with pytest.raises(gsm.GramSpaceError) as e:
        gsm.gs_compress(dev(C))
    assert e.value.status == gsm.GS_ERR_NUMERIC


# ----------------------------------------------------------------- project

def basis(r, D, seed):
    C = rq_codebook("bipolar", r, D, seed)
    Qo, Ro, kept, rr = oracle.compress(C)
    assert rr == r
    return C, Qo, Ro


@pytest.mark.parametrize("B,D,r,dtype,pad", [
    (300, 1000, 70, torch.float32, 0),
    (257, 2048, 130, torch.float32, 8),
    (64, 512, 1, torch.float32, 0),
    (1, 96, 33, torch.float32, 0),
    (333, 1030, 45, torch.float32, 1),     # odd leading dimension: scalar loads
    (200, 1024, 64, torch.bfloat16, 0),
    (129, 520, 140, torch.bfloat16, 3),
])
def test_project(B, D, r, dtype, pad):
    print("project", B, D, r, dtype, pad, flush=True)
    C, Qo, Ro = basis(r, D, 11)
    X = np.random.default_rng(B).standard_normal((B, D)).astype(np.float32)
    if dtype == torch.bfloat16:
        Xin, Qin = wl.round_bf16(X), wl.round_bf16(Qo.astype(np.float32))
    else:
        Xin, Qin = X, Qo.astype(np.float32)
    T, xn = gsm.gs_project(padded(Xin, pad, dtype), padded(Qin, pad, dtype), out_dtype=torch.float32,
                           xnorm2=True)
    torch.cuda.synchronize()
    tol = TOL_F32 if dtype == torch.float32 else TOL_BF16
    assert rowrel(host(T), oracle.project(X, Qo)) <= tol
    np.testing.assert_allclose(host(xn), oracle.row_norms(X) ** 2, rtol=tol)


def test_project_bf16_output():
    C, Qo, Ro = basis(40, 700, 12)
    X = np.random.default_rng(2).standard_normal((150, 700)).astype(np.float32)
    T = gsm.gs_project(dev(X), dev(Qo), out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    assert rowrel(host(T), oracle.project(X, Qo)) <= TOL_BF16


# ---------------------------------------------------------------- prob2vec

@pytest.mark.parametrize("B,M,D,dup,dtype", [
    (1000, 22, 1024, 0.0, torch.float32),    # small-codebook kernel
    (129, 5, 1024, 0.0, torch.float32),
    (700, 40, 1024, 0.0, torch.float32),     # small-codebook kernel, padded to 48
    (257, 64, 800, 0.1, torch.float32),      # padded to 64, rank-deficient
    (300, 47, 512, 0.0, torch.bfloat16),
    (333, 100, 512, 0.0, torch.float32),     # matrix-core path
    (300, 160, 900, 0.1, torch.float32),     # rank-deficient, r < M
    (250, 150, 800, 0.0, torch.bfloat16),
    (260, 20, 256, 0.0, torch.bfloat16),
    (400, 29, 768, 0.1, torch.float32),      # padded to 32 (matrix cores), r < M, ragged rows
    (333, 31, 512, 0.0, torch.bfloat16),
])
def test_prob2vec(B, M, D, dup, dtype):
    print("prob2vec", B, M, D, dup, dtype, flush=True)
    C = rq_codebook("bipolar", M, D, M, dup=dup)
    Qo, Ro, kept, r = oracle.compress(C)
    P = wl.dirichlet_probs(B, M, 0.5, M)
    Pin, Rin = (P, Ro.astype(np.float32)) if dtype == torch.float32 else (wl.round_bf16(P), wl.round_bf16(Ro.astype(np.float32)))
    T = gsm.gs_prob2vec(dev(Pin, dtype), dev(Rin, dtype), out_dtype=torch.float32)
    torch.cuda.synchronize()
    To = oracle.project(oracle.prob2vec(P, C), Qo)
    assert rowrel(host(T), To) <= (TOL_F32 if dtype == torch.float32 else TOL_BF16)


# -------------------------------------------------- similarity / attention

SIM_CASES = [  # (B, M, D, dup, in_span)
    (700, 10, 1024, 0.0, True),
    (513, 22, 1024, 0.0, False),
    (600, 40, 1024, 0.0, True),     # small-codebook kernels up to 64 entries
    (300, 64, 700, 0.1, False),     # r < M
    (300, 100, 1000, 0.0, True),
    (260, 300, 700, 0.1, False),    # r < M, three column blocks, ragged
]


def sim_inputs(B, M, D, dup, in_span, seed=0):
    C = rq_codebook("bipolar", M, D, 100 + M, dup=dup)
    Qo, Ro, kept, r = oracle.compress(C)
    P = wl.dirichlet_probs(B, M, 0.5, seed + M)
    X = oracle.prob2vec(P, C)
    if not in_span:
        X = X + np.sqrt(0.1) * np.random.default_rng(seed).standard_normal(X.shape)
    To = oracle.project(X, Qo)
    return C, Qo, Ro, X, To


@pytest.mark.parametrize("B,M,D,dup,in_span", SIM_CASES)
@pytest.mark.parametrize("mode", ["cosine", "dot"])
def test_similarity(B, M, D, dup, in_span, mode):
    print("similarity", B, M, D, dup, in_span, mode, flush=True)
    C, Qo, Ro, X, To = sim_inputs(B, M, D, dup, in_span)
    scale = 1.0 if mode == "cosine" else 1.0 / math.sqrt(D)
    qn = dev(oracle.row_norms(X) ** 2) if (mode == "cosine" and not in_span) else None
    cn = dev(oracle.row_norms(C)) if M > 50 else None
    S, idx = gsm.gs_similarity(dev(To), dev(Ro), qnorm2=qn, cnorm=cn, mode=mode, scale=scale)
    torch.cuda.synchronize()
    So = oracle.similarity(X, C, oracle.COSINE if mode == "cosine" else oracle.DOT, scale)
    assert rowrel(host(S), So) <= TOL_F32
    argmax_exact(idx, host(dev(To)), host(dev(Ro)), None if qn is None else host(qn), None if cn is None else host(cn),
                 mode, scale)
    # argmax alone (no score output) gives the same indices
    _, idx2 = gsm.gs_similarity(dev(To), dev(Ro), qnorm2=qn, cnorm=cn, mode=mode, scale=scale, scores=False)
    torch.cuda.synchronize()
    assert torch.equal(idx, idx2)


@pytest.mark.parametrize("B,M,D,dup,in_span", SIM_CASES)
@pytest.mark.parametrize("beta", [1.0, 16.0])
def test_attention(B, M, D, dup, in_span, beta):
    print("attention", B, M, D, dup, in_span, beta, flush=True)
    C, Qo, Ro, X, To = sim_inputs(B, M, D, dup, in_span, seed=1)
    qn = dev(oracle.row_norms(X) ** 2) if not in_span else None
    A, O = gsm.gs_attention(dev(To), dev(Ro), qnorm2=qn, mode="cosine", beta=beta, weighted_sum=True,
                            out_dtype=torch.float32)
    torch.cuda.synchronize()
    Ao = oracle.softmax(oracle.similarity(X, C, oracle.COSINE), beta)
    assert rowrel(host(A), Ao) <= TOL_F32
    np.testing.assert_allclose(host(A).sum(1), 1.0, atol=1e-5)
    Oo = oracle.project(oracle.prob2vec(Ao, C), Qo)
    assert rowrel(host(O), Oo) <= TOL_F32


def test_similarity_bf16():
    B, M, D = 400, 120, 600
    C, Qo, Ro, X, To = sim_inputs(B, M, D, 0.0, False, seed=3)
    qn = oracle.row_norms(X) ** 2
    Tb, Rb = wl.round_bf16(To.astype(np.float32)), wl.round_bf16(Ro.astype(np.float32))
    S, idx = gsm.gs_similarity(dev(Tb, torch.bfloat16), dev(Rb, torch.bfloat16), qnorm2=dev(qn), mode="cosine")
    A, _ = gsm.gs_attention(dev(Tb, torch.bfloat16), dev(Rb, torch.bfloat16), qnorm2=dev(qn), beta=4.0)
    torch.cuda.synchronize()
    So = oracle.similarity(X, C, oracle.COSINE)
    assert rowrel(host(S), So) <= TOL_BF16
    assert rowrel(host(A), oracle.softmax(So, 4.0)) <= TOL_BF16
    # argmax: exact against the oracle on the bf16-rounded inputs (coordinates)
    argmax_exact(idx, Tb, Rb, host(dev(qn)), None)


def test_argmax_ties_lowest_index():
    # identical codebook coordinates give exact ties: the lowest index wins
    M, r = 40, 8
    R = np.zeros((M, r), np.float32)
    R[:, 0] = 1.0
    R[7:, 1] = 0.5
    T = np.zeros((300, r), np.float32)
    T[:, 0] = 1.0
    for Mm in (M, 12):
        _, idx = gsm.gs_similarity(dev(T), dev(R[:Mm]), mode="dot", scores=False)
        torch.cuda.synchronize()
        assert int(host(idx).max()) == 0


# ----------------------------------------- similarity and attention together

SA_CASES = [
    # B, M, D, storage, beta
    (600, 40, 1024, torch.float32, 16.0),     # small-codebook scores
    (300, 100, 1000, torch.float32, 4.0),     # product scores, one column tile
    (520, 300, 700, torch.float32, -3.0),     # ragged column tiles, negative beta
    (400, 600, 1200, torch.bfloat16, 16.0),   # bf16 storage
    (500, 30, 700, torch.bfloat16, 8.0),      # bf16 storage, small-codebook scores
]


def softmax_of(S, beta):
    """fp64 softmax of beta times the returned fp32 scores."""
    z = beta * np.asarray(S, np.float64)
    e = np.exp(z - z.max(axis=1, keepdims=True))
    return e / e.sum(axis=1, keepdims=True)


def first_max(S):
    S = np.asarray(S)
    return (S == S.max(axis=1, keepdims=True)).argmax(axis=1)


@pytest.mark.parametrize("B,M,D,dt,beta", SA_CASES, ids=lambda v: _name_early(v) if isinstance(v, torch.dtype) else None)
def test_similarity_attention(B, M, D, dt, beta):
    print("similarity_attention", B, M, D, dt, beta, flush=True)
    C, Qo, Ro, X, To = sim_inputs(B, M, D, 0.1 if M >= 300 else 0.0, False, seed=7)
    qn = dev(oracle.row_norms(X) ** 2)
    cn = dev(oracle.row_norms(C))
    bf = dt == torch.bfloat16
    Tin, Rin = (wl.round_bf16(To.astype(np.float32)), wl.round_bf16(Ro.astype(np.float32))) if bf else (To, Ro)
    T, R = dev(Tin, dt), dev(Rin, dt)
    kw = dict(qnorm2=qn, cnorm=cn, mode="cosine")
    S, idx, A = gsm.gs_similarity_attention(T, R, beta=beta, **kw)
    torch.cuda.synchronize()
    tol = TOL_BF16 if bf else TOL_F32
    So = oracle.similarity(X, C, oracle.COSINE)
    assert rowrel(host(S), So) <= tol
    assert rowrel(host(A), oracle.softmax(So, beta)) <= tol
    # the three outputs derive from the one score matrix returned
    Sh = host(S)
    assert np.array_equal(host(idx), first_max(Sh))
    assert rowrel(host(A), softmax_of(Sh, beta)) <= 1e-5
    argmax_exact(idx, Tin, Rin, host(qn), host(cn))
    # the scores and argmax are gs_similarity's, bit for bit
    S1, idx1 = gsm.gs_similarity(T, R, **kw)
    A1, _ = gsm.gs_attention(T, R, beta=beta, **kw)
    torch.cuda.synchronize()
    assert torch.equal(S, S1) and torch.equal(idx, idx1)
    assert rowrel(host(A), host(A1)) <= 1e-5
    # partial outputs: weights formed in place, argmax alone, weights alone
    _, idx2, A2 = gsm.gs_similarity_attention(T, R, beta=beta, scores=False, **kw)
    _, idx3, _ = gsm.gs_similarity_attention(T, R, beta=beta, scores=False, attention=False, **kw)
    _, _, A4 = gsm.gs_similarity_attention(T, R, beta=beta, scores=False, argmax=False, **kw)
    torch.cuda.synchronize()
    assert torch.equal(A2, A) and torch.equal(A4, A)
    assert torch.equal(idx2, idx) and torch.equal(idx3, idx)


def test_similarity_attention_unaligned_and_long_rows():
    # rows past 2048 entries and rows not 16-byte aligned take the three-sweep
    # pass; the coordinates are arbitrary vectors (the dense form of the call)
    rng = np.random.default_rng(11)
    for B, M, r, ld_pad in [(300, 2500, 96, 0), (257, 700, 64, 1), (130, 5, 5, 2)]:
        print("similarity_attention rows", B, M, r, ld_pad, flush=True)
        T = rng.standard_normal((B, r)).astype(np.float32)
        R = rng.standard_normal((M, r)).astype(np.float32)
        S = torch.empty((B, M + ld_pad), device="cuda")[:, :M]
        A = torch.empty((B, M + ld_pad), device="cuda")[:, :M]
        for beta in (5.0, -2.0):
            S_, idx, A_ = gsm.gs_similarity_attention(dev(T), dev(R), mode="cosine", beta=beta, out=S, a_out=A)
            torch.cuda.synchronize()
            So = oracle.similarity(T.astype(np.float64), R.astype(np.float64), oracle.COSINE)
            assert rowrel(host(S), So) <= TOL_F32
            assert rowrel(host(A), oracle.softmax(So, beta)) <= TOL_F32
            assert np.array_equal(host(idx), first_max(host(S)))
            assert rowrel(host(A), softmax_of(host(S), beta)) <= 1e-5
            argmax_exact(idx, T, R)


def test_similarity_attention_single_entry():
    # one codebook entry: every weight is one and every argmax zero
    T = np.random.default_rng(12).standard_normal((100, 1)).astype(np.float32)
    S, idx, A = gsm.gs_similarity_attention(dev(T), dev(np.ones((1, 1), np.float32)), mode="dot", beta=3.0)
    torch.cuda.synchronize()
    assert np.array_equal(host(S)[:, 0], T[:, 0])
    assert not host(idx).any()
    assert np.array_equal(host(A), np.ones((100, 1), np.float32))


# -------------------------------------------------------------- reconstruct

@pytest.mark.parametrize("B,M,D,dtype,pad", [
    (300, 100, 1000, torch.float32, 0),
    (130, 33, 4100, torch.float32, 4),
    (64, 1, 300, torch.float32, 0),
    (200, 90, 1030, torch.float32, 1),
    (250, 70, 1024, torch.bfloat16, 0),
])
def test_reconstruct(B, M, D, dtype, pad):
    print("reconstruct", B, M, D, dtype, flush=True)
    C = rq_codebook("bipolar", M, D, 200 + M)
    Qo, Ro, kept, r = oracle.compress(C)
    P = wl.dirichlet_probs(B, M, 0.3, 7)
    To = P.astype(np.float64) @ Ro          # exact coordinates of P C
    if dtype == torch.bfloat16:
        Tin, Qin = wl.round_bf16(To.astype(np.float32)), wl.round_bf16(Qo.astype(np.float32))
    else:
        Tin, Qin = To.astype(np.float32), Qo.astype(np.float32)
    X = gsm.gs_reconstruct(padded(Tin, pad, dtype), padded(Qin, pad, dtype), out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert rowrel(host(X), oracle.prob2vec(P, C)) <= (TOL_F32 if dtype == torch.float32 else TOL_BF16)


@pytest.mark.parametrize("kind", ["binary", "bipolar"])
def test_bind_and_reproject(kind):
    B, M, D = 260, 150, 1100
    C = rq_codebook(kind, M, D, 300)
    Qo, Ro, kept, r = oracle.compress(C)
    Pa = wl.dirichlet_probs(B, M, 0.05, 1)
    Pb = wl.dirichlet_probs(B, M, 0.05, 2)
    Ta = dev(oracle.project(oracle.prob2vec(Pa, C), Qo))
    Tb = dev(oracle.project(oracle.prob2vec(Pb, C), Qo))
    Y = gsm.gs_reconstruct(Ta, dev(Qo), T2=Tb, bind="mul")
    torch.cuda.synchronize()
    Yo = oracle.bind(oracle.prob2vec(Pa, C), oracle.prob2vec(Pb, C))
    assert rowrel(host(Y), Yo) <= TOL_F32
    Ty = gsm.gs_project(Y, dev(Qo))
    torch.cuda.synchronize()
    assert rowrel(host(Ty), oracle.project(Yo, Qo)) <= TOL_F32


def _orthonormal_rows(r, D, seed):
    q, _ = np.linalg.qr(np.random.default_rng(seed).standard_normal((D, r)))
    return np.ascontiguousarray(q.T)


@pytest.mark.parametrize("B,r,D", [(260, 150, 1100), (129, 256, 4096), (1, 1, 40), (300, 32, 64),
                                   (257, 33, 1000), (128, 64, 2048), (5, 128, 160), (200, 100, 512)])
def test_bind_coords(B, r, D):
    # restore -> bind -> re-project in one pass against the oracle's three
    # steps in fp64, and against the library's two calls; ragged batch row
    # blocks (128 rows per work-group), ragged r (padded to 32, 64, 128 or
    # 256) and ragged column chunks of 32
    print("bind_coords", B, r, D, flush=True)
    rng = np.random.default_rng(B + r + D)
    Q = _orthonormal_rows(r, D, r + D).astype(np.float32)
    T = rng.standard_normal((B, r)).astype(np.float32)
    T2 = rng.standard_normal((B, r)).astype(np.float32)
    Z = gsm.gs_bind_coords(dev(T), dev(T2), dev(Q))
    X = gsm.gs_reconstruct(dev(T), dev(Q), T2=dev(T2), bind="mul")
    Zc = gsm.gs_project(X, dev(Q))
    torch.cuda.synchronize()
    Zo = oracle.project(oracle.bind(oracle.reconstruct(T, Q), oracle.reconstruct(T2, Q)), Q)
    assert rowrel(host(Z), Zo) <= TOL_F32
    assert rowrel(host(Z), host(Zc)) <= TOL_F32


def test_bind_coords_codebook_and_strides():
    # coordinates of codebook rows (the binding of two entries, projected
    # back), operands with leading dimensions that are not multiples of four
    # (element loads), and an output with a leading dimension larger than r
    C = rq_codebook("bipolar", 40, 1000, 17)
    Qo, Ro, kept, r = oracle.compress(C)
    ia, ib = np.arange(40), np.roll(np.arange(40), 7)
    Ta = torch.zeros((40, r + 3), dtype=torch.float32, device="cuda")[:, :r]
    Tb = torch.zeros((40, r + 1), dtype=torch.float32, device="cuda")[:, :r]
    Ta.copy_(dev(Ro[ia]))
    Tb.copy_(dev(Ro[ib]))
    Qs = torch.zeros((r, 1003), dtype=torch.float32, device="cuda")[:, :1000]
    Qs.copy_(dev(Qo))
    out = torch.full((40, r + 9), float("nan"), device="cuda")
    Z = gsm.gs_bind_coords(Ta, Tb, Qs, out=out[:, :r])
    torch.cuda.synchronize()
    Zo = oracle.project(oracle.bind(C[ia], C[ib]), Qo)
    assert rowrel(host(Z), Zo) <= TOL_F32
    assert torch.isnan(out[:, r:]).all()                 # nothing past column r is written
    Z0 = gsm.gs_bind_coords(Ta[:0], Tb[:0], Qs)          # empty batch
    assert Z0.shape == (0, r)


def test_bipolar_self_binding_is_ones():
    C = rq_codebook("bipolar", 30, 512, 5)
    Qo, Ro, kept, r = oracle.compress(C)
    T = dev(Ro)                      # coordinates of the codebook itself
    Y = gsm.gs_reconstruct(T, dev(Qo), T2=T, bind="mul")
    torch.cuda.synchronize()
    assert np.abs(host(Y) - 1.0).max() <= 1e-4


# ------------------------------------------------------------ end to end

@pytest.mark.parametrize("wname", ["tiny"])
def test_chain_tiny_workload(wname):
    w = wl.WORKLOADS[wname]
    C = wl.codebook(w)
    P = wl.probabilities(w)
    Q, R, r, kept, cnorm = gsm.gs_compress(dev(C), q_dtype=torch.float32, r_dtype=torch.float32)
    T = gsm.gs_prob2vec(dev(P), R)
    S, idx = gsm.gs_similarity(T, R, cnorm=cnorm, mode="cosine")
    A, _ = gsm.gs_attention(T, R, cnorm=cnorm, beta=16.0)
    X = gsm.gs_reconstruct(T, Q)
    torch.cuda.synchronize()
    V = oracle.prob2vec(P, C)
    So = oracle.similarity(V, C, oracle.COSINE)
    assert r == 10
    assert rowrel(host(S), So) <= TOL_F32
    argmax_exact(idx, host(T), host(R), None, host(cnorm))
    assert rowrel(host(A), oracle.softmax(So, 16.0)) <= TOL_F32
    assert rowrel(host(X), V) <= TOL_F32


def test_empty_batch_is_noop():
    R = dev(np.eye(4, dtype=np.float32))
    T = gsm.gs_prob2vec(torch.empty((0, 4), device="cuda"), R)
    S, idx = gsm.gs_similarity(torch.empty((0, 4), device="cuda"), R)
    torch.cuda.synchronize()
    assert T.shape == (0, 4) and S.shape == (0, 4) and idx.shape == (0,)


def test_deterministic():
    C = rq_codebook("binary", 70, 900, 12)
    a = gsm.gs_compress(dev(C))
    b = gsm.gs_compress(dev(C))
    X = dev(np.random.default_rng(0).standard_normal((300, 900)).astype(np.float32))
    t1 = gsm.gs_project(X, a[0].float())
    t2 = gsm.gs_project(X, a[0].float())
    torch.cuda.synchronize()
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])
    assert torch.equal(t1, t2)


# ------------------------------------ dense vs Gram-Space similarity (M = 40)

@pytest.mark.parametrize("D", [256, 2048])
def test_dense_and_gram_similarity_agree(D):
    # the dimension sweep's two forms of one lookup: cosine scores of D-space
    # queries against the codebook, and of their coordinates against R
    M, B = 40, 300
    C = wl.bipolar_codebook(M, D, 6, D)
    P = wl.softmax_probs(B, M, np.sqrt(2.0), 6, 100 + D)
    Q, R, r, kept, cn = gsm.gs_compress(dev(C), q_dtype=torch.float32, r_dtype=torch.float32)
    assert r == M
    X = dev(oracle.prob2vec(P, C).astype(np.float32))
    Sd, idd = gsm.gs_similarity(X, dev(C), cnorm=cn)
    T = gsm.gs_project(X, Q)
    Sg, idg = gsm.gs_similarity(T, R.contiguous(), cnorm=cn)
    torch.cuda.synchronize()
    So = oracle.similarity(oracle.prob2vec(P, C), C, oracle.COSINE)
    assert rowrel(host(Sd), So) <= TOL_F32
    assert rowrel(host(Sg), So) <= TOL_F32
    argmax_exact(idd, host(X), C, None, host(cn))
    argmax_exact(idg, host(T), host(R), None, host(cn))


@pytest.mark.parametrize("B,M,K,dtype", [(1, 40, 8192, torch.float32), (17, 1000, 300, torch.float32),
                                         (32, 40, 1000, torch.bfloat16), (5, 70, 45, torch.float32)])
@pytest.mark.parametrize("norms", ["computed", "given"])
def test_few_rows_scores(B, M, K, dtype, norms):
    # at most 32 query rows: the reduction over K is split over work-groups
    print("few rows", B, M, K, dtype, norms, flush=True)
    rng = np.random.default_rng(B * 1000 + M)
    T = rng.standard_normal((B, K)).astype(np.float32)
    R = rng.standard_normal((M, K)).astype(np.float32)
    if dtype == torch.bfloat16:
        T, R = wl.round_bf16(T), wl.round_bf16(R)
    qn = dev(oracle.row_norms(T) ** 2) if norms == "given" else None
    cn = dev(oracle.row_norms(R)) if norms == "given" else None
    S, idx = gsm.gs_similarity(dev(T, dtype), dev(R, dtype), qnorm2=qn, cnorm=cn, mode="cosine")
    Sd, idd = gsm.gs_similarity(dev(T, dtype), dev(R, dtype), mode="dot", scale=0.25)
    A, O = gsm.gs_attention(dev(T, dtype), dev(R, dtype), qnorm2=qn, cnorm=cn, mode="cosine", beta=12.0,
                            weighted_sum=True, out_dtype=torch.float32)
    torch.cuda.synchronize()
    So = oracle.similarity(T, R, oracle.COSINE)
    assert rowrel(host(S), So) <= TOL_F32
    argmax_exact(idx, T, R, None if qn is None else host(qn), None if cn is None else host(cn))
    Sdo = oracle.similarity(T, R, oracle.DOT, 0.25)
    assert rowrel(host(Sd), Sdo) <= TOL_F32
    argmax_exact(idd, T, R, mode="dot", scale=0.25)
    Ao = oracle.softmax(So, 12.0)
    assert rowrel(host(A), Ao) <= TOL_F32
    # weighted sum of the codebook rows, O = A R
    assert rowrel(host(O), Ao @ R.astype(np.float64)) <= (TOL_F32 if dtype == torch.float32 else TOL_BF16)


# ------------------------------------------------- fused soft selection

def soft_case(Ms, Bs, D, seed, dtype=torch.float32):
    books = []
    for i, (M, B) in enumerate(zip(Ms, Bs)):
        C = rq_codebook("bipolar", M, D, seed + i)
        Qo, Ro, kept, r = oracle.compress(C)
        P = wl.softmax_probs(B, M, math.sqrt(2), seed + i)
        Pin, Rin = (P, Ro.astype(np.float32)) if dtype == torch.float32 else \
            (wl.round_bf16(P), wl.round_bf16(Ro.astype(np.float32)))
        books.append(dict(C=C, Qo=Qo, Ro=Ro, P=P, Pd=dev(Pin, dtype), Rd=dev(Rin, dtype), M=M, B=B, r=r))
    return books


def soft_outputs(books, want=("T", "S", "argmax", "A")):
    groups = []
    for b in books:
        g = {"P": b["Pd"], "R": b["Rd"]}
        if "T" in want:
            g["T"] = torch.full((b["B"], b["r"]), np.nan, device="cuda")
        if "S" in want:
            g["S"] = torch.full((b["B"], b["M"]), np.nan, device="cuda")
        if "argmax" in want:
            g["argmax"] = torch.full((b["B"],), -1, dtype=torch.int32, device="cuda")
        if "A" in want:
            g["A"] = torch.full((b["B"], b["M"]), np.nan, device="cuda")
        groups.append(g)
    return groups


@pytest.mark.parametrize("form", ["auto-T", "auto", "coords", "gram"])
@pytest.mark.parametrize("mode,scale,beta", [("cosine", 1.0, 16.0), ("dot", 0.03, 1.0), ("cosine", 2.0, -3.0)])
def test_soft_select(mode, scale, beta, form):
    # auto-T: coordinates stored; auto and gram: scores through the codebook's
    # Gram matrix; coords: coordinates formed per row, not stored
    books = soft_case([5, 6, 10, 22, 32], [1000, 257, 1, 513, 300], 1024, 40)
    with_t = form == "auto-T"
    groups = soft_outputs(books, want=("T", "S", "argmax", "A") if with_t else ("S", "argmax", "A"))
    gsm.gs_soft_select(groups, mode=mode, scale=scale, beta=beta, form=form.split("-")[0])
    torch.cuda.synchronize()
    m = oracle.COSINE if mode == "cosine" else oracle.DOT
    for b, g in zip(books, groups):
        V = oracle.prob2vec(b["P"], b["C"])
        So = oracle.similarity(V, b["C"], m, scale)
        if with_t:
            assert rowrel(host(g["T"]), oracle.project(V, b["Qo"])) <= TOL_F32
        assert rowrel(host(g["S"]), So) <= TOL_F32
        assert rowrel(host(g["A"]), oracle.softmax(So, beta)) <= TOL_F32
        soft_argmax_exact(g["argmax"], host(b["Pd"]), host(b["Rd"]), None, mode, scale)


@pytest.mark.parametrize("tdt", [torch.float32, torch.bfloat16], ids=_name_early)
@pytest.mark.parametrize("form", ["auto-T", "coords"])
def test_soft_select_rank_deficient_coordinates(tdt, form):
    # codebooks with duplicated rows (r < M) on each of the coordinate form's
    # three paths (vector units up to 8 entries, 16 x 16 matrix blocks up to
    # 16, 32 x 32 beyond), ragged batches: T has r columns and the scores,
    # weights and argmax are those of the dense definitions
    Ms, Bs = [7, 8, 13, 16, 20, 31], [300, 64, 257, 1, 700, 129]
    books = []
    for i, (M, B) in enumerate(zip(Ms, Bs)):
        C = rq_codebook("bipolar", M, 256, 90 + i, dup=0.3)
        Qo, Ro, kept, r = oracle.compress(C)
        assert r < M
        P = wl.softmax_probs(B, M, math.sqrt(2), 90 + i)
        books.append(dict(C=C, Qo=Qo, Ro=Ro, P=P, Pd=dev(P), Rd=dev(Ro.astype(np.float32)), M=M, B=B, r=r))
    with_t = form == "auto-T"
    groups = soft_outputs(books, want=("T", "S", "argmax", "A") if with_t else ("S", "argmax", "A"))
    if with_t:
        for g, b in zip(groups, books):
            g["T"] = torch.full((b["B"], b["r"]), np.nan, device="cuda", dtype=tdt)
    gsm.gs_soft_select(groups, mode="cosine", scale=1.0, beta=16.0, form=form.split("-")[0])
    torch.cuda.synchronize()
    for b, g in zip(books, groups):
        V = oracle.prob2vec(b["P"], b["C"])
        So = oracle.similarity(V, b["C"], oracle.COSINE)
        if with_t:
            tol = TOL_F32 if tdt == torch.float32 else TOL_BF16
            assert rowrel(host(g["T"]), oracle.project(V, b["Qo"])) <= tol
        assert rowrel(host(g["S"]), So) <= TOL_F32
        assert rowrel(host(g["A"]), oracle.softmax(So, 16.0)) <= TOL_F32
        soft_argmax_exact(g["argmax"], b["P"], b["Ro"].astype(np.float32), None, "cosine", 1.0)


@pytest.mark.parametrize("pdt", [torch.float32, torch.bfloat16], ids=_name_early)
def test_soft_select_strided_rows(pdt):
    # probabilities and outputs as column slices of wider matrices (row
    # strides above M): element-wise tile moves instead of 16-byte pieces
    books = soft_case([6, 22, 32], [300, 777, 40], 1024, 45, dtype=pdt)
    groups = []
    for b in books:
        Pw = torch.full((b["B"], b["M"] + 3), np.nan, device="cuda", dtype=pdt)
        Pw[:, : b["M"]] = b["Pd"]
        Sw = torch.full((b["B"], b["M"] + 5), np.nan, device="cuda")
        Aw = torch.full((b["B"], b["M"] + 1), np.nan, device="cuda")
        groups.append({"P": Pw[:, : b["M"]], "R": b["Rd"], "S": Sw[:, : b["M"]],
                       "argmax": torch.full((b["B"],), -1, dtype=torch.int32, device="cuda"),
                       "A": Aw[:, : b["M"]], "_S": Sw, "_A": Aw})
    gsm.gs_soft_select([{k: v for k, v in g.items() if not k.startswith("_")} for g in groups],
                       mode="cosine", beta=16.0)
    torch.cuda.synchronize()
    tol = TOL_F32 if pdt == torch.float32 else TOL_BF16
    for b, g in zip(books, groups):
        V = oracle.prob2vec(b["P"], b["C"])
        So = oracle.similarity(V, b["C"], oracle.COSINE)
        assert rowrel(host(g["S"]), So) <= tol
        # the weights against the softmax of the exact scores of the values
        # the kernel read (a softmax of 16 s multiplies the bf16 rounding of
        # the inputs by up to 32 in the weights)
        Se, _ = soft_exact(host(b["Pd"]), host(b["Rd"]))
        assert rowrel(host(g["A"]), oracle.softmax(Se, 16.0)) <= TOL_F32
        if pdt == torch.float32:
            assert rowrel(host(g["A"]), oracle.softmax(So, 16.0)) <= TOL_F32
        soft_argmax_exact(g["argmax"], host(b["Pd"]), host(b["Rd"]))
        # the padding columns of the output rows are untouched
        assert torch.isnan(g["_S"][:, b["M"]:]).all() and torch.isnan(g["_A"][:, b["M"]:]).all()


def test_soft_select_bf16_and_partial_outputs():
    books = soft_case([10, 22], [700, 450], 1024, 50, dtype=torch.bfloat16)
    groups = soft_outputs(books, want=("argmax", "A"))
    gsm.gs_soft_select(groups, mode="cosine", beta=4.0)
    torch.cuda.synchronize()
    for b, g in zip(books, groups):
        V = oracle.prob2vec(b["P"], b["C"])
        So = oracle.similarity(V, b["C"], oracle.COSINE)
        assert rowrel(host(g["A"]), oracle.softmax(So, 4.0)) <= TOL_BF16
        # argmax against the oracle on the bf16-rounded inputs
        soft_argmax_exact(g["argmax"], host(b["Pd"]), host(b["Rd"]))


@pytest.mark.parametrize("tdt", [torch.float32, torch.bfloat16], ids=_name_early)
@pytest.mark.parametrize("form", ["auto", "coords"])
def test_soft_select_bf16_with_coordinates(tdt, form):
    # bf16 probabilities with a coordinate output of either type, ragged
    # batches whose waves end off an 8-value boundary (M = 22, B = 450;
    # M = 5 and 10 with B = 1000 and 257), and one group without T
    books = soft_case([22, 5, 10, 6], [450, 1000, 257, 333], 1024, 55, dtype=torch.bfloat16)
    groups = soft_outputs(books)
    for b, g in zip(books, groups):
        g["T"] = torch.full((b["B"], b["r"]), np.nan, device="cuda", dtype=tdt)
    del groups[3]["T"]
    gsm.gs_soft_select(groups, mode="cosine", beta=16.0, form=form)
    torch.cuda.synchronize()
    for i, (b, g) in enumerate(zip(books, groups)):
        V = oracle.prob2vec(b["P"], b["C"])
        So = oracle.similarity(V, b["C"], oracle.COSINE)
        assert rowrel(host(g["S"]), So) <= TOL_BF16
        Se, _ = soft_exact(host(b["Pd"]), host(b["Rd"]))
        assert rowrel(host(g["A"]), oracle.softmax(Se, 16.0)) <= TOL_F32
        if "T" in g:
            Tg = host(g["T"])
            assert np.isfinite(Tg).all()
            # against the dense definition on the original inputs ...
            assert rowrel(Tg, oracle.project(V, b["Qo"])) <= TOL_BF16
            # ... and, to fp32 accumulation (one rounding to bf16 on top), on
            # the bf16 values the kernel read
            To = oracle.prob2vec(host(b["Pd"]), host(b["Rd"]))
            assert rowrel(Tg, To) <= (1e-5 if tdt == torch.float32 else 8e-3)
        soft_argmax_exact(g["argmax"], host(b["Pd"]), host(b["Rd"]))


def test_soft_select_forms_agree():
    # the Gram form and the coordinate form compute the same scores up to
    # rounding order, and the same argmax outside the near-tie band
    books = soft_case([5, 6, 10, 22], [4096, 4096, 4096, 4096], 1024, 57)
    out = {}
    for form in ("gram", "coords"):
        groups = soft_outputs(books, want=("S", "argmax", "A"))
        gsm.gs_soft_select(groups, mode="cosine", beta=16.0, form=form)
        out[form] = groups
    torch.cuda.synchronize()
    for b, g0, g1 in zip(books, out["gram"], out["coords"]):
        assert rowrel(host(g0["S"]), host(g1["S"])) <= 1e-5
        soft_argmax_exact(g0["argmax"], host(b["Pd"]), host(b["Rd"]))
        soft_argmax_exact(g1["argmax"], host(b["Pd"]), host(b["Rd"]))


def test_soft_select_matches_separate_calls():
    books = soft_case([6, 22], [900, 333], 1024, 60)
    groups = soft_outputs(books)
    gsm.gs_soft_select(groups, mode="cosine", beta=16.0)
    for b, g in zip(books, groups):
        T = gsm.gs_prob2vec(b["Pd"], b["Rd"])
        S, idx = gsm.gs_similarity(T, b["Rd"], mode="cosine")
        A, _ = gsm.gs_attention(T, b["Rd"], mode="cosine", beta=16.0)
        torch.cuda.synchronize()
        assert torch.equal(idx, g["argmax"])
        assert rowrel(host(g["S"]), host(S)) <= 1e-6
        # the two paths sum in different orders; a softmax of beta * s moves
        # each weight by at most 2 beta max|ds| relative to itself
        assert rowrel(host(g["A"]), host(A)) <= 2 * 16.0 * 1e-6


@pytest.mark.parametrize("form", ["gram", "coords", "auto-T"])
def test_soft_select_full_vsa_workload(form):
    # the benchmark's workload at full size and launch configuration (GPU
    # compress, then one fused launch over the four attribute codebooks)
    w = wl.WORKLOADS["vsa"]
    groups, ref = [], []
    for i, M in enumerate(w.Ms):
        C = wl.codebook(w, i)
        P = wl.probabilities(w, i)
        Q, R, r, kept, cnorm = gsm.gs_compress(dev(C), q_dtype=torch.float32, r_dtype=torch.float32)
        assert r == M
        g = {"P": dev(P), "R": R.contiguous(), "cnorm": cnorm, "S": torch.empty((w.B, M), device="cuda"),
             "argmax": torch.empty(w.B, dtype=torch.int32, device="cuda"), "A": torch.empty((w.B, M), device="cuda")}
        if form == "auto-T":
            g["T"] = torch.empty((w.B, r), device="cuda")
        groups.append(g)
        ref.append((C, P))
    gsm.gs_soft_select(groups, mode="cosine", beta=16.0, form=form.split("-")[0])
    torch.cuda.synchronize()
    near = 0
    for (C, P), g in zip(ref, groups):
        V = oracle.prob2vec(P, C)
        So = oracle.similarity(V, C, oracle.COSINE)
        assert rowrel(host(g["S"]), So) <= TOL_F32
        assert rowrel(host(g["A"]), oracle.softmax(So, 16.0)) <= TOL_F32
        near += soft_argmax_exact(g["argmax"], P, host(g["R"]), host(g["cnorm"]))
    print("near-ties:", near)


def test_soft_select_rejects_bad_groups():
    R = dev(np.eye(4, dtype=np.float32))
    P = dev(np.full((10, 4), 0.25, np.float32))
    with pytest.raises(gsm.GramSpaceError) as e:
        gsm.gs_soft_select([{"P": dev(np.zeros((10, 40), np.float32)), "R": dev(np.zeros((40, 40), np.float32))}])
    assert e.value.status == gsm.GS_ERR_SHAPE
    out = torch.empty((10, 4), device="cuda")
    with pytest.raises(gsm.GramSpaceError) as e:
        gsm.gs_soft_select([{"P": P, "R": R, "S": out, "A": out}])
    assert e.value.status == gsm.GS_ERR_ARG


# ------------------------- bf16 pipelined path (16-byte aligned leading dims)

def nan_padded_bf16(a, ld):
    """bf16 device matrix with leading dimension ld whose padding columns hold
    NaN: the kernels may read them in 16-byte units but must not use them."""
    a = np.asarray(a, np.float32)
    full = np.full((a.shape[0], ld), np.nan, np.float32)
    full[:, : a.shape[1]] = a
    return dev(full, torch.bfloat16)[:, : a.shape[1]]


@pytest.mark.parametrize("B,D,r", [(300, 1000, 130), (257, 1001, 45), (64, 200, 136)])
def test_bf16_pipelined_project_reconstruct(B, D, r):
    print("bf16 pipelined", B, D, r, flush=True)
    C = rq_codebook("bipolar", r, D, 77)
    Qo, Ro, kept, rr = oracle.compress(C)
    assert rr == r
    ld_d = (D + 7) // 8 * 8 + 8
    ld_r = (r + 7) // 8 * 8
    X = np.random.default_rng(B).standard_normal((B, D)).astype(np.float32)
    Xb, Qb = wl.round_bf16(X), wl.round_bf16(Qo.astype(np.float32))
    T, xn = gsm.gs_project(nan_padded_bf16(Xb, ld_d), nan_padded_bf16(Qb, ld_d), out_dtype=torch.float32,
                           xnorm2=True)
    torch.cuda.synchronize()
    assert np.isfinite(host(T)).all()
    assert rowrel(host(T), oracle.project(X, Qo)) <= TOL_BF16
    np.testing.assert_allclose(host(xn), oracle.row_norms(Xb) ** 2, rtol=1e-4)
    # reconstruct and bind (K x N operand) from in-span coordinates
    P = wl.dirichlet_probs(B, r, 0.3, 9)
    P2 = wl.dirichlet_probs(B, r, 0.3, 10)
    To, To2 = (P.astype(np.float64) @ Ro), (P2.astype(np.float64) @ Ro)
    Tb, Tb2 = wl.round_bf16(To.astype(np.float32)), wl.round_bf16(To2.astype(np.float32))
    Xr = gsm.gs_reconstruct(nan_padded_bf16(Tb, ld_r), nan_padded_bf16(Qb, ld_d), out_dtype=torch.float32)
    Y = gsm.gs_reconstruct(nan_padded_bf16(Tb, ld_r), nan_padded_bf16(Qb, ld_d),
                           T2=nan_padded_bf16(Tb2, ld_r), bind="mul", out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert np.isfinite(host(Xr)).all() and np.isfinite(host(Y)).all()
    V, V2 = oracle.prob2vec(P, C), oracle.prob2vec(P2, C)
    assert rowrel(host(Xr), V) <= TOL_BF16
    assert rowrel(host(Y), oracle.bind(V, V2)) <= TOL_BF16


@pytest.mark.parametrize("B,M,D", [(300, 150, 700), (200, 300, 640)])
def test_bf16_pipelined_prob2vec_similarity(B, M, D):
    C = rq_codebook("bipolar", M, D, 88, dup=0.1)
    Qo, Ro, kept, r = oracle.compress(C)
    ld_m, ld_r = (M + 7) // 8 * 8 + 8, (r + 7) // 8 * 8
    P = wl.dirichlet_probs(B, M, 0.5, 3)
    Pb, Rb = wl.round_bf16(P), wl.round_bf16(Ro.astype(np.float32))
    T = gsm.gs_prob2vec(nan_padded_bf16(Pb, ld_m), nan_padded_bf16(Rb, ld_r), out_dtype=torch.float32)
    torch.cuda.synchronize()
    assert np.isfinite(host(T)).all()
    V = oracle.prob2vec(P, C)
    assert rowrel(host(T), oracle.project(V, Qo)) <= TOL_BF16
    X = V + np.sqrt(0.1) * np.random.default_rng(1).standard_normal(V.shape)
    Tx = wl.round_bf16(oracle.project(X, Qo).astype(np.float32))
    qn = dev(oracle.row_norms(X) ** 2)
    S, idx = gsm.gs_similarity(nan_padded_bf16(Tx, ld_r), nan_padded_bf16(Rb, ld_r), qnorm2=qn, mode="cosine")
    A, _ = gsm.gs_attention(nan_padded_bf16(Tx, ld_r), nan_padded_bf16(Rb, ld_r), qnorm2=qn, beta=8.0)
    torch.cuda.synchronize()
    So = oracle.similarity(X, C, oracle.COSINE)
    assert np.isfinite(host(S)).all() and np.isfinite(host(A)).all()
    assert rowrel(host(S), So) <= TOL_BF16
    assert rowrel(host(A), oracle.softmax(So, 8.0)) <= TOL_BF16
    # argmax: the oracle's exact scores of the bf16 coordinates and codebook
    # coordinates the kernel read (||x||^2 given, ||R_j|| summed by the kernel)
    argmax_exact(idx, Tx, Rb, host(qn), None)


# --------------------- large-tile path (>= 256 tiles of 256 x 256), bf16 and fp32
#
# Products large enough for the 256 x 256 tiles, with ragged M and N, K tails
# that are neither multiples of the K-step (64 bf16, 32 fp32) nor of a
# 16-byte chunk, NaN-filled row padding, and both output types.  Q and R are
# arbitrary here: project, prob2vec and reconstruct are plain products of
# their operands.  Rows are sampled: the first and last, the tile boundaries
# and random rows.

OP_DTYPES = [torch.bfloat16, torch.float32]


def _tile_rows(B, seed):
    fixed = [0, 1, 255, 256, 511, 512, B // 2, B - 2, B - 1]
    rnd = np.random.default_rng(seed).choice(B, size=24, replace=False)
    return np.array(sorted(set(f for f in fixed if f < B) | set(int(x) for x in rnd)))


def _mat(rows, cols, seed, dtype, scale=1.0):
    """Seeded matrix, exactly representable in `dtype`."""
    x = (scale * np.random.default_rng(seed).standard_normal((rows, cols))).astype(np.float32)
    return wl.round_bf16(x) if dtype == torch.bfloat16 else x


def _ld(cols, dtype, extra=0):
    per = 8 if dtype == torch.bfloat16 else 4          # elements per 16 bytes
    return (cols + per - 1) // per * per + extra


def nan_padded(a, ld, dtype):
    """Device matrix with leading dimension ld whose padding columns hold NaN."""
    a = np.asarray(a, np.float32)
    full = np.full((a.shape[0], ld), np.nan, np.float32)
    full[:, : a.shape[1]] = a
    return dev(full, dtype)[:, : a.shape[1]]


def _name(dt):
    return "bf16" if dt == torch.bfloat16 else "f32"


@pytest.mark.parametrize("op_dtype", OP_DTYPES, ids=_name)
@pytest.mark.parametrize("D", [300, 4100])
@pytest.mark.parametrize("out_dtype", [torch.float32, torch.bfloat16], ids=_name)
def test_large_tile_project(op_dtype, D, out_dtype):
    B, r = 8200, 2000
    print("large-tile project", _name(op_dtype), B, D, r, _name(out_dtype), flush=True)
    X, Q = _mat(B, D, 1, op_dtype), _mat(r, D, 2, op_dtype, 1 / np.sqrt(D))
    ld = _ld(D, op_dtype)
    T, xn = gsm.gs_project(nan_padded(X, ld, op_dtype), nan_padded(Q, ld, op_dtype), out_dtype=out_dtype,
                           xnorm2=True)
    torch.cuda.synchronize()
    rows = _tile_rows(B, 3)
    Tr = host(T[rows])
    assert np.isfinite(Tr).all()
    tol = TOL_BF16 if out_dtype == torch.bfloat16 else TOL_F32
    assert rowrel(Tr, oracle.project(X[rows], Q)) <= tol
    np.testing.assert_allclose(host(xn), oracle.row_norms(X) ** 2, rtol=1e-4)


@pytest.mark.parametrize("op_dtype", OP_DTYPES, ids=_name)
@pytest.mark.parametrize("out_dtype", [torch.float32, torch.bfloat16], ids=_name)
def test_large_tile_reconstruct(op_dtype, out_dtype):
    B, r, D = 2100, 45, 7700
    print("large-tile reconstruct", _name(op_dtype), B, r, D, _name(out_dtype), flush=True)
    T, Q = _mat(B, r, 4, op_dtype), _mat(r, D, 5, op_dtype)
    X = gsm.gs_reconstruct(nan_padded(T, _ld(r, op_dtype), op_dtype), nan_padded(Q, _ld(D, op_dtype, 8), op_dtype),
                           out_dtype=out_dtype)
    torch.cuda.synchronize()
    rows = _tile_rows(B, 6)
    Xr = host(X[rows])
    assert np.isfinite(Xr).all()
    tol = TOL_BF16 if out_dtype == torch.bfloat16 else TOL_F32
    assert rowrel(Xr, oracle.reconstruct(T[rows], Q)) <= tol
    # every column block, including the ragged last one, on a full row
    assert rowrel(host(X[B - 1:B]), oracle.reconstruct(T[B - 1:B], Q)) <= tol


@pytest.mark.parametrize("op_dtype", OP_DTYPES, ids=_name)
@pytest.mark.parametrize("out_dtype", [torch.float32, torch.bfloat16], ids=_name)
def test_large_tile_bind(op_dtype, out_dtype):
    # X = (T Q) .* (T2 Q): with an fp32 output the large-tile path forms the
    # two products one after the other, the second multiplied into the first
    B, r, D = 2100, 45, 7700
    print("large-tile bind", _name(op_dtype), B, r, D, _name(out_dtype), flush=True)
    T, T2, Q = _mat(B, r, 31, op_dtype), _mat(B, r, 32, op_dtype), _mat(r, D, 33, op_dtype)
    ldr, ldd = _ld(r, op_dtype), _ld(D, op_dtype, 8)
    X = gsm.gs_reconstruct(nan_padded(T, ldr, op_dtype), nan_padded(Q, ldd, op_dtype),
                           T2=nan_padded(T2, ldr, op_dtype), bind="mul", out_dtype=out_dtype)
    torch.cuda.synchronize()
    rows = _tile_rows(B, 34)
    Xr = host(X[rows])
    assert np.isfinite(Xr).all()
    tol = TOL_BF16 if out_dtype == torch.bfloat16 else TOL_F32
    Xo = oracle.bind(oracle.reconstruct(T[rows], Q), oracle.reconstruct(T2[rows], Q))
    assert rowrel(Xr, Xo) <= tol
    last = oracle.bind(oracle.reconstruct(T[B - 1:B], Q), oracle.reconstruct(T2[B - 1:B], Q))
    assert rowrel(host(X[B - 1:B]), last) <= tol


@pytest.mark.parametrize("op_dtype", OP_DTYPES, ids=_name)
def test_large_tile_prob2vec(op_dtype):
    B, M, r = 8200, 2050, 2000
    print("large-tile prob2vec", _name(op_dtype), B, M, r, flush=True)
    P = wl.dirichlet_probs(B, M, 0.5, 7)
    if op_dtype == torch.bfloat16:
        P = wl.round_bf16(P)
    R = _mat(M, r, 8, op_dtype)
    T = gsm.gs_prob2vec(nan_padded(P, _ld(M, op_dtype), op_dtype), nan_padded(R, _ld(r, op_dtype), op_dtype),
                        out_dtype=torch.float32)
    torch.cuda.synchronize()
    rows = _tile_rows(B, 9)
    Tr = host(T[rows])
    assert np.isfinite(Tr).all()
    assert rowrel(Tr, oracle.prob2vec(P[rows], R)) <= TOL_F32


# Products whose tiles all do the same work (M and N multiples of 256, no
# echelon range) run on a persistent grid that walks several tiles per
# work-group, loading each next tile's first stage while the previous
# output drains: 512 tiles here, so every work-group takes two, with a K tail
# (K = 300) and NaN row padding; project with its row norms, restore, and the
# fp32 bound product (whose second pass reads the output back).

@pytest.mark.parametrize("op_dtype", OP_DTYPES, ids=_name)
def test_persistent_tile_walk(op_dtype):
    B, K, N = 16384, 300, 2048
    print("persistent tile walk", _name(op_dtype), B, K, N, flush=True)
    X, Q = _mat(B, K, 81, op_dtype), _mat(N, K, 82, op_dtype, 1 / np.sqrt(K))
    ldk = _ld(K, op_dtype)
    T, xn = gsm.gs_project(nan_padded(X, ldk, op_dtype), nan_padded(Q, ldk, op_dtype), out_dtype=torch.float32,
                           xnorm2=True)
    Tc, Qr = _mat(B, K, 83, op_dtype), _mat(K, N, 84, op_dtype)
    Td, Qd = nan_padded(Tc, ldk, op_dtype), nan_padded(Qr, _ld(N, op_dtype, 8), op_dtype)
    Xr = gsm.gs_reconstruct(Td, Qd, out_dtype=torch.float32)
    T2 = _mat(B, K, 85, op_dtype)
    Y = gsm.gs_reconstruct(Td, Qd, T2=nan_padded(T2, ldk, op_dtype), bind="mul", out_dtype=torch.float32)
    torch.cuda.synchronize()
    rows = _tile_rows(B, 86)
    for got in (T, Xr, Y):
        assert np.isfinite(host(got[rows])).all()
    assert rowrel(host(T[rows]), oracle.project(X[rows], Q)) <= TOL_F32
    np.testing.assert_allclose(host(xn), oracle.row_norms(X) ** 2, rtol=1e-4)
    Xo = oracle.reconstruct(Tc[rows], Qr)
    assert rowrel(host(Xr[rows]), Xo) <= TOL_F32
    assert rowrel(host(Y[rows]), oracle.bind(Xo, oracle.reconstruct(T2[rows], Qr))) <= TOL_F32
    # every tile was written (the outputs start uninitialised)
    assert torch.isfinite(Xr).all().item() and torch.isfinite(Y).all().item() and torch.isfinite(T).all().item()


@pytest.mark.parametrize("op_dtype", OP_DTYPES, ids=_name)
def test_large_tiles_ragged_columns(op_dtype):
    # whole row blocks with a ragged last column tile (N = 1000 = 3 x 256 +
    # 232; 128 x 4 = 512 tiles, one work-group each), both output types
    B, K, N = 32768, 300, 1000
    print("large tiles, ragged columns", _name(op_dtype), B, K, N, flush=True)
    X, Q = _mat(B, K, 87, op_dtype), _mat(N, K, 88, op_dtype, 1 / np.sqrt(K))
    ldk = _ld(K, op_dtype)
    for out_dtype in (torch.float32, torch.bfloat16):
        T = gsm.gs_project(nan_padded(X, ldk, op_dtype), nan_padded(Q, ldk, op_dtype), out_dtype=out_dtype)
        torch.cuda.synchronize()
        rows = _tile_rows(B, 89)
        Tg = host(T[rows])
        assert np.isfinite(Tg).all() and torch.isfinite(T.float()).all().item()
        tol = TOL_F32 if out_dtype == torch.float32 else TOL_BF16
        assert rowrel(Tg, oracle.project(X[rows], Q)) <= tol


@pytest.mark.parametrize("op_dtype", OP_DTYPES, ids=_name)
@pytest.mark.parametrize("out_dtype", [torch.float32, torch.bfloat16], ids=_name)
def test_large_tiles_unaligned_outputs(op_dtype, out_dtype):
    # outputs whose rows are not 16-byte aligned (a view starting one element
    # into an odd-strided buffer): every tile leaves through the element
    # stores; the buffer's columns outside the view stay untouched
    print("large tiles, unaligned outputs", _name(op_dtype), _name(out_dtype), flush=True)
    tol = TOL_F32 if out_dtype == torch.float32 else TOL_BF16

    def view(B, N):
        buf = torch.full((B, N + 3), float("nan"), device="cuda", dtype=out_dtype)
        return buf, buf[:, 1:N + 1]

    def untouched(buf, N):
        return torch.isnan(buf[:, 0].float()).all().item() and torch.isnan(buf[:, N + 1:].float()).all().item()

    B, K, N = 16384, 300, 1000            # project: 64 x 4 tiles, ragged last column tile
    X, Q = _mat(B, K, 91, op_dtype), _mat(N, K, 92, op_dtype, 1 / np.sqrt(K))
    ldk = _ld(K, op_dtype)
    buf, T = view(B, N)
    gsm.gs_project(nan_padded(X, ldk, op_dtype), nan_padded(Q, ldk, op_dtype), out=T)
    torch.cuda.synchronize()
    rows = _tile_rows(B, 93)
    assert torch.isfinite(T.float()).all().item() and untouched(buf, N)
    assert rowrel(host(T[rows]), oracle.project(X[rows], Q)) <= tol

    B, r, D = 8192, 45, 2100              # restore: 32 x 9 tiles
    Tc, Qr = _mat(B, r, 94, op_dtype), _mat(r, D, 95, op_dtype)
    buf, Xo = view(B, D)
    gsm.gs_reconstruct(nan_padded(Tc, _ld(r, op_dtype), op_dtype), nan_padded(Qr, _ld(D, op_dtype, 8), op_dtype),
                       out=Xo)
    torch.cuda.synchronize()
    rows = _tile_rows(B, 96)
    assert torch.isfinite(Xo.float()).all().item() and untouched(buf, D)
    assert rowrel(host(Xo[rows]), oracle.reconstruct(Tc[rows], Qr)) <= tol


# ------------- row sweep / scored products (>= 256 row blocks of 256, 256-column blocks)
#
# With Q the identity, coordinates and codebook coordinates are themselves the
# D-space vectors, so the oracle's dense cosine / dot similarity and softmax
# apply directly to T and R.  Ragged row count, a codebook size that leaves a
# partial column block, r not a multiple of the K-step or of a 16-byte chunk,
# NaN row padding; bf16 and fp32 operands.

SWEEP_B, SWEEP_M, SWEEP_R = 65573, 600, 300


@pytest.fixture(scope="module", params=OP_DTYPES, ids=_name)
def sweep_case(request):
    dt = request.param
    T = _mat(SWEEP_B, SWEEP_R, 21, dt)
    R = _mat(SWEEP_M, SWEEP_R, 22, dt)
    ld = _ld(SWEEP_R, dt)
    Td, Rd = nan_padded(T, ld, dt), nan_padded(R, ld, dt)
    rows = _tile_rows(SWEEP_B, 23)
    return T, R, Td, Rd, rows


@pytest.mark.parametrize("norms", ["computed", "given"])
def test_sweep_similarity_cosine(sweep_case, norms):
    T, R, Td, Rd, rows = sweep_case
    print("sweep similarity cosine", Td.dtype, norms, flush=True)
    qn = cn = None
    if norms == "given":
        qn = dev(oracle.row_norms(T) ** 2)
        cn = dev(oracle.row_norms(R))
    S, idx = gsm.gs_similarity(Td, Rd, qnorm2=qn, cnorm=cn, mode="cosine")
    torch.cuda.synchronize()
    So = oracle.similarity(T[rows], R, oracle.COSINE)
    Sg = host(S[rows])
    assert np.isfinite(Sg).all()
    assert rowrel(Sg, So) <= TOL_F32
    argmax_exact(idx[rows], T[rows], R, None if qn is None else host(qn[rows]), None if cn is None else host(cn))
    # whole batch: the returned index points at a maximal score of its row
    Sf = S.float()
    assert torch.all(Sf.gather(1, idx.long()[:, None])[:, 0] >= Sf.max(dim=1).values).item()


def test_sweep_similarity_dot_argmax_only(sweep_case):
    T, R, Td, Rd, rows = sweep_case
    print("sweep similarity dot argmax", Td.dtype, flush=True)
    _, idx = gsm.gs_similarity(Td, Rd, mode="dot", scale=0.5, scores=False)
    torch.cuda.synchronize()
    argmax_exact(idx[rows], T[rows], R, mode="dot", scale=0.5)


@pytest.mark.parametrize("norms", ["computed", "given"])
def test_sweep_attention(sweep_case, norms):
    T, R, Td, Rd, rows = sweep_case
    print("sweep attention", Td.dtype, norms, flush=True)
    qn = cn = None
    if norms == "given":
        qn = dev(oracle.row_norms(T) ** 2)
        cn = dev(oracle.row_norms(R))
    A, _ = gsm.gs_attention(Td, Rd, qnorm2=qn, cnorm=cn, mode="cosine", beta=8.0)
    torch.cuda.synchronize()
    Ao = oracle.softmax(oracle.similarity(T[rows], R, oracle.COSINE), 8.0)
    Ag = host(A[rows])
    assert np.isfinite(Ag).all()
    assert rowrel(Ag, Ao) <= TOL_F32
    assert torch.allclose(A.sum(dim=1), torch.ones(A.shape[0], device=A.device), atol=1e-4)


def test_sweep_cosine_argmax_only(sweep_case):
    # no scores requested: the fused row sweep, norms taken from T and R
    T, R, Td, Rd, rows = sweep_case
    print("sweep cosine argmax", Td.dtype, flush=True)
    _, idx = gsm.gs_similarity(Td, Rd, mode="cosine", scores=False)
    torch.cuda.synchronize()
    argmax_exact(idx[rows], T[rows], R)


# ---------- whole rows in one 256-column tile: row argmax / softmax in the epilogue
#
# With a codebook of at most 256 entries every tile of the scored product
# holds whole rows, so the argmax and the softmax are taken in the product's
# epilogue from the four column quarters of the tile.  M = 200 leaves one
# quarter partly and one wholly outside the codebook; M = 256 fills the tile.

ROWS_B, ROWS_R = 65573, 300


@pytest.fixture(scope="module", params=[(dt, m) for dt in OP_DTYPES for m in (200, 256)],
                ids=lambda p: "%s-M%d" % (_name(p[0]), p[1]))
def rows_case(request):
    dt, M = request.param
    T = _mat(ROWS_B, ROWS_R, 31, dt)
    R = _mat(M, ROWS_R, 32 + M, dt)
    ld = _ld(ROWS_R, dt)
    Td, Rd = nan_padded(T, ld, dt), nan_padded(R, ld, dt)
    rows = _tile_rows(ROWS_B, 33)
    return T, R, Td, Rd, rows


@pytest.mark.parametrize("norms", ["computed", "given"])
def test_whole_row_similarity_cosine(rows_case, norms):
    T, R, Td, Rd, rows = rows_case
    print("whole-row similarity cosine", Td.dtype, R.shape[0], norms, flush=True)
    qn = cn = None
    if norms == "given":
        qn = dev(oracle.row_norms(T) ** 2)
        cn = dev(oracle.row_norms(R))
    S, idx = gsm.gs_similarity(Td, Rd, qnorm2=qn, cnorm=cn, mode="cosine")
    torch.cuda.synchronize()
    So = oracle.similarity(T[rows], R, oracle.COSINE)
    Sg = host(S[rows])
    assert np.isfinite(Sg).all()
    assert rowrel(Sg, So) <= TOL_F32
    argmax_exact(idx[rows], T[rows], R, None if qn is None else host(qn[rows]), None if cn is None else host(cn))
    # every row: the index is the first maximum of the stored scores
    assert torch.equal(idx.long(), torch.argmax(S, dim=1))


def test_whole_row_similarity_dot(rows_case):
    T, R, Td, Rd, rows = rows_case
    print("whole-row similarity dot", Td.dtype, R.shape[0], flush=True)
    S, idx = gsm.gs_similarity(Td, Rd, mode="dot", scale=0.25)
    torch.cuda.synchronize()
    So = oracle.similarity(T[rows], R, oracle.DOT, 0.25)
    assert rowrel(host(S[rows]), So) <= TOL_F32
    argmax_exact(idx[rows], T[rows], R, mode="dot", scale=0.25)
    assert torch.equal(idx.long(), torch.argmax(S, dim=1))


@pytest.mark.parametrize("mode", ["cosine", "dot"])
def test_whole_row_argmax_only(rows_case, mode):
    # no scores requested: the argmax comes from the epilogue and nothing else
    # is written
    T, R, Td, Rd, rows = rows_case
    print("whole-row argmax only", Td.dtype, R.shape[0], mode, flush=True)
    _, idx = gsm.gs_similarity(Td, Rd, mode=mode, scale=0.5, scores=False)
    torch.cuda.synchronize()
    argmax_exact(idx[rows], T[rows], R, mode=mode, scale=0.5)
    S, idx2 = gsm.gs_similarity(Td, Rd, mode=mode, scale=0.5)
    assert torch.equal(idx, idx2)


@pytest.mark.parametrize("beta", [8.0, -3.0])
def test_whole_row_attention(rows_case, beta):
    T, R, Td, Rd, rows = rows_case
    print("whole-row attention", Td.dtype, R.shape[0], beta, flush=True)
    A, O = gsm.gs_attention(Td, Rd, mode="cosine", beta=beta, weighted_sum=True, out_dtype=torch.float32)
    torch.cuda.synchronize()
    Ao = oracle.softmax(oracle.similarity(T[rows], R, oracle.COSINE), beta)
    Ag = host(A[rows])
    assert np.isfinite(Ag).all()
    assert rowrel(Ag, Ao) <= TOL_F32
    assert torch.allclose(A.sum(dim=1), torch.ones(A.shape[0], device=A.device), atol=1e-4)
    # the weighted sum reads the normalised weights back
    assert rowrel(host(O[rows]), oracle.prob2vec(Ao, R)) <= TOL_F32


# ------------------------------------- lower-echelon R (GS_ECHELON) on the large tiles
#
# R from compress is lower echelon, R[j, k] == 0 for k > j; with the flag the
# large-tile products skip the K-steps whose part of R is zero.  On a clean
# echelon R the flagged and unflagged calls agree exactly (the skipped terms
# are exact zeros); NaN put where a flagged call never reads (R[j, k] with k
# in a later 256-block than j) shows the skip is taken, and the results still
# match the oracle on the clean R.


def echelon_pair(M, r, dtype, seed):
    """(clean lower-echelon R, the same with NaN in the blocks a flagged call skips)."""
    R = np.tril(_mat(M, r, seed, dtype))
    j, k = np.meshgrid(np.arange(M), np.arange(r), indexing="ij")
    dirty = R.copy()
    dirty[(k // 256) > (j // 256)] = np.nan
    return R, dirty


@pytest.mark.parametrize("op_dtype", OP_DTYPES, ids=_name)
def test_echelon_prob2vec(op_dtype):
    B, M, r = 8200, 2050, 2000
    print("echelon prob2vec", _name(op_dtype), B, M, r, flush=True)
    P = wl.dirichlet_probs(B, M, 0.5, 41)
    if op_dtype == torch.bfloat16:
        P = wl.round_bf16(P)
    R, Rnan = echelon_pair(M, r, op_dtype, 42)
    ldp, ldr = _ld(M, op_dtype), _ld(r, op_dtype)
    Pd = nan_padded(P, ldp, op_dtype)
    full = gsm.gs_prob2vec(Pd, nan_padded(R, ldr, op_dtype), out_dtype=torch.float32)
    flagged = gsm.gs_prob2vec(Pd, nan_padded(R, ldr, op_dtype), out_dtype=torch.float32, echelon=True)
    skipped = gsm.gs_prob2vec(Pd, nan_padded(Rnan, ldr, op_dtype), out_dtype=torch.float32, echelon=True)
    torch.cuda.synchronize()
    assert torch.equal(full, flagged)
    rows = _tile_rows(B, 43)
    Tr = host(skipped[rows])
    assert np.isfinite(Tr).all()
    assert rowrel(Tr, oracle.prob2vec(P[rows], R)) <= TOL_F32


@pytest.mark.parametrize("op_dtype", OP_DTYPES, ids=_name)
@pytest.mark.parametrize("mode", ["cosine", "dot"])
def test_echelon_similarity(op_dtype, mode):
    B, M, r = 65573, 600, 500
    print("echelon similarity", _name(op_dtype), mode, B, M, r, flush=True)
    T = _mat(B, r, 44, op_dtype)
    R, Rnan = echelon_pair(M, r, op_dtype, 45)
    ld = _ld(r, op_dtype)
    Td = nan_padded(T, ld, op_dtype)
    qn = dev(oracle.row_norms(T) ** 2)
    m = oracle.COSINE if mode == "cosine" else oracle.DOT
    S0, i0 = gsm.gs_similarity(Td, nan_padded(R, ld, op_dtype), qnorm2=qn, mode=mode, scale=0.5)
    S1, i1 = gsm.gs_similarity(Td, nan_padded(R, ld, op_dtype), qnorm2=qn, mode=mode, scale=0.5, echelon=True)
    S2, i2 = gsm.gs_similarity(Td, nan_padded(Rnan, ld, op_dtype), qnorm2=qn, mode=mode, scale=0.5, echelon=True)
    torch.cuda.synchronize()
    assert torch.equal(S0, S1) and torch.equal(i0, i1)
    rows = _tile_rows(B, 46)
    So = oracle.similarity(T[rows], R, m, 0.5)
    Sg = host(S2[rows])
    assert np.isfinite(Sg).all()
    assert rowrel(Sg, So) <= TOL_F32
    argmax_exact(i2[rows], T[rows], R, host(qn[rows]), None, mode=mode, scale=0.5)


def test_echelon_similarity_norms_from_t_keep_full_range():
    # cosine with ||x|| taken from T: the flagged call walks the whole K range
    # (so it reads the whole of R) and still agrees exactly
    dt = torch.bfloat16
    B, M, r = 65573, 600, 500
    print("echelon similarity, norms from T", B, M, r, flush=True)
    T = _mat(B, r, 47, dt)
    R, _ = echelon_pair(M, r, dt, 48)
    ld = _ld(r, dt)
    Td, Rd = nan_padded(T, ld, dt), nan_padded(R, ld, dt)
    S0, i0 = gsm.gs_similarity(Td, Rd, mode="cosine")
    S1, i1 = gsm.gs_similarity(Td, Rd, mode="cosine", echelon=True)
    torch.cuda.synchronize()
    assert torch.equal(S0, S1) and torch.equal(i0, i1)
    rows = _tile_rows(B, 49)
    assert rowrel(host(S1[rows]), oracle.similarity(T[rows], R, oracle.COSINE)) <= TOL_F32


def test_echelon_attention_weighted_sum():
    dt = torch.float32
    B, M, r = 65573, 600, 500
    print("echelon attention + weighted sum", B, M, r, flush=True)
    T = _mat(B, r, 50, dt)
    R, Rnan = echelon_pair(M, r, dt, 51)
    ld = _ld(r, dt)
    Td = nan_padded(T, ld, dt)
    qn = dev(oracle.row_norms(T) ** 2)
    A0, O0 = gsm.gs_attention(Td, nan_padded(R, ld, dt), qnorm2=qn, beta=4.0, weighted_sum=True)
    A1, O1 = gsm.gs_attention(Td, nan_padded(R, ld, dt), qnorm2=qn, beta=4.0, weighted_sum=True, echelon=True)
    A2, O2 = gsm.gs_attention(Td, nan_padded(Rnan, ld, dt), qnorm2=qn, beta=4.0, weighted_sum=True, echelon=True)
    torch.cuda.synchronize()
    assert torch.equal(A0, A1) and torch.equal(O0, O1)
    rows = _tile_rows(B, 52)
    Ao = oracle.softmax(oracle.similarity(T[rows], R, oracle.COSINE), 4.0)
    Ag, Og = host(A2[rows]), host(O2[rows])
    assert np.isfinite(Ag).all() and np.isfinite(Og).all()
    assert rowrel(Ag, Ao) <= TOL_F32
    assert rowrel(Og, oracle.prob2vec(Ao, R)) <= TOL_F32


def test_echelon_on_compressed_rank_deficient_codebook():
    # R as gs_compress returns it for a codebook with duplicated rows (rank
    # below M, pivots shifted left): flagged and unflagged products agree
    # exactly, and match the oracle's dense definitions
    M, D, B = 1100, 2048, 16400
    print("echelon, compressed rank-deficient codebook", M, D, B, flush=True)
    C = wl.bipolar_codebook(M, D, 71)
    rng = np.random.default_rng(72)
    tgt = rng.choice(M, size=110, replace=False)
    src = rng.choice(np.setdiff1d(np.arange(M), tgt), size=110)
    C[tgt] = C[src]
    Q, R, r, kept, cn = gsm.gs_compress(dev(C), q_dtype=torch.float32, r_dtype=torch.float32)
    torch.cuda.synchronize()
    assert r == M - 110
    Rh = host(R)
    assert np.all(np.triu(Rh, 1) == 0)                    # R[j, k] == 0 for k > j
    P = wl.dirichlet_probs(B, M, 0.5, 73)
    Pd = dev(P)
    T0 = gsm.gs_prob2vec(Pd, R)
    T1 = gsm.gs_prob2vec(Pd, R, echelon=True)
    X = _mat(B, D, 74, torch.float32)
    Tx, xn = gsm.gs_project(dev(X), Q, xnorm2=True)
    S0, i0 = gsm.gs_similarity(Tx, R, qnorm2=xn, cnorm=cn)
    S1, i1 = gsm.gs_similarity(Tx, R, qnorm2=xn, cnorm=cn, echelon=True)
    torch.cuda.synchronize()
    assert torch.equal(T0, T1)
    assert torch.equal(S0, S1) and torch.equal(i0, i1)
    rows = _tile_rows(B, 75)
    Qo = oracle.compress(C)[0]
    assert rowrel(host(T1[rows]), oracle.project(oracle.prob2vec(P[rows], C), Qo)) <= TOL_F32
    So = oracle.similarity(X[rows], C, oracle.COSINE)
    assert rowrel(host(S1[rows]), So) <= TOL_F32
    argmax_exact(i1[rows], host(Tx[rows]), host(R), host(xn[rows]), host(cn))


# ---------------------------- more entries than dimensions (D < M): partitioned bases
#
# The paper's treatment of D < M: split the M entries into subsets of at most
# D and give each its own orthonormal basis; after the restore, the subsets
# are put side by side again.  gs_compress_partitioned stacks the subsets'
# bases in Q and puts their coordinates on R's block diagonal; each block is
# checked against the oracle's compression of that subset, and the calls on
# the stacked form against the oracle's dense definitions.


def partitioned_codebook():
    """100 x 32 bipolar codebook with a duplicate inside a subset, one across
    subsets and a negation: subsets of 32 have ranks 31, 31, 32, 4."""
    C = wl.bipolar_codebook(100, 32, 61)
    C[20] = C[5]          # inside subset 0
    C[40] = -C[3]         # subset 1 repeats a direction of subset 0: independent within subset 1
    C[50] = C[41]         # inside subset 1
    return C


@pytest.mark.parametrize("dt", [torch.float32, torch.bfloat16], ids=_name)
def test_partitioned_codebook_d_below_m(dt):
    M, D, B = 100, 32, 300
    print("partitioned codebook", M, D, B, _name(dt), flush=True)
    C = partitioned_codebook()
    Q64, R64, r64, ranks, kept, cn = gsm.gs_compress_partitioned(dev(C), subset=32)
    torch.cuda.synchronize()
    # each block is the oracle's compression of its subset
    off = 0
    Qh, Rh = host(Q64), host(R64)
    for g, m0 in enumerate(range(0, M, 32)):
        Cg = C[m0:m0 + 32]
        Qo, Ro, ko, ro = oracle.compress(Cg)
        assert ranks[g] == ro
        assert np.abs(Qh[off:off + ro] - Qo).max() <= 1e-12
        assert np.abs(Rh[m0:m0 + len(Cg), off:off + ro] - Ro).max() <= 1e-12 * np.abs(Ro).max()
        assert list(host(kept[off:off + ro]).astype(int)) == list(ko + m0)
        Rz = Rh[m0:m0 + len(Cg)].copy()
        Rz[:, off:off + ro] = 0
        assert np.all(Rz == 0)                        # block diagonal
        off += ro
    assert r64 == off == sum(ranks) == 31 + 31 + 32 + 4
    assert np.abs(Rh @ Qh - C).max() <= 1e-12 * np.abs(C).max()
    assert np.all(np.triu(Rh, 1) == 0)                # lower echelon
    # calls on the stacked form (the benchmark's element types)
    Q, R, r, ranks2, kept2, cn = gsm.gs_compress_partitioned(dev(C), subset=32, q_dtype=dt, r_dtype=dt)
    X = _mat(B, D, 62, dt)
    P = wl.dirichlet_probs(B, M, 0.5, 63)
    if dt == torch.bfloat16:
        P = wl.round_bf16(P)
    T, xn = gsm.gs_project(dev(X, dt), Q, xnorm2=True)
    S, idx = gsm.gs_similarity(T, R, qnorm2=xn, cnorm=cn, mode="cosine", echelon=True)
    Sd, _ = gsm.gs_similarity(T, R, mode="dot", scale=0.5, echelon=True)
    V = gsm.gs_reconstruct(gsm.gs_prob2vec(dev(P, dt), R, out_dtype=dt, echelon=True), Q, out_dtype=torch.float32)
    torch.cuda.synchronize()
    tol = TOL_BF16 if dt == torch.bfloat16 else TOL_F32      # bf16: Q and R rounded from fp64
    So = oracle.similarity(X, C, oracle.COSINE)
    assert rowrel(host(S), So) <= tol
    assert rowrel(host(Sd), oracle.similarity(X, C, oracle.DOT, 0.5)) <= tol
    argmax_exact(idx, host(T), host(R), host(xn), host(cn))
    assert rowrel(host(V), oracle.prob2vec(P, C)) <= tol


def test_partitioned_equals_plain_compress_when_m_fits():
    C = rq_codebook("binary", 60, 500, 64)
    a = gsm.gs_compress(dev(C))
    b = gsm.gs_compress_partitioned(dev(C), subset=60)
    c = gsm.gs_compress_partitioned(dev(C))                  # default subset D >= M
    torch.cuda.synchronize()
    for x in (b, c):
        assert x[2] == a[2] and torch.equal(x[0], a[0]) and torch.equal(x[1], a[1]) and torch.equal(x[4], a[3])


# ------------------------------------------- binding of restored vectors

@pytest.mark.parametrize("B,D,L", [(37, 4096, 4096), (33, 1024, 128), (5, 8192, 8192), (9, 64, 2), (300, 512, 512)])
@pytest.mark.parametrize("op", ["conv", "corr"])
@pytest.mark.parametrize("dt", [torch.float32, torch.bfloat16], ids=["f32", "bf16"])
def test_bind_circular(B, D, L, op, dt):
    print("bind", op, B, D, L, dt, flush=True)
    rng = np.random.default_rng(D + L + B)
    X = rng.standard_normal((B, D)).astype(np.float32)
    Y = rng.standard_normal((B, D)).astype(np.float32)
    if dt == torch.bfloat16:
        X, Y = wl.round_bf16(X), wl.round_bf16(Y)
    Z = gsm.gs_bind_restored(dev(X, dt), dev(Y, dt), op=op, L=L, out_dtype=torch.float32)
    Zb = gsm.gs_bind_restored(dev(X, dt), dev(Y, dt), op=op, L=L, out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    Zo = oracle.circular(X, Y, L, corr=(op == "corr"))
    assert rowrel(host(Z), Zo) <= TOL_F32
    assert rowrel(host(Zb), Zo) <= TOL_BF16


@pytest.mark.parametrize("L", [1 << k for k in range(1, 14)])
@pytest.mark.parametrize("op", ["conv", "corr"])
@pytest.mark.parametrize("dt", [torch.float32, torch.bfloat16], ids=["f32", "bf16"])
@pytest.mark.parametrize("split", ["full", "partial"])
def test_bind_circular_every_block_length(L, op, dt, split):
    # the transform is compiled once per block length: every length from 2 to
    # 8192, with rows of 8192 values (every work-group holding 4096 values)
    # and, where blocks are shorter than 4096, rows of 6144 values (the
    # second work-group of a row holding fewer blocks)
    if split == "partial" and L > 2048:
        pytest.skip("blocks of 4096 and more always take one work-group each")
    B, D = 3, (6144 if split == "partial" else 8192)
    print("bind all L", op, L, D, dt, flush=True)
    rng = np.random.default_rng(1000 + L)
    X = rng.standard_normal((B, D)).astype(np.float32)
    Y = rng.standard_normal((B, D)).astype(np.float32)
    if dt == torch.bfloat16:
        X, Y = wl.round_bf16(X), wl.round_bf16(Y)
    Z = gsm.gs_bind_restored(dev(X, dt), dev(Y, dt), op=op, L=L, out_dtype=torch.float32)
    Zb = gsm.gs_bind_restored(dev(X, dt), dev(Y, dt), op=op, L=L, out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    Zo = oracle.circular(X, Y, L, corr=(op == "corr"))
    assert rowrel(host(Z), Zo) <= TOL_F32
    assert rowrel(host(Zb), Zo) <= TOL_BF16


def test_bind_restored_codebook_vectors():
    # restored bipolar codebook vectors (reconstruct of their coordinates):
    # bind two of them, unbind with the second, and compare each step with the
    # oracle's sums; also the element-wise product against gs_reconstruct's
    # fused bind
    D, M = 1024, 12
    C = rq_codebook("bipolar", M, D, 91)
    Q, R, r, kept, cn = gsm.gs_compress(dev(C), q_dtype=torch.float32, r_dtype=torch.float32)
    idx_a, idx_b = np.arange(M), np.roll(np.arange(M), 3)
    Xa = gsm.gs_reconstruct(R[idx_a].contiguous(), Q)
    Xb = gsm.gs_reconstruct(R[idx_b].contiguous(), Q)
    Zc = gsm.gs_bind_restored(Xa, Xb, op="conv")
    Zu = gsm.gs_bind_restored(Zc, Xb, op="corr")
    Zm = gsm.gs_bind_restored(Xa, Xb, op="mul")
    Zf = gsm.gs_reconstruct(R[idx_a].contiguous(), Q, T2=R[idx_b].contiguous(), bind="mul")
    torch.cuda.synchronize()
    Ca, Cb = C[idx_a], C[idx_b]
    Zco = oracle.circular(Ca, Cb, D)
    assert rowrel(host(Zc), Zco) <= TOL_F32
    assert rowrel(host(Zu), oracle.circular(Zco, Cb, D, corr=True)) <= TOL_F32
    assert rowrel(host(Zm), oracle.bind(Ca, Cb)) <= TOL_F32
    assert rowrel(host(Zm), host(Zf)) <= 1e-6


@pytest.mark.parametrize("dt", [torch.float32, torch.bfloat16], ids=["f32", "bf16"])
def test_bind_xor_binary(dt):
    # restored binary vectors carry rounding noise around 0 and 1; the bits
    # (value >= 0.5) decide, bit-exact against the oracle on the same inputs
    rng = np.random.default_rng(5)
    B, D = 300, 4100
    Xb = rng.integers(0, 2, (B, D)).astype(np.float32) + rng.uniform(-0.2, 0.2, (B, D)).astype(np.float32)
    Yb = rng.integers(0, 2, (B, D)).astype(np.float32) + rng.uniform(-0.2, 0.2, (B, D)).astype(np.float32)
    if dt == torch.bfloat16:
        Xb, Yb = wl.round_bf16(Xb), wl.round_bf16(Yb)
    Z = gsm.gs_bind_restored(dev(Xb, dt), dev(Yb, dt), op="xor", out_dtype=torch.float32)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(host(Z), oracle.xor(Xb, Yb))


# ------------------------------------------------ sparse probability rows (CSR)
#
# prob2vec of rows given by their stored entries: the oracle sums the dense
# rows (zeros elsewhere); rows without entries, column indices in any order,
# r not a multiple of the 256-coordinate chunk, both value and output types.


def csr_rows(B, M, per_row, seed, sort=True):
    """Seeded CSR rows with 0 .. per_row entries (Dirichlet values on the
    chosen columns) and the dense matrix they stand for."""
    g = np.random.default_rng(seed)
    counts = g.integers(0, per_row + 1, size=B)
    counts[::7] = 0                                   # some empty rows
    rowptr = np.zeros(B + 1, np.int64)
    rowptr[1:] = np.cumsum(counts)
    cols = np.empty(rowptr[-1], np.int32)
    vals = np.empty(rowptr[-1], np.float32)
    dense = np.zeros((B, M), np.float32)
    for b in range(B):
        c = g.choice(M, size=counts[b], replace=False)
        if sort:
            c = np.sort(c)
        v = g.dirichlet(np.full(max(counts[b], 1), 0.5))[: counts[b]].astype(np.float32)
        cols[rowptr[b]:rowptr[b + 1]] = c
        vals[rowptr[b]:rowptr[b + 1]] = v
        dense[b, c] = v
    return rowptr, cols, vals, dense


@pytest.mark.parametrize("dt", [torch.float32, torch.bfloat16], ids=_name_early)
@pytest.mark.parametrize("M,D,per_row,sort", [(1000, 1500, 24, True), (300, 800, 300, False), (40, 256, 5, True)])
def test_prob2vec_sparse(dt, M, D, per_row, sort):
    B = 777
    print("sparse prob2vec", M, D, per_row, sort, _name_early(dt), flush=True)
    C = rq_codebook("binary", M, D, 90 + M)
    Qo, Ro, kept, r = oracle.compress(C)
    rowptr, cols, vals, dense = csr_rows(B, M, per_row, M, sort)
    if dt == torch.bfloat16:
        vals = wl.round_bf16(vals)
        dense = wl.round_bf16(dense)
    Rin = Ro.astype(np.float32) if dt == torch.float32 else wl.round_bf16(Ro.astype(np.float32))
    rp, cd = torch.from_numpy(rowptr).cuda(), torch.from_numpy(cols).cuda()
    vd, Rd = dev(vals, dt), dev(Rin, dt)
    for out_dtype in (torch.float32, torch.bfloat16):
        T = gsm.gs_prob2vec_sparse(rp, cd, vd, Rd, out_dtype=out_dtype)
        Tdense = gsm.gs_prob2vec(dev(dense, dt), Rd, out_dtype=torch.float32)
        torch.cuda.synchronize()
        Tg = host(T)
        assert np.isfinite(Tg).all()
        tol = TOL_F32 if (dt == torch.float32 and out_dtype == torch.float32) else TOL_BF16
        # the dense definition on the stored entries (in span: t = Q v)
        assert rowrel(Tg, oracle.project(oracle.prob2vec(dense, C), Qo)) <= tol
        # and the dense call on the same values, to fp32 accumulation
        if out_dtype == torch.float32:
            assert rowrel(Tg, host(Tdense)) <= 1e-5
        empty = np.nonzero(np.diff(rowptr) == 0)[0]
        assert np.all(Tg[empty] == 0.0)


def test_prob2vec_sparse_skips_out_of_range_entries():
    # stored indices outside [0, M) and entries past rowptr[B] contribute nothing
    M, D, B = 50, 300, 40
    C = rq_codebook("bipolar", M, D, 95)
    Qo, Ro, kept, r = oracle.compress(C)
    rowptr, cols, vals, dense = csr_rows(B, M, 6, 96)
    bad = cols.copy()
    bad[::5] = -1
    bad[1::5] = M
    keep = (bad >= 0) & (bad < M)
    dense2 = np.zeros_like(dense)
    for b in range(B):
        for e in range(rowptr[b], rowptr[b + 1]):
            if keep[e]:
                dense2[b, bad[e]] += vals[e]
    # stored arrays one entry longer than rowptr[B] says (never read)
    cols_x = np.concatenate([bad, [3]]).astype(np.int32)
    vals_x = np.concatenate([vals, [1.0]]).astype(np.float32)
    T = gsm.gs_prob2vec_sparse(torch.from_numpy(rowptr).cuda(), torch.from_numpy(cols_x).cuda(), dev(vals_x),
                               dev(Ro.astype(np.float32)))
    torch.cuda.synchronize()
    assert rowrel(host(T), oracle.project(oracle.prob2vec(dense2, C), Qo)) <= TOL_F32


# ------------------------------------------------ padded bases (k > M)
#
# The basis completed to k vectors by unit vectors and, optionally, turned by
# an orthogonal k x k matrix (a normalised Hadamard matrix here).  Compared
# element by element with the oracle's padded compression, and the calls on
# padded coordinates with the oracle's dense definitions.


@pytest.mark.parametrize("transform", [False, True])
@pytest.mark.parametrize("M,D,k,dup", [(22, 1024, 64, 0.0), (40, 700, 64, 0.1), (100, 2000, 256, 0.1)])
def test_compress_padded(M, D, k, dup, transform):
    print("padded", M, D, k, dup, transform, flush=True)
    C = rq_codebook("bipolar", M, D, 120 + M, dup=dup)
    H = (wl.hadamard_codebook(k).astype(np.float64) / math.sqrt(k)) if transform else None
    Qo, Ro, kept_o, ro = oracle.compress_padded(C, k, H)
    Hd = None if H is None else dev(H, torch.float64)
    Q, R, r, kept, cn = gsm.gs_compress_padded(dev(C), k, Hd)
    torch.cuda.synchronize()
    assert r == ro == M - int(round(dup * M))
    assert list(host(kept[:r]).astype(int)) == list(kept_o) and np.all(host(kept[r:]) == -1)
    Qg, Rg = host(Q), host(R)
    assert np.abs(Qg - Qo).max() <= 1e-12
    assert np.abs(Rg - Ro).max() <= 1e-12 * np.abs(Ro).max()
    assert np.abs(Qg @ Qg.T - np.eye(k)).max() <= 1e-12
    np.testing.assert_allclose(host(cn), oracle.row_norms(C), rtol=1e-6)
    # the operators on padded coordinates (fp32 copies)
    Q32, R32, _, _, _ = gsm.gs_compress_padded(dev(C), k, Hd, q_dtype=torch.float32, r_dtype=torch.float32)
    B = 300
    P = wl.dirichlet_probs(B, M, 0.5, M)
    X = oracle.prob2vec(P, C) + np.sqrt(0.1) * np.random.default_rng(M).standard_normal((B, D))
    T, xn = gsm.gs_project(dev(X), Q32, xnorm2=True)
    S, idx = gsm.gs_similarity(T, R32, qnorm2=xn, cnorm=cn, mode="cosine")
    Tp = gsm.gs_prob2vec(dev(P), R32)
    V = gsm.gs_reconstruct(Tp, Q32)
    torch.cuda.synchronize()
    So = oracle.similarity(X, C, oracle.COSINE)
    assert rowrel(host(S), So) <= TOL_F32
    argmax_exact(idx, host(T), host(R32), host(xn), host(cn))
    assert rowrel(host(V), oracle.prob2vec(P, C)) <= TOL_F32
    assert rowrel(host(Tp), oracle.project(oracle.prob2vec(P, C), Qo)) <= TOL_F32
