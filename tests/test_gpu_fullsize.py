"""Parity at the configured full sizes, in the shapes and launch configuration
the benchmark uses.

The GPU processes every row of each batch; the fp64 oracle recomputes a
sample of rows one by one from the same inputs, read back from the device:
4096 seeded rows, the first and last 16 rows, and the two rows on either side
of every 256-row tile boundary.  Two kinds of check:

* against the oracle's dense D-space definitions on the workload's inputs
  (tolerance 1e-4 for fp32 paths, 2e-2 for bf16 storage);
* the argmax against the oracle's exact scores of the very values the kernel
  read (its coordinates, codebook coordinates and norms, upcast exactly):
  bit-exact wherever the top two are further apart than twice the a-priori
  bound of the fp32 evaluation (tests/gpu_util.py), near-ties counted.

Properties that hold at any size are checked on every row: the returned index
is the first maximum of the returned scores, softmax rows sum to one, cosines
lie in [-1, 1].
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_01528_amd import gramspace as gsm
from paper_2608_01528_amd import workloads as wl
from tests.gpu_util import (TOL_BF16, TOL_F32, check_argmax_bound, dev, exact_scores_bound, host, rowrel)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    gsm.lib()


def sample_rows(B, seed, n_random=4096):
    """4096 seeded rows, the first and last 16, and rows 256k - 1 and 256k of
    every tile boundary."""
    fixed = set(range(min(16, B))) | set(range(max(0, B - 16), B))
    for k in range(256, B, 256):
        fixed |= {k - 1, k}
    rnd = np.random.default_rng(seed).choice(B, size=min(n_random, B), replace=False)
    return np.array(sorted(fixed | set(int(x) for x in rnd)))


def take(t, rows):
    return t.index_select(0, torch.from_numpy(rows).to(t.device))


def whole_batch_properties(S, idx, A=None, cosine=True):
    """Every row: idx is the lowest index of the row maximum of the returned
    scores (exact), softmax rows sum to one, cosines within [-1, 1]."""
    Sg = S.float()
    mx = Sg.max(dim=1, keepdim=True).values
    first = (Sg == mx).to(torch.int32).argmax(dim=1)          # first True = lowest maximal index
    assert torch.equal(first.to(torch.int32), idx.to(torch.int32))
    if cosine:
        assert Sg.abs().max().item() <= 1.0 + 1e-4
    if A is not None:
        assert torch.allclose(A.sum(dim=1), torch.ones(A.shape[0], device=A.device), atol=1e-4)


def test_large_workload_full_size():
    w = wl.WORKLOADS["large"]
    C = wl.codebook(w)
    print("large: compress", C.shape, flush=True)
    Cd = dev(C)
    Qo, Ro, kept_o, ro = oracle.compress(C)
    Q64, R64, r64, kept64, _ = gsm.gs_compress(Cd)
    Q, R, r, kept, cnorm = gsm.gs_compress(Cd, q_dtype=torch.float32, r_dtype=torch.float32)
    torch.cuda.synchronize()
    assert r == r64 == ro == 256
    assert np.abs(host(Q64) - Qo).max() <= 1e-12
    assert np.abs(host(R64) - Ro).max() <= 1e-12 * np.abs(Ro).max()
    print("large: batch", flush=True)
    P = wl.device_dirichlet_half(w.B, 256, w.seed, torch, "cuda")
    X = wl.device_noisy_queries(P, Cd, w.noise_var, w.seed, torch)
    T, xn = gsm.gs_project(X, Q, xnorm2=True)
    # R from compress is lower echelon: flagged as the benchmark does
    S, idx = gsm.gs_similarity(T, R, qnorm2=xn, cnorm=cnorm, mode="cosine", echelon=True)
    A, _ = gsm.gs_attention(T, R, qnorm2=xn, cnorm=cnorm, mode="cosine", beta=16.0, echelon=True)
    torch.cuda.synchronize()
    whole_batch_properties(S, idx, A)
    rows = sample_rows(w.B, 3)
    print("large: oracle on %d rows" % len(rows), flush=True)
    Xs = host(take(X, rows))
    assert rowrel(host(take(T, rows)), oracle.project(Xs, Qo)) <= TOL_F32
    np.testing.assert_allclose(host(take(xn, rows)), oracle.row_norms(Xs) ** 2, rtol=TOL_F32)
    So = oracle.similarity(Xs, C, oracle.COSINE)
    assert rowrel(host(take(S, rows)), So) <= TOL_F32
    assert rowrel(host(take(A, rows)), oracle.softmax(So, 16.0)) <= TOL_F32
    # argmax on the kernel's own inputs
    Se, E = exact_scores_bound(host(take(T, rows)), host(R), host(take(xn, rows)), host(cnorm))
    print("large: near-ties", check_argmax_bound(host(take(idx, rows)), Se, E), "of", len(rows), flush=True)


def test_binary_workload_full_size():
    w = wl.WORKLOADS["binary"]
    C = wl.codebook(w)
    print("binary: compress", C.shape, flush=True)
    Cd = dev(C)
    Qo, Ro, kept_o, ro = oracle.compress(C)
    Q64, R64, r64, _, _ = gsm.gs_compress(Cd)
    Q, R, r, kept, cnorm = gsm.gs_compress(Cd, q_dtype=torch.float32, r_dtype=torch.float32)
    torch.cuda.synchronize()
    assert r == r64 == ro == 1000
    assert np.abs(host(Q64) - Qo).max() <= 1e-12
    assert np.abs(host(R64) - Ro).max() <= 1e-12 * np.abs(Ro).max()
    rows = sample_rows(w.B, 4)
    print("binary: batch", flush=True)
    Pa = wl.probabilities(w, 0)
    Pb = wl.probabilities(w, 0, stream=wl.STREAM_PROBS_B)
    Ta = gsm.gs_prob2vec(dev(Pa), R, echelon=True)
    Tb = gsm.gs_prob2vec(dev(Pb), R, echelon=True)
    S, idx = gsm.gs_similarity(Ta, R, cnorm=cnorm, mode="cosine", echelon=True)
    Y = gsm.gs_reconstruct(Ta, Q, T2=Tb, bind="mul")
    Ty = gsm.gs_project(Y, Q)
    torch.cuda.synchronize()
    whole_batch_properties(S, idx)
    print("binary: oracle on %d rows" % len(rows), flush=True)
    Va = oracle.prob2vec(Pa[rows], C)
    Vb = oracle.prob2vec(Pb[rows], C)
    assert rowrel(host(take(Ta, rows)), oracle.project(Va, Qo)) <= TOL_F32
    So = oracle.similarity(Va, C, oracle.COSINE)
    assert rowrel(host(take(S, rows)), So) <= TOL_F32
    Yo = oracle.bind(Va, Vb)
    assert rowrel(host(take(Y, rows)), Yo) <= TOL_F32
    assert rowrel(host(take(Ty, rows)), oracle.project(Yo, Qo)) <= TOL_F32
    # argmax on the kernel's own inputs (||x|| summed from Ta by the kernel)
    Se, E = exact_scores_bound(host(take(Ta, rows)), host(R), None, host(cnorm), norms_given=False)
    print("binary: near-ties", check_argmax_bound(host(take(idx, rows)), Se, E), "of", len(rows), flush=True)


@pytest.mark.timeout(900)
def test_stress_workload_full_size():
    w = wl.WORKLOADS["stress"]
    C = wl.codebook(w)
    print("stress: oracle compress", C.shape, flush=True)
    Qo, Ro, kept_o, ro = oracle.compress(C)
    assert ro == 2048 - 205
    Cd = dev(C)
    print("stress: gpu compress", flush=True)
    Q64, R64, r64, kept64, _ = gsm.gs_compress(Cd)
    torch.cuda.synchronize()
    assert r64 == ro
    assert list(host(kept64).astype(int)) == list(kept_o)
    assert np.abs(host(Q64) - Qo).max() <= 1e-12
    assert np.abs(host(R64) - Ro).max() <= 1e-12 * np.abs(Ro).max()
    del Q64, R64
    Q, R, r, kept, cnorm = gsm.gs_compress(Cd, q_dtype=torch.bfloat16, r_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    assert r == ro
    print("stress: batch", flush=True)
    P = wl.device_dirichlet_half(w.B, 2048, w.seed, torch, "cuda", dtype=torch.bfloat16)
    X = wl.device_noisy_queries(P, Cd, w.noise_var, w.seed, torch, dtype=torch.bfloat16)
    print("stress: calls", flush=True)
    # the benchmark's step: the same calls, flags and output types
    T, xn = gsm.gs_project(X, Q, out_dtype=torch.bfloat16, xnorm2=True)
    T2 = gsm.gs_prob2vec(P, R, out_dtype=torch.bfloat16, echelon=True)
    S, idx, A = gsm.gs_similarity_attention(T, R, qnorm2=xn, cnorm=cnorm, mode="cosine", beta=16.0,
                                            echelon=True)
    Xr = gsm.gs_reconstruct(T2, Q, out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    whole_batch_properties(S, idx, A)
    rows = sample_rows(w.B, 5)
    print("stress: oracle on %d rows" % len(rows), flush=True)
    Xs = host(take(X, rows))
    Ps = host(take(P, rows))
    assert rowrel(host(take(T, rows)), oracle.project(Xs, Qo)) <= TOL_BF16
    np.testing.assert_allclose(host(take(xn, rows)), oracle.row_norms(Xs) ** 2, rtol=1e-4)
    Vs = oracle.prob2vec(Ps, C)
    assert rowrel(host(take(T2, rows)), oracle.project(Vs, Qo)) <= TOL_BF16
    assert rowrel(host(take(Xr, rows)), Vs) <= TOL_BF16
    So = oracle.similarity(Xs, C, oracle.COSINE)
    assert rowrel(host(take(S, rows)), So) <= TOL_BF16
    assert rowrel(host(take(A, rows)), oracle.softmax(So, 16.0)) <= TOL_BF16
    # argmax: the oracle's exact scores of the bf16 coordinates and codebook
    # coordinates the kernel read, with the norms it was given
    print("stress: argmax on the kernel's inputs", flush=True)
    Se, E = exact_scores_bound(host(take(T, rows)), host(R), host(take(xn, rows)), host(cnorm))
    near = check_argmax_bound(host(take(idx, rows)), Se, E)
    print("stress: near-ties %d of %d rows (median bound %.2e)" % (near, len(rows), float(np.median(E))),
          flush=True)
