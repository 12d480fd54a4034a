"""Helpers for the GPU parity tests: device transfer and the comparison rules.

Comparison rules (what "match the oracle" means):
* floating point: row-scaled maximum relative error
      max_ij |g_ij - o_ij| / max(max_j |o_ij|, 1e-30)
  at most 1e-4 for fp32 paths and 2e-2 for paths with bf16 inputs;
* integers (rank, kept rows, argmax): bit-exact, except argmax rows whose top
  two exact scores are closer than twice an a-priori bound of the GPU's fp32
  evaluation error, where any index inside that band is accepted (and
  counted).  The bound (score_bound) follows the standard error analysis of
  a floating-point inner product: a sum of n products evaluated in fp32, in
  any order, is off by at most gamma_n = n u / (1 - n u) (u = 2^-24) times
  the sum of the products' magnitudes.
"""
import numpy as np
import torch

TOL_F32 = 1e-4
TOL_BF16 = 2e-2


def dev(a, dtype=torch.float32):
    return torch.from_numpy(np.ascontiguousarray(a)).to(device="cuda", dtype=dtype)


def host(t):
    if t.dtype == torch.bfloat16:
        t = t.float()
    return t.detach().cpu().numpy().astype(np.float64)


def rowrel(g, o):
    g = np.asarray(g, np.float64)
    o = np.asarray(o, np.float64)
    assert g.shape == o.shape, (g.shape, o.shape)
    if g.size == 0:
        return 0.0
    scale = np.maximum(np.abs(o).max(axis=1, keepdims=True), 1e-30)
    return float((np.abs(g - o) / scale).max())


U32 = 2.0 ** -24


def gamma(n):
    """gamma_n of the error analysis of an n-term fp32 sum of products."""
    return n * U32 / (1.0 - n * U32)


def score_bound(S_exact, absdot, factor, gam, rel):
    """Per-row bound of |S_gpu - S_exact| over the row's entries, where
    S_exact[i, j] = factor[i, j] * dot[i, j] is the score from the exact
    values of the kernel's inputs, absdot[i, j] the sum of the magnitudes of
    the products making up dot[i, j], `gam` the relative bound of the fp32
    accumulation (gamma of the number of terms, plus any rounding of the
    inputs) and `rel` the relative error of the scaling (norms, square roots,
    divisions)."""
    S = np.asarray(S_exact, np.float64)
    E = np.abs(np.asarray(factor, np.float64)) * gam * np.asarray(absdot, np.float64) + rel * np.abs(S)
    return E.max(axis=1)


def cosine_factor(qnorm2, cnorm, scale=1.0):
    """scale / (||x_i|| ||c_j||) as the kernel applies it (0 where a norm is 0)."""
    qn = np.sqrt(np.asarray(qnorm2, np.float64))[:, None]
    cn = np.asarray(cnorm, np.float64)[None, :]
    den = qn * cn
    return np.where(den > 0, scale / np.where(den > 0, den, 1.0), 0.0)


def check_argmax_bound(gpu_idx, S_exact, E_row):
    """Bit-exact argmax (lowest index on exact ties) wherever the exact top
    two scores of a row are more than 2 E_row apart; elsewhere the GPU's
    index must score within 2 E_row of the row maximum.  Returns the number
    of such near-tie rows."""
    S = np.asarray(S_exact, np.float64)
    gi = np.asarray(gpu_idx).astype(np.int64)
    E = np.asarray(E_row, np.float64)
    best = S.argmax(axis=1)  # numpy: first occurrence = lowest index
    top = S[np.arange(len(S)), best]
    srt = np.sort(S, axis=1)
    gap = srt[:, -1] - srt[:, -2] if S.shape[1] > 1 else np.full(len(S), np.inf)
    near = gap <= 2 * E
    exact = ~near
    assert np.array_equal(gi[exact], best[exact]), \
        "argmax mismatch on rows %s" % np.nonzero(gi[exact] != best[exact])[0][:10]
    if near.any():
        got = S[np.nonzero(near)[0], gi[near]]
        assert np.all(got >= top[near] - 2 * E[near])
    return int(near.sum())


def exact_scores_bound(T, R, qnorm2=None, cnorm=None, cosine=True, scale=1.0, norms_given=True, input_rel=0.0):
    """Exact scores of T (B x r) against R (M x r), both the values the
    kernel read (bf16 or fp32, upcast exactly), and the per-row bound of the
    fp32 evaluation.  Cosine norms: given (qnorm2, cnorm: the values passed to
    the kernel) or, when norms_given is False, summed by the kernel from T and
    R in fp32 (their relative error, gamma_r, joins `rel`).  input_rel: extra
    relative error of the inputs against the values the exact scores use."""
    import oracle
    T = np.asarray(T, np.float64)
    R = np.asarray(R, np.float64)
    r = T.shape[1]
    dot = oracle.similarity(T, R, oracle.DOT)
    absdot = oracle.similarity(np.abs(T), np.abs(R), oracle.DOT)
    if cosine:
        if qnorm2 is None:
            qnorm2 = (T * T).sum(1)
        if cnorm is None:
            cnorm = np.sqrt((R * R).sum(1))
        factor = cosine_factor(qnorm2, cnorm, scale)
    else:
        factor = np.full(dot.shape, float(scale))
    S = factor * dot
    rel = 8 * U32 + input_rel + (0.0 if (norms_given or not cosine) else gamma(r) + 2 * U32)
    return S, score_bound(S, absdot, factor, gamma(r) + input_rel, rel)
