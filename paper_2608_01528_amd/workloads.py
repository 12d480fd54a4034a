"""Seeded synthetic inputs shaped like the paper's VSA workloads.

This module generates inputs only.  Both the HIP path (through the tests and
the benchmark) and the fp64 oracle receive the arrays it returns; it holds no
code of either side.

Codebooks follow the paper's description of atomic vectors: pseudorandom,
quasi-orthogonal in high dimension (Sec. 2.1), bipolar +-1 or binary {0,1}.
Probability rows stand in for the perception front-end's attribute
distributions (Sec. 2.2, Sec. 3.1): a softmax of Gaussian logits, or a
Dirichlet draw.  Query vectors for hard selection (Sec. 3.1) are mixtures of
codebook vectors plus Gaussian noise.  RAVEN / I-RAVEN are not used: these
inputs stand in for their shapes (attribute codebook sizes, panels per
problem, vector dimension).

Large batches are generated in chunks of CHUNK rows, each from its own child
seed, so any chunk can be regenerated on its own.  Normal distributions are
read as N(mu, sigma^2): "N(0,2)" has standard deviation sqrt(2), "N(0,0.1)"
has standard deviation sqrt(0.1).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

CHUNK = 4096

STREAM_CODEBOOK = 0
STREAM_PROBS = 1
STREAM_NOISE = 2
STREAM_DUP = 3
STREAM_PROBS_B = 4


def rng(seed: int, stream: int, sub: int = 0) -> np.random.Generator:
    """Independent generator for (seed, stream, sub-index)."""
    return np.random.default_rng(np.random.SeedSequence(seed, spawn_key=(stream, sub)))


# --------------------------------------------------------------- codebooks

def bipolar_codebook(M: int, D: int, seed: int, sub: int = 0) -> np.ndarray:
    """M x D i.i.d. fair +-1 entries (fp32)."""
    g = rng(seed, STREAM_CODEBOOK, sub)
    return (2.0 * g.integers(0, 2, size=(M, D)) - 1.0).astype(np.float32)


def binary_codebook(M: int, D: int, seed: int, sub: int = 0) -> np.ndarray:
    """M x D i.i.d. Bernoulli(0.5) {0,1} entries (fp32)."""
    g = rng(seed, STREAM_CODEBOOK, sub)
    return g.integers(0, 2, size=(M, D)).astype(np.float32)


def hadamard_codebook(n: int) -> np.ndarray:
    """Sylvester-Hadamard matrix of order n (a power of two): +-1 rows that are
    exactly orthogonal."""
    assert n >= 1 and (n & (n - 1)) == 0
    H = np.ones((1, 1), np.float32)
    while H.shape[0] < n:
        H = np.block([[H, H], [H, -H]])
    return H


def duplicate_rows(C: np.ndarray, frac: float, seed: int):
    """Overwrite round(frac*M) distinct target rows with copies of rows drawn
    from the non-target rows.  Returns (C', targets, sources)."""
    M = C.shape[0]
    n = int(round(frac * M))
    g = rng(seed, STREAM_DUP)
    targets = np.sort(g.choice(M, size=n, replace=False))
    pool = np.setdiff1d(np.arange(M), targets)
    sources = g.choice(pool, size=n, replace=True)
    C = C.copy()
    C[targets] = C[sources]
    return C, targets, sources


# ----------------------------------------------------------- probabilities

def _chunks(B: int):
    for c in range((B + CHUNK - 1) // CHUNK):
        yield c, c * CHUNK, min(B, (c + 1) * CHUNK)


def softmax_probs(B: int, M: int, sigma: float, seed: int,
                  stream: int = STREAM_PROBS, chunks=None) -> np.ndarray:
    """Rows p = softmax(z), z ~ N(0, sigma^2)^M (fp32).  `chunks` restricts
    generation to the listed chunk indices (rows of other chunks are zero)."""
    P = np.zeros((B, M), np.float32)
    for c, a, b in _chunks(B):
        if chunks is not None and c not in chunks:
            continue
        z = rng(seed, stream, c).standard_normal((b - a, M)) * sigma
        z -= z.max(axis=1, keepdims=True)
        e = np.exp(z)
        P[a:b] = (e / e.sum(axis=1, keepdims=True)).astype(np.float32)
    return P


def dirichlet_probs(B: int, M: int, alpha: float, seed: int,
                    stream: int = STREAM_PROBS, chunks=None) -> np.ndarray:
    """Rows p ~ Dirichlet(alpha * 1_M) (fp32)."""
    P = np.zeros((B, M), np.float32)
    for c, a, b in _chunks(B):
        if chunks is not None and c not in chunks:
            continue
        P[a:b] = rng(seed, stream, c).dirichlet(np.full(M, alpha), size=b - a).astype(np.float32)
    return P


def noisy_queries(P: np.ndarray, C: np.ndarray, var: float, seed: int,
                  chunks=None) -> np.ndarray:
    """Hard-selection query rows: a probability mixture of codebook rows plus
    N(0, var) noise in every component (fp32)."""
    B = P.shape[0]
    D = C.shape[1]
    X = np.zeros((B, D), np.float32)
    sd = np.float32(np.sqrt(var))
    for c, a, b in _chunks(B):
        if chunks is not None and c not in chunks:
            continue
        X[a:b] = P[a:b] @ C
        X[a:b] += sd * rng(seed, STREAM_NOISE, c).standard_normal((b - a, D), dtype=np.float32)
    return X


# -------------------------------------------------------------- bfloat16

def to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns (uint16), round to nearest even.  Finite
    inputs only."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    return ((u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def round_bf16(a: np.ndarray) -> np.ndarray:
    """fp32 values rounded to the nearest bf16 (returned as fp32)."""
    return bf16_bits_to_f32(to_bf16_bits(a))


# ------------------------------------------------------- named workloads

@dataclass
class Workload:
    name: str
    seed: int
    D: int
    Ms: list
    B: int
    codebook: str          # "bipolar" | "binary"
    probs: str             # "softmax" | "dirichlet"
    prob_param: float      # sigma for softmax, alpha for dirichlet
    noise_var: float = 0.0  # >0: hard-selection queries X = P C + noise
    dup_frac: float = 0.0
    bf16: bool = False
    pairs: bool = False    # bind workload: two probability batches
    note: str = ""
    ops: list = field(default_factory=list)


WORKLOADS = {
    "tiny": Workload("tiny", 1, 1024, [10], 16, "bipolar", "softmax", 1.0,
                     ops=["compress", "prob2vec", "similarity", "argmax", "attention"]),
    "vsa": Workload("vsa", 2, 1024, [5, 6, 10, 22], 4096 * 16, "bipolar", "softmax",
                    float(np.sqrt(2.0)),
                    note="4096 problems x 16 panels (8 context + 8 candidates)",
                    ops=["compress", "prob2vec", "similarity", "attention"]),
    "large": Workload("large", 3, 8192, [256], 65536, "bipolar", "dirichlet", 0.5,
                      noise_var=0.1,
                      ops=["compress", "project", "similarity", "attention"]),
    "binary": Workload("binary", 4, 4096, [1000], 16384, "binary", "dirichlet", 0.05,
                       pairs=True,
                       ops=["compress", "prob2vec", "similarity", "reconstruct_bind",
                            "project"]),
    "stress": Workload("stress", 5, 16384, [2048], 262144, "bipolar", "dirichlet", 0.5,
                       noise_var=0.1, dup_frac=0.1, bf16=True,
                       ops=["compress", "project", "prob2vec", "similarity", "attention",
                            "reconstruct"]),
}


def codebook(w: Workload, i: int = 0) -> np.ndarray:
    """Codebook i of workload w (fp32; duplicates applied)."""
    M = w.Ms[i]
    if w.codebook == "bipolar":
        C = bipolar_codebook(M, w.D, w.seed, i)
    else:
        C = binary_codebook(M, w.D, w.seed, i)
    if w.dup_frac > 0:
        C, _, _ = duplicate_rows(C, w.dup_frac, w.seed)
    return C


def probabilities(w: Workload, i: int = 0, B: int | None = None, stream: int = STREAM_PROBS,
                  chunks=None) -> np.ndarray:
    """Probability batch for codebook i of workload w (first B rows)."""
    B = w.B if B is None else B
    M = w.Ms[i]
    # one stream per codebook: shift the stream id by 8 per codebook index
    s = stream + 8 * i
    if w.probs == "softmax":
        return softmax_probs(B, M, w.prob_param, w.seed, s, chunks)
    return dirichlet_probs(B, M, w.prob_param, w.seed, s, chunks)


# ------------------------------------------------- device-side large batches

def device_dirichlet_half(B: int, M: int, seed: int, torch, device, dtype=None):
    """B x M rows of Dirichlet(1/2 * 1_M), generated on the device: Gamma(1/2)
    equals Z^2 / 2 for a standard normal Z, so normalising Z^2 gives the
    Dirichlet(1/2) law exactly.  Seeded torch generator on the device."""
    g = torch.Generator(device=device)
    g.manual_seed(seed * 1000003 + 11)
    Z = torch.randn((B, M), generator=g, device=device, dtype=torch.float32)
    Z = Z * Z
    P = Z / Z.sum(dim=1, keepdim=True)
    return P if dtype is None else P.to(dtype)


def device_noisy_queries(P, C, var: float, seed: int, torch, dtype=None, chunk: int = 16384):
    """Hard-selection queries on the device: rows p C + N(0, var) noise, built
    in row chunks (fp32 arithmetic, optional cast of the result)."""
    B, D = P.shape[0], C.shape[1]
    out = torch.empty((B, D), dtype=dtype or torch.float32, device=P.device)
    g = torch.Generator(device=P.device)
    g.manual_seed(seed * 1000003 + 29)
    Cf = C.float()
    sd = float(np.sqrt(var))
    for a in range(0, B, chunk):
        b = min(B, a + chunk)
        x = P[a:b].float() @ Cf
        x += sd * torch.randn((b - a, D), generator=g, device=P.device, dtype=torch.float32)
        out[a:b] = x.to(out.dtype)
    return out
