"""Helpers for the GPU parity tests: device transfer and the comparison rules.

Comparison rules (what "match the oracle" means):
* floating point: row-scaled maximum relative error
      max_ij |g_ij - o_ij| / max(max_j |o_ij|, 1e-30)
  at most 1e-4 for fp32 paths and 2e-2 for paths with bf16 inputs;
* integers (rank, kept rows, argmax): bit-exact, except argmax rows whose top
  two oracle scores are closer than the rounding band of the GPU's inputs,
  where any index inside the band is accepted (and counted).
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


def check_argmax(gpu_idx, S_oracle, band_rel=1e-5):
    """Exact argmax except inside the near-tie band; returns the near-tie count."""
    S = np.asarray(S_oracle, np.float64)
    gi = np.asarray(gpu_idx).astype(np.int64)
    best = S.argmax(axis=1)  # numpy: first occurrence = lowest index
    top = S[np.arange(len(S)), best]
    band = band_rel * np.maximum(np.abs(S).max(axis=1), 1e-30)
    srt = np.sort(S, axis=1)
    gap = srt[:, -1] - srt[:, -2] if S.shape[1] > 1 else np.full(len(S), np.inf)
    near = gap <= 2 * band
    exact = ~near
    assert np.array_equal(gi[exact], best[exact]), \
        "argmax mismatch on rows %s" % np.nonzero(gi[exact] != best[exact])[0][:10]
    if near.any():
        got = S[np.nonzero(near)[0], gi[near]]
        assert np.all(got >= top[near] - 2 * band[near])
    return int(near.sum())
