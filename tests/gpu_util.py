"""Helpers for the GPU parity tests: host copies for the oracle and the tolerance check.

Tolerance (bf16 inputs, fp32 accumulation): over each compared output tensor,
max |gpu - oracle| <= 1e-2 and ||gpu - oracle||_2 / ||oracle||_2 <= 5e-3.
"""
import numpy as np

from synth import bits, compact_rows  # noqa: F401  (re-export)

MAX_ABS = 1e-2
REL_L2 = 5e-3
# Log-sum-exp of an append query. The kernel sums the weights after rounding
# each to bf16 (the values the P·V product uses), a relative error of at most
# 2^-8 per weight; when one key dominates the sum the whole sum can carry that
# error, so |lse_gpu - lse| <= ln(1 + 2^-8) = 3.90e-3 plus fp32 rounding of the
# scores and exponentials (below 1e-5 at these magnitudes).
APPEND_LSE_ATOL = 4e-3
# Decode keeps the weights in fp32 (hi + lo bf16 parts in the products).
DECODE_LSE_ATOL = 1e-4


def attn_stats(gpu, ref):
    g = np.asarray(gpu, np.float64)
    r = np.asarray(ref, np.float64)
    diff = g - r
    max_abs = float(np.abs(diff).max()) if diff.size else 0.0
    rel = float(np.linalg.norm(diff) / max(np.linalg.norm(r), 1e-300)) if diff.size else 0.0
    return max_abs, rel


def worst_row_head_rel(gpu, ref) -> float:
    """Largest rel-L2 over the 128-dim output vectors of single (row, head) pairs
    (vectors whose reference is all zeros, e.g. empty rows, are skipped)."""
    g = np.asarray(gpu, np.float64).reshape(-1, np.shape(gpu)[-1])
    r = np.asarray(ref, np.float64).reshape(g.shape)
    n = np.linalg.norm(r, axis=1)
    keep = n > 0
    if not keep.any():
        return 0.0
    return float((np.linalg.norm(g - r, axis=1)[keep] / n[keep]).max())


def assert_attn_close(gpu, ref, what: str = ""):
    """The tolerance is over the whole compared tensor; the worst single (row,
    head) vector's rel-L2 is reported beside it."""
    g = np.asarray(gpu, np.float64)
    assert np.all(np.isfinite(g)), f"{what}: non-finite output"
    max_abs, rel = attn_stats(g, ref)
    worst = worst_row_head_rel(g, ref)
    print(f"[parity] {what}: max_abs={max_abs:.3e} rel_l2={rel:.3e} "
          f"worst_row_head_rel_l2={worst:.3e}", flush=True)
    assert max_abs <= MAX_ABS and rel <= REL_L2, (what, max_abs, rel)
    return max_abs, rel


def sample_rows(lens, k: int, seed: int):
    """The longest row, the shortest row and k - 2 seeded random others."""
    lens = np.asarray(lens)
    n = lens.shape[0]
    rng = np.random.default_rng(seed)
    pick = {int(np.argmax(lens)), int(np.argmin(lens))}
    for r in rng.permutation(n):
        if len(pick) >= min(k, n):
            break
        pick.add(int(r))
    return np.array(sorted(pick), np.int64)
