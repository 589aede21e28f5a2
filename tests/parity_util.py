"""Comparators shared by the GPU parity tests.

Selection: the GPU's kept set is checked against the oracle's float64 scores
with the near-tie band rule (exact outside a 1e-6 relative band around the
k-th score). Attention: elementwise tolerances per output precision, plus
per-row relative L2 as a second, stricter-in-the-tail measure.
"""
from __future__ import annotations

import math
import sys

import numpy as np
import torch

BAND = 1e-6

# attention tolerances
BF16_RTOL, BF16_ATOL = 2e-2, 1e-2       # elementwise |o - ref| <= atol + rtol*|ref|
BF16_ROW_L2 = 2e-2                      # per-row ||o - ref|| <= 2e-2 ||ref||
FP8_ROW_L2 = 6e-2                       # per-row relative L2 for E4M3 inputs
F32_RTOL, F32_ATOL = 1e-4, 1e-5


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def to_device(bits: np.ndarray, dtype: str) -> torch.Tensor:
    """Stored bits (synth encodings) -> device tensor of the matching torch dtype."""
    if dtype == "bf16":
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()
    if dtype == "fp8":
        return torch.from_numpy(np.ascontiguousarray(bits)).cuda()
    return torch.from_numpy(np.ascontiguousarray(bits, dtype=np.float32)).cuda()


def to_float64(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float64)


def bits_of(t: torch.Tensor) -> np.ndarray:
    """Raw stored bits of a device tensor as a numpy array (for bitwise checks)."""
    t = t.detach().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


def check_selection(ref_scores: np.ndarray, keep_b: np.ndarray, V_full: int, k: int,
                    gpu_sel: np.ndarray) -> tuple:
    """Band rule. Returns (identical_to_oracle, band_size)."""
    cand = np.nonzero(keep_b[:V_full])[0]
    sel = np.asarray(gpu_sel, np.int64)
    assert sel.shape[0] == k, f"GPU kept {sel.shape[0]} tokens, want {k}"
    assert np.all(np.diff(sel) > 0), "kept positions not strictly ascending"
    assert np.all(np.isin(sel, cand)), "GPU kept a token of a dropped view"
    if k == 0:
        return True, 0
    s = ref_scores
    order = np.lexsort((cand, -s[cand]))
    ref_sel = np.sort(cand[order[:k]])
    sk = s[cand[order[k - 1]]]
    hi = s[cand] > sk * (1 + BAND)
    lo = s[cand] < sk * (1 - BAND)
    band = ~(hi | lo)
    must = set(cand[hi].tolist())
    never = set(cand[lo].tolist())
    got = set(sel.tolist())
    missing = must - got
    extra = got & never
    assert not missing, f"{len(missing)} tokens above the band were dropped, e.g. {sorted(missing)[:5]}"
    assert not extra, f"{len(extra)} tokens below the band were kept, e.g. {sorted(extra)[:5]}"
    return bool(np.array_equal(ref_sel, sel)), int(band.sum())


def score_rel_err(ref: np.ndarray, got: np.ndarray) -> float:
    fin = np.isfinite(ref)
    assert np.array_equal(np.isneginf(ref), np.isneginf(got)), "-inf pattern differs"
    if not fin.any():
        return 0.0
    return float(np.max(np.abs(got[fin] - ref[fin]) / np.abs(ref[fin])))


def row_rel_l2(got: np.ndarray, ref: np.ndarray) -> np.ndarray:
    """Per (row, head) relative L2 error over the head dimension."""
    num = np.linalg.norm(got - ref, axis=-1)
    den = np.linalg.norm(ref, axis=-1)
    return num / np.maximum(den, 1e-30)


def check_attention(got: np.ndarray, ref: np.ndarray, kind: str, what: str = "") -> dict:
    """kind: 'bf16' (bf16/f32 output from bf16 input), 'fp8' or 'f32'."""
    err = np.abs(got - ref)
    rl2 = row_rel_l2(got, ref)
    stats = dict(max_abs=float(err.max()) if err.size else 0.0,
                 max_row_rel_l2=float(rl2.max()) if rl2.size else 0.0)
    if kind == "f32":
        bad = err > F32_ATOL + F32_RTOL * np.abs(ref)
        assert not bad.any(), f"{what}: fp32 tolerance exceeded at {bad.sum()} elements, {stats}"
    elif kind == "bf16":
        bad = err > BF16_ATOL + BF16_RTOL * np.abs(ref)
        assert not bad.any(), f"{what}: bf16 tolerance exceeded at {bad.sum()} elements, {stats}"
        assert stats["max_row_rel_l2"] <= BF16_ROW_L2, f"{what}: bf16 row L2 {stats}"
    elif kind == "fp8":
        assert stats["max_row_rel_l2"] <= FP8_ROW_L2, f"{what}: fp8 row L2 {stats}"
    else:
        raise ValueError(kind)
    return stats


def sample_rows(cu: np.ndarray, per_seq: int, seed: int) -> np.ndarray:
    """Packed row indices to check at full size: each sequence's first and
    last rows, rows around 128-row tile edges, and seeded random rows."""
    rng = np.random.default_rng(seed)
    rows = []
    for b in range(len(cu) - 1):
        lo, hi = int(cu[b]), int(cu[b + 1])
        n = hi - lo
        if n == 0:
            continue
        local = {0, n - 1, min(n - 1, 127), min(n - 1, 128), min(n - 1, 63), min(n - 1, 64)}
        local |= set(rng.integers(0, n, size=min(per_seq, n)).tolist())
        rows += [lo + i for i in sorted(local)]
    return np.asarray(rows, np.int64)


def softmax_scale(D: int) -> float:
    return 1.0 / math.sqrt(D)
