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
VIEW_BAND = 1e-6   # relative band around the patch-selection threshold

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


def acceptable_view_keeps(s_b: np.ndarray, tau: float) -> set:
    """Every view mask an implementation may return for one sample whose fused
    view scores differ from the float64 oracle's s_b by rounding: a view with
    |s_v - tau| <= VIEW_BAND*max(|tau|, 1e-30) may fall on either side of the
    threshold, and when no view passes, any view within VIEW_BAND (relative) of
    the best score may be the fallback. Outside those bands the mask is exact."""
    s_b = np.asarray(s_b, np.float64)
    band = VIEW_BAND * max(abs(tau), 1e-30)
    sure = (s_b - tau) > band
    unsure = np.nonzero(np.abs(s_b - tau) <= band)[0]
    out = set()
    for bits in range(1 << len(unsure)):
        keep = sure.copy()
        for i, v in enumerate(unsure):
            if (bits >> i) & 1:
                keep[v] = True
        if keep.any():
            out.add(tuple(int(x) for x in keep))
            continue
        best = s_b.max()
        for v in np.nonzero(s_b >= best - VIEW_BAND * max(abs(best), 1e-30))[0]:
            k = np.zeros(len(s_b), np.int64)
            k[v] = 1
            out.add(tuple(int(x) for x in k))
    return out


def check_view_keep(scores: np.ndarray, tau: float, gpu_keep: np.ndarray) -> int:
    """Patch-selection comparator: each sample's GPU view mask must be one of
    acceptable_view_keeps (exactly the oracle's mask when no score lies in a
    band). Returns the number of views that fell in a threshold band."""
    n_band = 0
    for b in range(scores.shape[0]):
        ok = acceptable_view_keeps(scores[b], tau)
        got = tuple(int(x) for x in gpu_keep[b])
        assert got in ok, f"sample {b}: GPU view mask {got} not among {sorted(ok)} (scores {scores[b]})"
        n_band += int(np.sum(np.abs(scores[b] - tau) <= VIEW_BAND * max(abs(tau), 1e-30)))
    return n_band


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
    """kind: 'bf16' (bf16/f32 output from bf16 input), 'fp8' or 'f32'. Every
    element of ref must be computed (no NaN rows)."""
    assert not np.isnan(ref).any(), f"{what}: reference has uncomputed rows"
    err = np.abs(got - ref)
    rl2 = row_rel_l2(got, ref)
    stats = dict(max_abs=float(err.max()) if err.size else 0.0,
                 max_row_rel_l2=float(rl2.max()) if rl2.size else 0.0,
                 rows=int(np.prod(ref.shape[:-1])))
    if kind == "fp8" and err.size:
        # elementwise diagnostic: error against 6e-2 of the output's rms
        rms = float(np.sqrt(np.mean(ref * ref)))
        stats["max_abs_over_rms"] = float(err.max() / max(rms, 1e-30))
        stats["frac_over_6e-2_rms"] = float(np.mean(err > 6e-2 * rms))
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


def softmax_scale(D: int) -> float:
    return 1.0 / math.sqrt(D)
