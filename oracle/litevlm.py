"""Plain float64 definitions of the LiteVLM select + prefill path (test infrastructure only).

Paper: "LiteVLM: A Low-Latency Vision-Language Model Inference Pipeline for
Resource-Constrained Environments" (arXiv 2506.07416). Only tests, the smoke
check and the benchmark's CPU-baseline leg use this module.

Each function restates the passage it follows and the reading taken where the
paper is silent. Everything runs in float64 on the exact stored input values.
"""
from __future__ import annotations

import math
from typing import Optional, Sequence

import numpy as np

from . import e4m3


# --------------------------------------------------------------------------- inputs

def decode_stored(x: np.ndarray, dtype: str, scale: float = 1.0) -> np.ndarray:
    """Exact float64 values of stored bits: fp32 as is, bf16 bit patterns
    (uint16) widened to fp32, fp8 E4M3FN bytes through the OCP table times the
    per-tensor scale."""
    if dtype == "f32":
        return np.asarray(x, dtype=np.float32).astype(np.float64)
    if dtype == "bf16":
        u = np.asarray(x, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
        return u.view(np.float32).astype(np.float64)
    if dtype == "fp8":
        return e4m3.decode(x, scale)
    raise ValueError(dtype)


def decode_inputs(case):
    """(q, k, v) of a synthetic case as float64 arrays."""
    return (decode_stored(case.q, case.dtype, case.q_scale),
            decode_stored(case.k, case.dtype, case.k_scale),
            decode_stored(case.v, case.dtype, case.v_scale))


# --------------------------------------------------------------------------- patch selection

def view_scores(view_logit: np.ndarray, view_lexical: Optional[np.ndarray],
                w_lexical: float) -> np.ndarray:
    """Fused view score (Design section, Patch Selection Module paragraph: the
    final score of a view is a weighted sum of the lexical mapping and the
    module's logit). Reading: the logit enters through the logistic function
    so that both terms live on [0, 1], s_v = w*lex_v + (1-w)*sigmoid(logit_v),
    and a missing lexical term counts as 0. float64 throughout. Returns [B, N]."""
    logit = np.asarray(view_logit, dtype=np.float64)
    lex = np.zeros_like(logit) if view_lexical is None else np.asarray(view_lexical, np.float64)
    w = float(w_lexical)
    sig = 1.0 / (1.0 + np.exp(-logit))
    return w * lex + (1.0 - w) * sig


def patch_select(view_logit: np.ndarray, view_lexical: Optional[np.ndarray],
                 w_lexical: float, threshold: float) -> np.ndarray:
    """View selection at inference (Design section, Patch Selection Module
    paragraph): views whose fused score (view_scores) lies above a threshold
    are kept. Reading: "above" is strict (s_v > threshold); if no view passes,
    the single best view is kept (lowest index among equal scores), since a
    prompt needs at least one view. The decision is taken in float64 on the
    float64 fused score. Returns uint8 [B, N]."""
    s = view_scores(view_logit, view_lexical, w_lexical)
    tau = float(threshold)
    B, N = s.shape
    keep = np.zeros((B, N), np.uint8)
    for b in range(B):
        for v in range(N):
            keep[b, v] = 1 if s[b, v] > tau else 0
        if not keep[b].any():
            best = 0
            for v in range(1, N):
                if s[b, v] > s[b, best]:
                    best = v
            keep[b, best] = 1
    return keep


def token_keep_from_views(view_keep: np.ndarray, view_offsets: Sequence[int], S: int) -> np.ndarray:
    """Only the tiles of selected views reach the vision encoder, so only their
    visual tokens reach the LLM (Design section, Patch Selection Module
    paragraph; Experiments section, Training paragraph). Visual tokens of view v
    occupy [off[v], off[v+1]); text tokens [off[N], S) are always kept.
    Returns uint8 [B, S]."""
    B, N = view_keep.shape
    off = [int(o) for o in view_offsets]
    tk = np.zeros((B, S), np.uint8)
    for b in range(B):
        for v in range(N):
            if view_keep[b, v]:
                tk[b, off[v]:off[v + 1]] = 1
        tk[b, off[N]:] = 1
    return tk


def patch_selected_positions(token_keep_b: np.ndarray, V_full: int) -> np.ndarray:
    """Original positions of the patch-selected sequence of one sample: kept
    visual tokens ascending, then every text token."""
    S = token_keep_b.shape[0]
    vis = np.nonzero(token_keep_b[:V_full])[0]
    return np.concatenate([vis, np.arange(V_full, S)]).astype(np.int64)


# --------------------------------------------------------------------------- token scoring

def token_scores(q: np.ndarray, k: np.ndarray, token_keep: np.ndarray, V_full: int,
                 Hq: int, Hkv: int, scale: float, query_rows: Optional[int] = None) -> np.ndarray:
    """Visual-token importance (Design section, Token Selection Module
    paragraph: a standalone copy of the first decoder layer scores visual
    tokens in the manner of FastV, i.e. from self-attention, Related Work,
    Visual Token Compression).

    Reading: the head-averaged attention mass that the text rows put on each
    visual token. For query head h (KV head g = h // (Hq/Hkv)) and text token t
    at position p_t = V_b + t of the patch-selected sequence, the attention row
    is the causal softmax of q_t . k_j * scale over keys j = 0..p_t of that
    sequence (tokens of dropped views do not exist; the preceding text keys are
    included; no renormalisation over visual keys). The score of visual token j
    is the sum of those rows' entries at j over all (h, t), divided by Hq*T.
    Tokens of dropped views score -inf. q, k: float64 [B, S, H, D].

    query_rows = n keeps only the last n text tokens as query rows (divided by
    Hq*n instead): n = 1 is the FastV-style readout from the last token
    (Related Work, Visual Token Compression: FastV prunes by the attention the
    last token pays); n = T (the default) is the reading above.
    Returns float64 [B, V_full].
    """
    B, S = token_keep.shape
    T = S - V_full
    n = T if query_rows is None else int(query_rows)
    if not 1 <= n <= T:
        raise ValueError("query_rows must lie in 1..T")
    G = Hq // Hkv
    out = np.full((B, V_full), -np.inf)
    for b in range(B):
        idx = patch_selected_positions(token_keep[b], V_full)
        V_b = idx.shape[0] - T
        S_b = idx.shape[0]
        acc = np.zeros(V_b)
        tq = np.arange(T - n, T)                     # the query text tokens
        p = V_b + tq                                 # their positions in the selected sequence
        blocked = np.arange(S_b)[None, :] > p[:, None]
        for h in range(Hq):
            g = h // G
            qt = q[b, V_full + tq, h, :]             # [n, D] text query rows
            kp = k[b, idx, g, :]                     # [S_b, D] keys of the selected sequence
            logits = (qt @ kp.T) * scale
            logits[blocked] = -np.inf
            logits -= logits.max(axis=1, keepdims=True)
            e = np.exp(logits)
            prob = e / e.sum(axis=1, keepdims=True)
            acc += prob[:, :V_b].sum(axis=0)
        out[b, idx[:V_b]] = acc / (Hq * n)
    return out


# --------------------------------------------------------------------------- top-k

def keep_count(keep_ratio: float, V_b: int) -> int:
    """Visual tokens kept at compression ratio r (Results section, Visual Token
    Compression paragraph; Table 1 token counts): r is the fraction of visual
    tokens kept, text is never pruned, k = floor(r*V_b), evaluated in float64
    with a 1e-6 guard so that decimal ratios whose product is an integer are
    not rounded down by binary representation: k = min(V_b, floor(r*V_b + 1e-6))."""
    return int(min(V_b, math.floor(float(keep_ratio) * float(V_b) + 1e-6)))


def select_topk(scores_b: np.ndarray, token_keep_b: np.ndarray, V_full: int, k: int) -> np.ndarray:
    """Keep the k highest-scoring visual tokens of the patch-selected set,
    ordered by (score descending, original position ascending): exactly equal
    scores keep the lower position. Returns the kept positions ascending."""
    cand = np.nonzero(token_keep_b[:V_full])[0]
    order = np.lexsort((cand, -scores_b[cand]))     # primary: -score, secondary: position
    return np.sort(cand[order[:k]]).astype(np.int64)


# --------------------------------------------------------------------------- compaction

def compact(selected: Sequence[np.ndarray], V_full: int, S: int):
    """Compacted sequence per sample (Design section, Token Selection Module
    paragraph: pruning happens outside the LLM, which then prefills the shorter
    sequence). Reading: original order is kept, so kept visual positions
    ascending, then all text positions. Returns (kept_index int32 [sum S'_b],
    cu_seqlens int32 [B+1])."""
    parts, cu = [], [0]
    for sel in selected:
        row = np.concatenate([np.asarray(sel, np.int64), np.arange(V_full, S)])
        parts.append(row)
        cu.append(cu[-1] + row.shape[0])
    return (np.concatenate(parts).astype(np.int32) if parts else np.zeros(0, np.int32),
            np.asarray(cu, np.int32))


def gather_rows(x: np.ndarray, kept_index: np.ndarray, cu_seqlens: np.ndarray) -> np.ndarray:
    """Packed copy: row i of sample b is x[b, kept_index[i]] (exact bits)."""
    out = []
    for b in range(cu_seqlens.shape[0] - 1):
        out.append(x[b, kept_index[cu_seqlens[b]:cu_seqlens[b + 1]]])
    return np.concatenate(out, axis=0) if out else x[:0, 0]


# --------------------------------------------------------------------------- attention

def prefill_attention(qc: np.ndarray, kc: np.ndarray, vc: np.ndarray, cu_seqlens: np.ndarray,
                      Hq: int, Hkv: int, scale: float,
                      rows: Optional[Sequence[int]] = None, causal: bool = True) -> np.ndarray:
    """LLM prefill self-attention over the compacted sequence (Introduction and
    Related Work: the quadratic self-attention of the prefill stage is what
    token compression saves; Figure 3b). Per sample: O = softmax(Q K^T * scale
    with a causal mask) V, query head h reading KV head h // (Hq/Hkv), softmax
    taken in float64 after subtracting the row maximum.

    qc: float64 [total, Hq, D]; kc, vc: float64 [total, Hkv, D] packed by
    cu_seqlens. rows: optional packed row indices to compute (the rest are NaN).
    causal=False drops the mask (full attention; not part of the prefill path).
    Returns float64 [total, Hq, D].
    """
    total, _, D = qc.shape
    G = Hq // Hkv
    out = np.full((total, Hq, vc.shape[2]), np.nan)
    want = None if rows is None else np.zeros(total, bool)
    if want is not None:
        want[np.asarray(rows, np.int64)] = True
    for b in range(cu_seqlens.shape[0] - 1):
        lo, hi = int(cu_seqlens[b]), int(cu_seqlens[b + 1])
        if hi == lo:
            continue
        local = np.arange(hi - lo) if want is None else np.nonzero(want[lo:hi])[0]
        if local.size == 0:
            continue
        blocked = np.arange(hi - lo)[None, :] > local[:, None]
        if not causal:
            blocked[:] = False
        for h in range(Hq):
            g = h // G
            logits = (qc[lo + local, h, :] @ kc[lo:hi, g, :].T) * scale
            logits[blocked] = -np.inf
            logits -= logits.max(axis=1, keepdims=True)
            e = np.exp(logits)
            prob = e / e.sum(axis=1, keepdims=True)
            out[lo + local, h, :] = prob @ vc[lo:hi, g, :]
    return out


def decode_attention(q1: np.ndarray, k1: np.ndarray, v1: np.ndarray, kc: np.ndarray, vc: np.ndarray,
                     cu_seqlens: np.ndarray, Hq: int, Hkv: int, scale: float) -> np.ndarray:
    """Extend-one decode step over the compacted KV cache (Results section:
    decoding one token after the prefill, where token compression saves little
    because the work per token is one pass over the cached keys and values).
    Sample b's new token attends to the S'_b cached tokens of the compacted
    sequence (packed rows cu_seqlens[b] .. cu_seqlens[b+1] of kc, vc) and to
    itself, which comes last: o = softmax(q1 . [K; k1]^T * scale) [V; v1], query
    head h reading KV head h // (Hq/Hkv), softmax in float64 after subtracting
    the row maximum.

    q1: float64 [B, Hq, D]; k1, v1: float64 [B, Hkv, D]; kc, vc: float64
    [total, Hkv, D]. Returns float64 [B, Hq, D].
    """
    B, _, D = q1.shape
    G = Hq // Hkv
    out = np.zeros((B, Hq, v1.shape[2]))
    for b in range(B):
        lo, hi = int(cu_seqlens[b]), int(cu_seqlens[b + 1])
        for h in range(Hq):
            g = h // G
            keys = np.concatenate([kc[lo:hi, g, :], k1[b, g][None, :]], axis=0)
            vals = np.concatenate([vc[lo:hi, g, :], v1[b, g][None, :]], axis=0)
            logits = (keys @ q1[b, h]) * scale
            logits -= logits.max()
            p = np.exp(logits)
            p /= p.sum()
            out[b, h] = p @ vals
    return out


# --------------------------------------------------------------------------- whole path

def run_path(case, keep_ratio: Optional[float] = None, attention: bool = True,
             attention_rows: Optional[Sequence[int]] = None, query_rows: Optional[int] = None) -> dict:
    """All steps in order on a synthetic case: patch select, patch-selected
    scoring (over the last query_rows text tokens; all of them by default),
    k rule, top-k, compaction, gather, prefill attention."""
    r = case.keep_ratio if keep_ratio is None else keep_ratio
    q, k, v = decode_inputs(case)
    scale = 1.0 / math.sqrt(case.D)
    view_keep = patch_select(case.view_logit, case.view_lexical, case.w_lexical, case.threshold)
    tk = token_keep_from_views(view_keep, case.view_offsets, case.S)
    V_b = tk[:, :case.V_full].sum(axis=1).astype(np.int64)
    scores = token_scores(q, k, tk, case.V_full, case.Hq, case.Hkv, scale, query_rows=query_rows)
    k_b = np.array([keep_count(r, int(n)) for n in V_b], np.int64)
    selected = [select_topk(scores[b], tk[b], case.V_full, int(k_b[b])) for b in range(case.B)]
    kept_index, cu = compact(selected, case.V_full, case.S)
    res = dict(view_keep=view_keep, token_keep=tk, V_b=V_b, scores=scores, k_b=k_b,
               selected=selected, kept_index=kept_index, cu_seqlens=cu,
               qc_bits=gather_rows(case.q, kept_index, cu),
               kc_bits=gather_rows(case.k, kept_index, cu),
               vc_bits=gather_rows(case.v, kept_index, cu))
    if attention:
        res["o"] = prefill_attention(gather_rows(q, kept_index, cu), gather_rows(k, kept_index, cu),
                                     gather_rows(v, kept_index, cu), cu, case.Hq, case.Hkv, scale,
                                     rows=attention_rows)
    return res
