"""Plain float64 definition of the Token Selection Module's front end (test
infrastructure only: tests, the smoke check and the benchmark's CPU-baseline
leg use it).

Paper: the Design section's Token Selection Module paragraph takes the first
decoder layer of the finetuned LLM and runs it standalone to score the visual
tokens; the Experiments section names the decoder (InternLM2.5, for the 2B
model). That layer's attention reads queries and keys produced from the hidden
states by a pre-attention RMS normalisation, linear projections and rotary
position embeddings. The paper prints none of these formulas; the readings
taken here are the decoder family's standard ones:

* RMS normalisation: x * gamma / sqrt(mean(x^2) + eps) over the model width.
* Projections: q = x_n W_q^T, k = x_n W_k^T, bias-free, W of shape [H*D, Dm].
* Rotary embedding, rotate-half pairing: element d < D/2 of a head is paired
  with element d + D/2 and the pair is rotated by the angle
  pos * theta^(-2d/D).
* Positions are those of the patch-selected sequence: tokens of dropped views
  do not exist, so a token's position is the number of kept tokens before it.

The keys are produced for every token (the scoring reads those of the kept
tokens only) and the queries for the text tokens.
"""
from __future__ import annotations

import numpy as np


def rms_norm(x: np.ndarray, gamma: np.ndarray, eps: float) -> np.ndarray:
    """x * gamma / sqrt(mean(x**2, last axis) + eps), float64."""
    x = np.asarray(x, np.float64)
    r = 1.0 / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)
    return x * r * np.asarray(gamma, np.float64)


def rope(x: np.ndarray, pos: np.ndarray, theta: float) -> np.ndarray:
    """Rotate-half rotary embedding of x [..., H, D] at positions pos [...]:
    (x_d, x_{d+D/2}) -> (x_d cos a - x_{d+D/2} sin a, x_{d+D/2} cos a + x_d sin a),
    a = pos * theta**(-2d/D), d < D/2."""
    x = np.asarray(x, np.float64)
    D = x.shape[-1]
    half = D // 2
    inv_freq = theta ** (-2.0 * np.arange(half, dtype=np.float64) / D)
    ang = np.asarray(pos, np.float64)[..., None, None] * inv_freq       # [..., 1, D/2]
    c, s = np.cos(ang), np.sin(ang)
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def positions(token_keep_b: np.ndarray) -> np.ndarray:
    """Position of every token of one sample in its patch-selected sequence:
    the number of kept tokens before it (text tokens are always kept)."""
    keep = np.asarray(token_keep_b, np.int64)
    return np.cumsum(keep) - keep


def tsm_qk(hidden: np.ndarray, token_keep: np.ndarray, V_full: int, gamma: np.ndarray,
           w_q: np.ndarray, w_k: np.ndarray, Hq: int, Hkv: int, D: int, eps: float,
           theta: float):
    """The scoring queries and keys of the standalone first decoder layer.

    hidden [B, S, Dm], token_keep [B, S] (uint8, 1 = kept), gamma [Dm],
    w_q [Hq*D, Dm], w_k [Hkv*D, Dm]. Returns float64 q [B, T, Hq, D] for the text
    tokens (positions V_full..S-1) and k [B, S, Hkv, D] for every token."""
    B, S, _ = hidden.shape
    xn = rms_norm(hidden, gamma, eps)
    q = np.empty((B, S - V_full, Hq, D))
    k = np.empty((B, S, Hkv, D))
    for b in range(B):
        pos = positions(token_keep[b])
        kb = (xn[b] @ np.asarray(w_k, np.float64).T).reshape(S, Hkv, D)
        qb = (xn[b, V_full:] @ np.asarray(w_q, np.float64).T).reshape(S - V_full, Hq, D)
        k[b] = rope(kb, pos, theta)
        q[b] = rope(qb, pos[V_full:], theta)
    return q, k
