"""Plain float64 definition of the Patch Selection Module forward pass (test
infrastructure only: tests, the smoke check and the benchmark's CPU-baseline
leg use it).

Paper, Design section, Patch Selection Module paragraph: a small transformer
encoder of 4 layers encodes the tokenised text query; a cross-attention relates
the encoded query to N learnable latent queries, one per camera view, and each
view's result is mapped to its own logit (N independent binary decisions). The
logits then enter the fused view score of the patch selection.

Readings (the paper gives no sizes or layer details):
* the token embeddings are the input (tokeniser and embedding table are not
  part of the module's arithmetic);
* encoder layers are pre-norm: h += MHA(LN1(h)); h += W2 GELU(W1 LN2(h) + b1) + b2,
  with biased projections, exact (erf) GELU and LayerNorm epsilon 1e-5;
* the cross-attention is single-headed with the latents as queries over the
  final-normalised encoded tokens: z_v = softmax((l_v Wq + bq)(X Wk + bk)^T /
  sqrt(d)) (X Wv + bv), and logit_v = w_v . z_v + c_v (one linear head per view).

Parameters travel as one float32 vector in the order of ``param_layout``.
"""
from __future__ import annotations

import math

import numpy as np

LN_EPS = 1e-5


def param_layout(d: int, d_ff: int, n_views: int, n_layers: int):
    """[(name, shape)] in storage order: per layer ln1_g, ln1_b, w_qkv [3d, d],
    b_qkv, w_o [d, d], b_o, ln2_g, ln2_b, w_up [d_ff, d], b_up, w_down [d, d_ff],
    b_down; then lnf_g, lnf_b, latents [N, d], w_cq, b_cq, w_ck, b_ck, w_cv, b_cv
    (each [d, d] / [d]), w_head [N, d], b_head [N]."""
    out = []
    for i in range(n_layers):
        out += [(f"l{i}.ln1_g", (d,)), (f"l{i}.ln1_b", (d,)), (f"l{i}.w_qkv", (3 * d, d)),
                (f"l{i}.b_qkv", (3 * d,)), (f"l{i}.w_o", (d, d)), (f"l{i}.b_o", (d,)),
                (f"l{i}.ln2_g", (d,)), (f"l{i}.ln2_b", (d,)), (f"l{i}.w_up", (d_ff, d)),
                (f"l{i}.b_up", (d_ff,)), (f"l{i}.w_down", (d, d_ff)), (f"l{i}.b_down", (d,))]
    out += [("lnf_g", (d,)), ("lnf_b", (d,)), ("latents", (n_views, d)), ("w_cq", (d, d)), ("b_cq", (d,)),
            ("w_ck", (d, d)), ("b_ck", (d,)), ("w_cv", (d, d)), ("b_cv", (d,)), ("w_head", (n_views, d)),
            ("b_head", (n_views,))]
    return out


def unpack(params: np.ndarray, d: int, d_ff: int, n_views: int, n_layers: int) -> dict:
    """Name -> float64 array views of the flat parameter vector."""
    p = np.asarray(params, np.float64)
    out, off = {}, 0
    for name, shape in param_layout(d, d_ff, n_views, n_layers):
        n = int(np.prod(shape))
        out[name] = p[off:off + n].reshape(shape)
        off += n
    assert off == p.size, (off, p.size)
    return out


def layer_norm(x, g, b, eps=LN_EPS):
    x = np.asarray(x, np.float64)
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps) * g + b


def gelu(x):
    """Exact GELU: x * Phi(x), Phi the standard normal CDF."""
    erf = np.vectorize(math.erf)
    return 0.5 * x * (1.0 + erf(x / math.sqrt(2.0)))


def softmax(x, axis=-1):
    e = np.exp(x - x.max(axis=axis, keepdims=True))
    return e / e.sum(axis=axis, keepdims=True)


def encoder_layer(h, P, i, n_heads):
    """One pre-norm layer on h [T, d] (float64)."""
    T, d = h.shape
    dh = d // n_heads
    x = layer_norm(h, P[f"l{i}.ln1_g"], P[f"l{i}.ln1_b"])
    qkv = x @ P[f"l{i}.w_qkv"].T + P[f"l{i}.b_qkv"]
    q, k, v = qkv[:, :d], qkv[:, d:2 * d], qkv[:, 2 * d:]
    heads = []
    for hh in range(n_heads):
        s = slice(hh * dh, (hh + 1) * dh)
        a = softmax(q[:, s] @ k[:, s].T / math.sqrt(dh))
        heads.append(a @ v[:, s])
    h = h + np.concatenate(heads, axis=1) @ P[f"l{i}.w_o"].T + P[f"l{i}.b_o"]
    x = layer_norm(h, P[f"l{i}.ln2_g"], P[f"l{i}.ln2_b"])
    f = gelu(x @ P[f"l{i}.w_up"].T + P[f"l{i}.b_up"])
    return h + f @ P[f"l{i}.w_down"].T + P[f"l{i}.b_down"]


def cross_logits(h, P):
    """Per-view logits from the encoded tokens h [T, d]."""
    d = h.shape[1]
    x = layer_norm(h, P["lnf_g"], P["lnf_b"])
    q = P["latents"] @ P["w_cq"].T + P["b_cq"]          # [N, d]
    k = x @ P["w_ck"].T + P["b_ck"]                      # [T, d]
    v = x @ P["w_cv"].T + P["b_cv"]
    z = softmax(q @ k.T / math.sqrt(d)) @ v              # [N, d]
    return np.sum(z * P["w_head"], axis=1) + P["b_head"]


def psm_forward(emb: np.ndarray, params: np.ndarray, n_heads: int, d_ff: int, n_views: int,
                n_layers: int) -> np.ndarray:
    """View logits [B, N] from token embeddings emb [B, T, d]."""
    B, T, d = emb.shape
    P = unpack(params, d, d_ff, n_views, n_layers)
    out = np.empty((B, n_views))
    for b in range(B):
        h = np.asarray(emb[b], np.float64)
        for i in range(n_layers):
            h = encoder_layer(h, P, i, n_heads)
        out[b] = cross_logits(h, P)
    return out
