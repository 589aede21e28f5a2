"""Seeded synthetic multi-camera workloads.

Shared by the tests, the benchmark and the smoke check. This module only draws
and encodes inputs; it holds none of the method's arithmetic (no patch
selection, no scoring, no top-k, no attention).

The stand-in for the paper's DriveLM / nuScenes multi-camera prompts (Section
"Experiments", Dataset and Training paragraphs): N camera views of T_v visual
tokens each, laid out view-major, followed by T text tokens, one decoder layer's
post-RoPE Q/K/V drawn from N(0,1)/sqrt(D), with a seeded set of "salient"
visual tokens whose keys get a bias beta. Values are returned as the exact
stored bits of the compute dtype:

* ``f32``  -> float32 arrays
* ``bf16`` -> uint16 arrays (the bf16 bit patterns, round-to-nearest-even)
* ``fp8``  -> uint8 arrays (OCP E4M3FN bytes) plus per-tensor float32 scales

Draw order per sample b (each sample has its own PCG64 generator seeded with
``1_000_003*cfg + 1009*run + b``): view mask, salient fraction, salient set,
Q, K, V, key plant. Casts happen after the whole batch is drawn (fp8 scales are
per tensor over the batch).
"""
from __future__ import annotations

import dataclasses
from typing import List, Optional, Sequence

import numpy as np
import torch

F32, BF16, FP8 = "f32", "bf16", "fp8"
E4M3_MAX = 448.0


@dataclasses.dataclass
class Case:
    """One synthetic workload, inputs in their stored encodings."""

    name: str
    B: int
    N: int
    Tv: int
    T: int
    Hq: int
    Hkv: int
    D: int
    dtype: str
    keep_ratio: float
    view_offsets: np.ndarray          # int32 [N+1]; view v owns visual positions [off[v], off[v+1])
    view_logit: np.ndarray            # float32 [B, N]
    view_lexical: Optional[np.ndarray]  # float32 [B, N] or None
    w_lexical: float
    threshold: float
    q: np.ndarray                     # [B, S, Hq, D] stored bits
    k: np.ndarray                     # [B, S, Hkv, D]
    v: np.ndarray                     # [B, S, Hkv, D]
    q_scale: float = 1.0
    k_scale: float = 1.0
    v_scale: float = 1.0
    masked_views: List[np.ndarray] = dataclasses.field(default_factory=list)
    salient: List[np.ndarray] = dataclasses.field(default_factory=list)

    @property
    def V_full(self) -> int:
        return int(self.view_offsets[-1])

    @property
    def S(self) -> int:
        return self.V_full + self.T

    @property
    def G(self) -> int:
        return self.Hq // self.Hkv


def _to_bf16_bits(x: np.ndarray) -> np.ndarray:
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def _to_e4m3(x: np.ndarray):
    """Per-tensor scale amax/448, clamp to +-448, round-to-nearest-even to E4M3FN."""
    amax = float(np.max(np.abs(x))) if x.size else 0.0
    scale = np.float32(amax / E4M3_MAX) if amax > 0 else np.float32(1.0)
    y = np.clip(x / scale, -E4M3_MAX, E4M3_MAX).astype(np.float32)
    t = torch.from_numpy(np.ascontiguousarray(y)).to(torch.float8_e4m3fn)
    return t.view(torch.uint8).numpy().copy(), float(scale)


def encode(x: np.ndarray, dtype: str):
    """Encode a float32 tensor into the stored bits of ``dtype``; returns (bits, scale)."""
    if dtype == F32:
        return np.ascontiguousarray(x, dtype=np.float32), 1.0
    if dtype == BF16:
        return _to_bf16_bits(x), 1.0
    if dtype == FP8:
        return _to_e4m3(x)
    raise ValueError(dtype)


def make_case(*, name: str, B: int, N: int, Tv: int, T: int, Hq: int, Hkv: int, D: int,
              dtype: str, keep_ratio: float, n_masked, salient, beta: float,
              cfg: int, run: int = 0, plant: str = "literal", peaked: bool = False,
              view_sizes: Optional[Sequence[int]] = None,
              w_lexical: float = 0.0, threshold: float = 0.5) -> Case:
    """Draw one seeded batch.

    n_masked: int, or (lo, hi) for a per-sample uniform integer draw in [lo, hi].
    salient:  int (token count), float (fraction of V_full), or (lo, hi) for a
              per-sample uniform fraction draw.
    plant:    "literal" adds beta to every element of the salient keys (all KV
              heads); "aligned" adds beta*sqrt(D)*u_g, u_g the unit vector of the
              sum of KV group g's text queries; "none" plants nothing.
    peaked:   draw Q and K from N(0,1) without the 1/sqrt(D) factor, so that
              attention rows are far from uniform.
    """
    sizes = list(view_sizes) if view_sizes is not None else [Tv] * N
    assert len(sizes) == N
    offsets = np.zeros(N + 1, dtype=np.int32)
    offsets[1:] = np.cumsum(sizes)
    V_full = int(offsets[-1])
    S = V_full + T
    G = Hq // Hkv
    qs = np.empty((B, S, Hq, D), np.float32)
    ks = np.empty((B, S, Hkv, D), np.float32)
    vs = np.empty((B, S, Hkv, D), np.float32)
    logits = np.empty((B, N), np.float32)
    masked_all, salient_all = [], []
    for b in range(B):
        rng = np.random.Generator(np.random.PCG64(1_000_003 * cfg + 1009 * run + b))
        m_b = int(rng.integers(n_masked[0], n_masked[1] + 1)) if isinstance(n_masked, tuple) else int(n_masked)
        masked = np.sort(rng.choice(N, m_b, replace=False)) if m_b else np.zeros(0, np.int64)
        if isinstance(salient, tuple):
            frac = float(rng.uniform(salient[0], salient[1]))
            n_sal = int(round(frac * V_full))
        elif isinstance(salient, float):
            n_sal = int(round(salient * V_full))
        else:
            n_sal = int(salient)
        sal = np.sort(rng.choice(V_full, n_sal, replace=False)) if n_sal else np.zeros(0, np.int64)
        qk_div = 1.0 if peaked else np.sqrt(D)
        qs[b] = rng.standard_normal((S, Hq, D), dtype=np.float32) / np.float32(qk_div)
        ks[b] = rng.standard_normal((S, Hkv, D), dtype=np.float32) / np.float32(qk_div)
        vs[b] = rng.standard_normal((S, Hkv, D), dtype=np.float32) / np.float32(np.sqrt(D))
        if n_sal and plant == "literal":
            ks[b, sal] += np.float32(beta)
        elif n_sal and plant == "aligned":
            for g in range(Hkv):
                qsum = qs[b, V_full:, g * G:(g + 1) * G, :].astype(np.float64).sum(axis=(0, 1))
                u = qsum / max(np.linalg.norm(qsum), 1e-30)
                ks[b, sal, g, :] += (beta * np.sqrt(D) * u).astype(np.float32)
        logits[b] = 8.0
        logits[b, masked] = -8.0
        masked_all.append(masked)
        salient_all.append(sal)
    qb, qsc = encode(qs, dtype)
    kb, ksc = encode(ks, dtype)
    vb, vsc = encode(vs, dtype)
    return Case(name=name, B=B, N=N, Tv=Tv, T=T, Hq=Hq, Hkv=Hkv, D=D, dtype=dtype,
                keep_ratio=float(keep_ratio), view_offsets=offsets, view_logit=logits,
                view_lexical=None, w_lexical=float(w_lexical), threshold=float(threshold),
                q=qb, k=kb, v=vb, q_scale=qsc, k_scale=ksc, v_scale=vsc,
                masked_views=masked_all, salient=salient_all)


# The five workloads: (B, N, Tv, T, Hq, Hkv, D, dtype, keep_ratio, views masked, salient, beta)
CONFIGS = {
    # tiny CPU-checkable case: 2 views x 64 + 16 text, 4 heads, D=64, fp32
    1: dict(B=1, N=2, Tv=64, T=16, Hq=4, Hkv=4, D=64, dtype=F32, keep_ratio=0.5,
            n_masked=0, salient=8, beta=3.0),
    # 6 views x 256 + 64 text, 16 heads, D=128, bf16, 2 views masked
    2: dict(B=1, N=6, Tv=256, T=64, Hq=16, Hkv=16, D=128, dtype=BF16, keep_ratio=0.25,
            n_masked=2, salient=0.05, beta=2.5),
    # 6 views x 1024 + 128 text, GQA 32/8, D=128, bf16
    3: dict(B=1, N=6, Tv=1024, T=128, Hq=32, Hkv=8, D=128, dtype=BF16, keep_ratio=0.5,
            n_masked=0, salient=0.05, beta=2.5),
    # batch 8 ragged of the same shape, 0-4 views masked per sample
    4: dict(B=8, N=6, Tv=1024, T=128, Hq=32, Hkv=8, D=128, dtype=BF16, keep_ratio=0.3,
            n_masked=(0, 4), salient=(0.02, 0.10), beta=2.5),
    # fp8 e4m3 variant of the batch-8 ragged case
    5: dict(B=8, N=6, Tv=1024, T=128, Hq=32, Hkv=8, D=128, dtype=FP8, keep_ratio=0.25,
            n_masked=(0, 4), salient=(0.02, 0.10), beta=2.5),
}
CFG3_KEEP_SWEEP = (1.0, 0.5, 0.25)


def config_case(cfg: int, run: int = 0, **overrides) -> Case:
    """The seeded batch of workload ``cfg`` (1..5); keyword overrides replace fields."""
    params = dict(CONFIGS[cfg])
    params.update(overrides)
    return make_case(name=f"cfg{cfg}", cfg=cfg, run=run, **params)


def random_attention_inputs(seqlens: Sequence[int], Hq: int, Hkv: int, D: int, dtype: str,
                            seed: int, peaked: bool = False):
    """Packed varlen Q/K/V ``[sum(seqlens), H, D]`` stored bits plus cu_seqlens, for
    driving the prefill attention call directly. Returns (q, k, v, scales, cu)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    total = int(sum(seqlens))
    div = np.float32(1.0 if peaked else np.sqrt(D))
    q = rng.standard_normal((total, Hq, D), dtype=np.float32) / div
    k = rng.standard_normal((total, Hkv, D), dtype=np.float32) / div
    v = rng.standard_normal((total, Hkv, D), dtype=np.float32) / np.float32(np.sqrt(D))
    cu = np.zeros(len(seqlens) + 1, np.int32)
    cu[1:] = np.cumsum(seqlens)
    qb, qs = encode(q, dtype)
    kb, ks = encode(k, dtype)
    vb, vsc = encode(v, dtype)
    return qb, kb, vb, (qs, ks, vsc), cu


def encode_with_scale(x: np.ndarray, dtype: str, scale: float) -> np.ndarray:
    """Stored bits of ``x`` under a given per-tensor scale (fp8: clamp x/scale to
    +-448 and round to nearest even; other dtypes ignore the scale, which is 1)."""
    if dtype != FP8:
        return encode(x, dtype)[0]
    y = np.clip(x / np.float32(scale), -E4M3_MAX, E4M3_MAX).astype(np.float32)
    return torch.from_numpy(np.ascontiguousarray(y)).to(torch.float8_e4m3fn).view(torch.uint8).numpy().copy()


def decode_token_inputs(B: int, Hq: int, Hkv: int, D: int, dtype: str, seed: int,
                        scales: Optional[Sequence[float]] = None, peaked: bool = False):
    """The query, key and value of one new token per sample for a decode step
    after the prefill: q1 ``[B,Hq,D]``, k1/v1 ``[B,Hkv,D]`` from the same
    distribution as the prompt (N(0,1)/sqrt(D); Q and K unscaled when peaked).
    For fp8, ``scales`` = (q, k, v) scales of the cache the token joins; without
    them each tensor gets its own amax/448 scale. Returns (q1, k1, v1, scales)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    div = np.float32(1.0 if peaked else np.sqrt(D))
    q = rng.standard_normal((B, Hq, D), dtype=np.float32) / div
    k = rng.standard_normal((B, Hkv, D), dtype=np.float32) / div
    v = rng.standard_normal((B, Hkv, D), dtype=np.float32) / np.float32(np.sqrt(D))
    if scales is None:
        (qb, qs), (kb, ks), (vb, vs) = encode(q, dtype), encode(k, dtype), encode(v, dtype)
        return qb, kb, vb, (qs, ks, vs)
    return (encode_with_scale(q, dtype, scales[0]), encode_with_scale(k, dtype, scales[1]),
            encode_with_scale(v, dtype, scales[2]), tuple(float(s) for s in scales))


def tsm_inputs(B: int, S: int, Dm: int, Hq: int, Hkv: int, D: int, seed: int):
    """Inputs of the Token Selection Module front end: hidden states [B,S,Dm]
    from N(0,1), an RMS gain [Dm] from 1 + 0.1*N(0,1) (fp32), and projection
    weights w_q [Hq*D, Dm], w_k [Hkv*D, Dm] from N(0, 1/Dm), the bf16 ones as
    round-to-nearest-even bits. Returns (hidden, gamma, w_q, w_k)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    hidden = rng.standard_normal((B, S, Dm), dtype=np.float32)
    gamma = (1.0 + 0.1 * rng.standard_normal(Dm)).astype(np.float32)
    w_q = rng.standard_normal((Hq * D, Dm), dtype=np.float32) / np.float32(np.sqrt(Dm))
    w_k = rng.standard_normal((Hkv * D, Dm), dtype=np.float32) / np.float32(np.sqrt(Dm))
    return _to_bf16_bits(hidden), gamma, _to_bf16_bits(w_q), _to_bf16_bits(w_k)


def psm_inputs(B: int, T: int, d: int, d_ff: int, n_views: int, n_layers: int, seed: int):
    """Inputs of the Patch Selection Module forward pass: text token embeddings
    [B, T, d] from N(0,1) and the flat float32 parameter vector in the order the
    C ABI documents (per layer: LN1 gain, bias; QKV weight [3d, d], bias; output
    weight [d, d], bias; LN2 gain, bias; up weight [d_ff, d], bias; down weight
    [d, d_ff], bias; then final LN gain, bias; latents [N, d]; cross Q, K, V
    weights [d, d] with biases; head weights [N, d], biases [N]). Gains are
    1 + 0.1*N(0,1), biases 0.02*N(0,1), weights N(0, 1/fan_in), latents N(0,1).
    Returns (emb float32 [B, T, d], params float32)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    emb = rng.standard_normal((B, T, d), dtype=np.float32)
    segs = []

    def gain(n):
        segs.append(1.0 + 0.1 * rng.standard_normal(n))

    def bias(n):
        segs.append(0.02 * rng.standard_normal(n))

    def weight(rows, fan_in):
        segs.append(rng.standard_normal(rows * fan_in) / np.sqrt(fan_in))

    for _ in range(n_layers):
        gain(d), bias(d), weight(3 * d, d), bias(3 * d), weight(d, d), bias(d)
        gain(d), bias(d), weight(d_ff, d), bias(d_ff), weight(d, d_ff), bias(d)
    gain(d), bias(d)
    segs.append(rng.standard_normal(n_views * d))
    weight(d, d), bias(d), weight(d, d), bias(d), weight(d, d), bias(d)
    weight(n_views, d), bias(n_views)
    return emb, np.concatenate(segs).astype(np.float32)


def with_zero_queries(case: Case) -> Case:
    """A copy of ``case`` whose queries are all zero (stored bits 0 encode +0.0
    in every dtype): every attention row is then uniform over its visible keys."""
    return dataclasses.replace(case, q=np.zeros_like(case.q))


def with_duplicated_keys(case: Case, b: int, members: Sequence[int], beta: float) -> Case:
    """A copy of ``case`` in which the visual tokens ``members`` of sample b share
    one key row (every KV head): the key of members[0] plus beta*sqrt(D)*u_g,
    u_g the unit vector of the sum of KV group g's text queries (the "aligned"
    plant, which lifts the group's attention above the other tokens). The row
    is encoded once and its stored bits copied to every member, so the members'
    keys are bitwise identical."""
    G = case.Hq // case.Hkv
    k = case.k.copy()
    scale = case.k_scale
    if case.dtype == F32:
        qf = case.q[b].astype(np.float64)
        kf = case.k[b, members[0]].astype(np.float64)
    elif case.dtype == BF16:
        qf = (case.q[b].astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
        kf = (case.k[b, members[0]].astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    else:
        tq = torch.from_numpy(np.ascontiguousarray(case.q[b])).view(torch.float8_e4m3fn)
        tk = torch.from_numpy(np.ascontiguousarray(case.k[b, members[0]])).view(torch.float8_e4m3fn)
        qf = tq.to(torch.float64).numpy() * case.q_scale
        kf = tk.to(torch.float64).numpy() * scale
    row = np.empty((case.Hkv, case.D), np.float32)
    for g in range(case.Hkv):
        qsum = qf[case.V_full:, g * G:(g + 1) * G, :].sum(axis=(0, 1))
        u = qsum / max(np.linalg.norm(qsum), 1e-30)
        row[g] = (kf[g] + beta * np.sqrt(case.D) * u).astype(np.float32)
    bits = encode_with_scale(row, case.dtype, scale) if case.dtype == FP8 else encode(row, case.dtype)[0]
    for j in members:
        k[b, j] = bits
    return dataclasses.replace(case, k=k)

