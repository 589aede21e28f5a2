"""Pins of the Token Selection Module front end in the oracle (CPU only):
RMS normalisation against torch's float64 rms_norm and closed forms, the
rotary embedding against a complex-number rotation built from torch's polar
form (a different pairing layout, mapped by a permutation), its relative
position property and a hand-worked example, the position rule against
explicit counting, and planted mistakes that at least one pin must reject."""
import math

import numpy as np
import pytest
import torch

from oracle import tsm as T


def rope_complex_torch(x, pos, theta):
    """Rotary embedding by complex multiplication in torch: elements d and
    d + D/2 become one complex number (d < D/2), multiplied by
    exp(i * pos * theta**(-2d/D)) built with torch.polar."""
    x = torch.from_numpy(np.asarray(x, np.float64))
    D = x.shape[-1]
    half = D // 2
    z = torch.complex(x[..., :half], x[..., half:])
    inv = torch.pow(torch.tensor(float(theta), dtype=torch.float64),
                    -2.0 * torch.arange(half, dtype=torch.float64) / D)
    ang = torch.from_numpy(np.asarray(pos, np.float64))[..., None, None] * inv
    rot = torch.polar(torch.ones_like(ang), ang)
    w = z * rot
    return torch.cat([w.real, w.imag], dim=-1).numpy()


def reference_qk(hidden, keep, V_full, gamma, w_q, w_k, Hq, Hkv, D, eps, theta):
    """The front end from torch library calls: F.rms_norm, F.linear and the
    complex rotation above, positions by explicit counting."""
    B, S, Dm = hidden.shape
    x = torch.from_numpy(hidden)
    xn = torch.nn.functional.rms_norm(x, (Dm,), weight=torch.from_numpy(gamma), eps=eps)
    k = torch.nn.functional.linear(xn, torch.from_numpy(w_k)).numpy().reshape(B, S, Hkv, D)
    q = torch.nn.functional.linear(xn[:, V_full:], torch.from_numpy(w_q)).numpy().reshape(B, S - V_full, Hq, D)
    qo, ko = np.empty_like(q), np.empty_like(k)
    for b in range(B):
        pos, n = np.zeros(S), 0
        for j in range(S):
            pos[j] = n
            n += int(keep[b, j])
        ko[b] = rope_complex_torch(k[b], pos, theta)
        qo[b] = rope_complex_torch(q[b], pos[V_full:], theta)
    return qo, ko


def case(seed=0, B=2, N=3, Tv=5, T_=4, Dm=16, Hq=4, Hkv=2, D=8, drop=True):
    rng = np.random.default_rng(seed)
    V_full = N * Tv
    S = V_full + T_
    hidden = rng.standard_normal((B, S, Dm)) * 2.0
    gamma = 1.0 + 0.3 * rng.standard_normal(Dm)
    w_q = rng.standard_normal((Hq * D, Dm)) / math.sqrt(Dm)
    w_k = rng.standard_normal((Hkv * D, Dm)) / math.sqrt(Dm)
    keep = np.ones((B, S), np.uint8)
    if drop:
        keep[0, Tv:2 * Tv] = 0        # sample 0 drops its second view
    return dict(hidden=hidden, keep=keep, V_full=V_full, gamma=gamma, w_q=w_q, w_k=w_k, Hq=Hq, Hkv=Hkv,
                D=D, eps=1e-3, theta=10000.0)


def tsm_pins(fn_qk=T.tsm_qk, fn_rope=T.rope, fn_rms=T.rms_norm, fn_pos=T.positions):
    """Names of the pins that fail for the given implementations."""
    failed = []
    rng = np.random.default_rng(7)
    # RMS normalisation: torch float64 rms_norm, and the constant-row closed form
    x = rng.standard_normal((3, 5, 16)) * 3
    g = 1 + 0.5 * rng.standard_normal(16)
    want = torch.nn.functional.rms_norm(torch.from_numpy(x), (16,), weight=torch.from_numpy(g), eps=0.25).numpy()
    if not np.allclose(fn_rms(x, g, 0.25), want, rtol=1e-13, atol=1e-14):
        failed.append("rms_torch")
    c = np.full((1, 16), -1.5)
    if not np.allclose(fn_rms(c, g, 0.25), -1.5 / math.sqrt(2.25 + 0.25) * g, rtol=1e-14):
        failed.append("rms_constant")
    # rotary embedding: complex rotation, position 0, relative positions, worked example
    xr = rng.standard_normal((6, 3, 8))
    pos = np.array([0, 1, 5, 17, 400, 6271])
    if not np.allclose(fn_rope(xr, pos, 10000.0), rope_complex_torch(xr, pos, 10000.0), rtol=1e-12, atol=1e-12):
        failed.append("rope_complex")
    if not np.array_equal(fn_rope(xr[:1], np.zeros(1), 10000.0), xr[:1]):
        failed.append("rope_pos0")
    qv, kv = rng.standard_normal((1, 1, 8)), rng.standard_normal((1, 1, 8))
    for m, n in ((7, 3), (100, 96), (4, 0)):
        lhs = np.sum(fn_rope(qv, np.array([m]), 10000.0) * fn_rope(kv, np.array([n]), 10000.0))
        rhs = np.sum(fn_rope(qv, np.array([m - n]), 10000.0) * kv)
        if not math.isclose(lhs, rhs, rel_tol=1e-12, abs_tol=1e-12):
            failed.append("rope_relative")
            break
    # D = 4, theta = 100: frequencies 1 and 1/10; x = (1, 2, 3, 4) at position 2
    ex = fn_rope(np.array([[[1.0, 2.0, 3.0, 4.0]]]), np.array([2.0]), 100.0)[0, 0]
    a0, a1 = 2.0, 0.2
    hand = [1 * math.cos(a0) - 3 * math.sin(a0), 2 * math.cos(a1) - 4 * math.sin(a1),
            3 * math.cos(a0) + 1 * math.sin(a0), 4 * math.cos(a1) + 2 * math.sin(a1)]
    if not np.allclose(ex, hand, rtol=1e-14, atol=1e-15):
        failed.append("rope_hand")
    # positions: explicit counting
    keep = np.array([1, 1, 0, 0, 1, 0, 1, 1], np.uint8)
    if not np.array_equal(fn_pos(keep), [0, 1, 2, 2, 2, 3, 3, 4]):
        failed.append("positions")
    # the whole front end against torch library calls
    cs = case()
    q, k = fn_qk(cs["hidden"], cs["keep"], cs["V_full"], cs["gamma"], cs["w_q"], cs["w_k"], cs["Hq"],
                 cs["Hkv"], cs["D"], cs["eps"], cs["theta"])
    qr, kr = reference_qk(cs["hidden"], cs["keep"], cs["V_full"], cs["gamma"], cs["w_q"], cs["w_k"], cs["Hq"],
                          cs["Hkv"], cs["D"], cs["eps"], cs["theta"])
    if not (np.allclose(q, qr, rtol=1e-12, atol=1e-12) and np.allclose(k, kr, rtol=1e-12, atol=1e-12)):
        failed.append("front_end_torch")
    return failed


def test_tsm_pins():
    assert tsm_pins() == []


def test_gain_folds_into_the_projection():
    """gamma applied to x equals gamma folded into the weight columns (exact in
    real arithmetic; float64 here): the form the GPU path consumes."""
    cs = case(seed=3)
    q1, k1 = T.tsm_qk(cs["hidden"], cs["keep"], cs["V_full"], cs["gamma"], cs["w_q"], cs["w_k"], cs["Hq"],
                      cs["Hkv"], cs["D"], cs["eps"], cs["theta"])
    ones = np.ones_like(cs["gamma"])
    q2, k2 = T.tsm_qk(cs["hidden"], cs["keep"], cs["V_full"], ones, cs["w_q"] * cs["gamma"],
                      cs["w_k"] * cs["gamma"], cs["Hq"], cs["Hkv"], cs["D"], cs["eps"], cs["theta"])
    assert np.allclose(q1, q2, rtol=1e-12, atol=1e-13) and np.allclose(k1, k2, rtol=1e-12, atol=1e-13)


def test_dropped_view_shifts_text_positions():
    """A dropped view removes its tokens from the sequence: the text queries of
    sample 0 (second view dropped) equal those of a sequence built without the
    view's tokens."""
    cs = case(seed=5)
    q, k = T.tsm_qk(cs["hidden"], cs["keep"], cs["V_full"], cs["gamma"], cs["w_q"], cs["w_k"], cs["Hq"],
                    cs["Hkv"], cs["D"], cs["eps"], cs["theta"])
    keep0 = cs["keep"][0].astype(bool)
    h = cs["hidden"][0:1, keep0]
    V_kept = int(keep0[:cs["V_full"]].sum())
    q2, k2 = T.tsm_qk(h, np.ones(h.shape[:2], np.uint8), V_kept, cs["gamma"], cs["w_q"], cs["w_k"], cs["Hq"],
                      cs["Hkv"], cs["D"], cs["eps"], cs["theta"])
    assert np.allclose(q[0], q2[0], rtol=1e-12, atol=1e-13)
    assert np.allclose(k[0][keep0], k2[0], rtol=1e-12, atol=1e-13)


# ----------------------------------------------------------------------------- planted mistakes

def _rope_interleaved(x, pos, theta):
    x = np.asarray(x, np.float64)
    D = x.shape[-1]
    inv = theta ** (-2.0 * np.arange(D // 2) / D)
    a = np.asarray(pos, np.float64)[..., None, None] * inv
    out = x.copy()
    out[..., 0::2] = x[..., 0::2] * np.cos(a) - x[..., 1::2] * np.sin(a)
    out[..., 1::2] = x[..., 1::2] * np.cos(a) + x[..., 0::2] * np.sin(a)
    return out


def _rope_sign(x, pos, theta):
    return T.rope(x, -np.asarray(pos, np.float64), theta)


def _rope_freq(x, pos, theta):
    x = np.asarray(x, np.float64)
    D = x.shape[-1]
    half = D // 2
    inv = theta ** (-1.0 * np.arange(half) / D)
    a = np.asarray(pos, np.float64)[..., None, None] * inv
    x1, x2 = x[..., :half], x[..., half:]
    return np.concatenate([x1 * np.cos(a) - x2 * np.sin(a), x2 * np.cos(a) + x1 * np.sin(a)], -1)


def _rms_no_gamma(x, g, eps):
    return T.rms_norm(x, np.ones_like(g), eps)


def _rms_no_eps(x, g, eps):
    return T.rms_norm(x, g, 0.0)


def _pos_no_skip(keep):
    return np.arange(len(keep))


def _qk_with(**kw):
    def fn(hidden, token_keep, V_full, gamma, w_q, w_k, Hq, Hkv, D, eps, theta):
        rope_f = kw.get("rope", T.rope)
        rms_f = kw.get("rms", T.rms_norm)
        pos_f = kw.get("pos", T.positions)
        B, S, _ = hidden.shape
        xn = rms_f(hidden, gamma, eps)
        q = np.empty((B, S - V_full, Hq, D))
        k = np.empty((B, S, Hkv, D))
        for b in range(B):
            p = pos_f(token_keep[b])
            k[b] = rope_f((xn[b] @ w_k.T).reshape(S, Hkv, D), p, theta)
            q[b] = rope_f((xn[b, V_full:] @ w_q.T).reshape(S - V_full, Hq, D), p[V_full:], theta)
        return q, k
    return fn


MUTANTS = {
    "rope_interleaved": dict(fn_rope=_rope_interleaved, fn_qk=_qk_with(rope=_rope_interleaved)),
    "rope_sign": dict(fn_rope=_rope_sign, fn_qk=_qk_with(rope=_rope_sign)),
    "rope_freq": dict(fn_rope=_rope_freq, fn_qk=_qk_with(rope=_rope_freq)),
    "rms_no_gamma": dict(fn_rms=_rms_no_gamma, fn_qk=_qk_with(rms=_rms_no_gamma)),
    "rms_no_eps": dict(fn_rms=_rms_no_eps, fn_qk=_qk_with(rms=_rms_no_eps)),
    "pos_no_skip": dict(fn_pos=_pos_no_skip, fn_qk=_qk_with(pos=_pos_no_skip)),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_tsm_pins_reject_planted_mistakes(name):
    assert tsm_pins(**MUTANTS[name]) != []
