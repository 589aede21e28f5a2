"""Pins of the Patch Selection Module forward pass in the oracle (CPU only):
each encoder layer against torch's float64 TransformerEncoderLayer (pre-norm,
exact GELU) with the same weights, the latent cross-attention and heads against
torch's layer_norm, linear and scaled_dot_product_attention, the whole stack
against the torch composition, closed forms, and planted mistakes."""
import math

import numpy as np
import pytest
import torch

import synth
from oracle import psm as P

D, H, DFF, N, L, T = 32, 4, 64, 6, 2, 9


def params(seed=0, d=D, dff=DFF, n=N, layers=L):
    emb, par = synth.psm_inputs(2, T, d, dff, n, layers, seed)
    return emb.astype(np.float64), par.astype(np.float64)


def torch_layer(Pd, i, d=D, heads=H, dff=DFF):
    lay = torch.nn.TransformerEncoderLayer(d, heads, dff, dropout=0.0, activation="gelu", batch_first=True,
                                           norm_first=True, dtype=torch.float64)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a))  # noqa: E731
    with torch.no_grad():
        lay.self_attn.in_proj_weight.copy_(t(Pd[f"l{i}.w_qkv"]))
        lay.self_attn.in_proj_bias.copy_(t(Pd[f"l{i}.b_qkv"]))
        lay.self_attn.out_proj.weight.copy_(t(Pd[f"l{i}.w_o"]))
        lay.self_attn.out_proj.bias.copy_(t(Pd[f"l{i}.b_o"]))
        lay.linear1.weight.copy_(t(Pd[f"l{i}.w_up"]))
        lay.linear1.bias.copy_(t(Pd[f"l{i}.b_up"]))
        lay.linear2.weight.copy_(t(Pd[f"l{i}.w_down"]))
        lay.linear2.bias.copy_(t(Pd[f"l{i}.b_down"]))
        lay.norm1.weight.copy_(t(Pd[f"l{i}.ln1_g"]))
        lay.norm1.bias.copy_(t(Pd[f"l{i}.ln1_b"]))
        lay.norm2.weight.copy_(t(Pd[f"l{i}.ln2_g"]))
        lay.norm2.bias.copy_(t(Pd[f"l{i}.ln2_b"]))
    return lay.eval()


def torch_cross(h, Pd):
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a))  # noqa: E731
    F = torch.nn.functional
    x = F.layer_norm(t(h), (h.shape[1],), t(Pd["lnf_g"]), t(Pd["lnf_b"]), eps=1e-5)
    q = F.linear(t(Pd["latents"]), t(Pd["w_cq"]), t(Pd["b_cq"]))
    k = F.linear(x, t(Pd["w_ck"]), t(Pd["b_ck"]))
    v = F.linear(x, t(Pd["w_cv"]), t(Pd["b_cv"]))
    z = F.scaled_dot_product_attention(q[None], k[None], v[None])[0]
    return (z * t(Pd["w_head"])).sum(dim=1).numpy() + Pd["b_head"]


def psm_pins(layer=P.encoder_layer, cross=P.cross_logits, forward=P.psm_forward):
    failed = []
    emb, par = params()
    Pd = P.unpack(par, D, DFF, N, L)
    h = emb[0]
    with torch.no_grad():
        want = torch_layer(Pd, 0)(torch.from_numpy(h)[None])[0].numpy()
    if not np.allclose(layer(h, Pd, 0, H), want, rtol=1e-11, atol=1e-12):
        failed.append("layer_torch")
    if not np.allclose(cross(h, Pd), torch_cross(h, Pd), rtol=1e-11, atol=1e-12):
        failed.append("cross_torch")
    with torch.no_grad():
        x = torch.from_numpy(emb)
        for i in range(L):
            x = torch_layer(Pd, i)(x)
    want_all = np.stack([torch_cross(x[b].numpy(), Pd) for b in range(emb.shape[0])])
    if not np.allclose(forward(emb, par, H, DFF, N, L), want_all, rtol=1e-10, atol=1e-11):
        failed.append("stack_torch")
    # closed form: identical latents and zero head biases give one logit value per
    # head weight direction; with all head weights equal every view's logit is equal
    Pz = dict(Pd)
    Pz["latents"] = np.tile(Pd["latents"][:1], (N, 1))
    Pz["w_head"] = np.tile(Pd["w_head"][:1], (N, 1))
    Pz["b_head"] = np.zeros(N)
    lz = cross(h, Pz)
    if not np.allclose(lz, lz[0], rtol=1e-13, atol=1e-14):
        failed.append("equal_views")
    # closed form: a zero query projection gives uniform attention, z = mean of v
    Pu = dict(Pd)
    Pu["w_cq"] = np.zeros_like(Pd["w_cq"])
    Pu["b_cq"] = np.zeros_like(Pd["b_cq"])
    xf = P.layer_norm(h, Pd["lnf_g"], Pd["lnf_b"])
    vmean = (xf @ Pd["w_cv"].T + Pd["b_cv"]).mean(axis=0)
    if not np.allclose(cross(h, Pu), Pd["w_head"] @ vmean + Pd["b_head"], rtol=1e-12, atol=1e-13):
        failed.append("uniform_cross")
    return failed


def test_psm_pins():
    assert psm_pins() == []


def test_layout_size_matches_generator():
    for (d, dff, n, layers) in ((32, 64, 6, 2), (256, 1024, 6, 4)):
        _, par = synth.psm_inputs(1, 3, d, dff, n, layers, 0)
        assert par.size == sum(int(np.prod(s)) for _, s in P.param_layout(d, dff, n, layers))


# ----------------------------------------------------------------------------- planted mistakes

def _layer_post_norm(h, Pd, i, heads):
    y = P.encoder_layer(h, {**Pd, f"l{i}.ln1_g": np.ones_like(Pd[f"l{i}.ln1_g"]),
                            f"l{i}.ln1_b": np.zeros_like(Pd[f"l{i}.ln1_b"])}, i, heads)
    return y


def _layer_tanh_gelu(h, Pd, i, heads):
    saved = P.gelu
    try:
        P.gelu = lambda x: 0.5 * x * (1 + np.tanh(math.sqrt(2 / math.pi) * (x + 0.044715 * x ** 3)))
        return P.encoder_layer(h, Pd, i, heads)
    finally:
        P.gelu = saved


def _layer_one_head(h, Pd, i, heads):
    return P.encoder_layer(h, Pd, i, 1)


def _cross_no_scale(h, Pd):
    d = h.shape[1]
    x = P.layer_norm(h, Pd["lnf_g"], Pd["lnf_b"])
    q = Pd["latents"] @ Pd["w_cq"].T + Pd["b_cq"]
    k = x @ Pd["w_ck"].T + Pd["b_ck"]
    v = x @ Pd["w_cv"].T + Pd["b_cv"]
    return np.sum(P.softmax(q @ k.T) @ v * Pd["w_head"], axis=1) + Pd["b_head"] + 0 * d


def _cross_no_final_norm(h, Pd):
    return P.cross_logits(h, {**Pd, "lnf_g": np.ones_like(Pd["lnf_g"]), "lnf_b": np.zeros_like(Pd["lnf_b"])})


def _fwd_with(layer=None, cross=None):
    def fn(emb, par, heads, dff, n, layers):
        B, T_, d = emb.shape
        Pd = P.unpack(par, d, dff, n, layers)
        out = np.empty((B, n))
        for b in range(B):
            h = emb[b]
            for i in range(layers):
                h = (layer or P.encoder_layer)(h, Pd, i, heads)
            out[b] = (cross or P.cross_logits)(h, Pd)
        return out
    return fn


MUTANTS = {
    "no_first_norm": dict(layer=_layer_post_norm, forward=_fwd_with(layer=_layer_post_norm)),
    "tanh_gelu": dict(layer=_layer_tanh_gelu, forward=_fwd_with(layer=_layer_tanh_gelu)),
    "one_head": dict(layer=_layer_one_head, forward=_fwd_with(layer=_layer_one_head)),
    "cross_no_scale": dict(cross=_cross_no_scale, forward=_fwd_with(cross=_cross_no_scale)),
    "no_final_norm": dict(cross=_cross_no_final_norm, forward=_fwd_with(cross=_cross_no_final_norm)),
}


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_psm_pins_reject_planted_mistakes(name):
    assert psm_pins(**MUTANTS[name]) != []
