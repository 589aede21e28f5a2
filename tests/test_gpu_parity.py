"""GPU parity: the HIP path, called through the C ABI, against the CPU oracle.

Inputs come from the seeded generator only; expected values come from the
oracle only. Selection follows the near-tie band rule; index lists, lengths
and gathered rows are bit-exact; attention is held to the per-precision
tolerances in parity_util.
"""
import dataclasses
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2506_07416_amd as lv
import synth
from parity_util import (bits_of, check_attention, check_selection, check_view_keep, log,
                         score_rel_err, to_device, to_float64)

pytestmark = pytest.mark.gpu

SCORE_RTOL = 1e-5   # diagnostic bound on fp32 score error; selection uses the band rule


def attn_kind(dtype):
    return {"f32": "f32", "bf16": "bf16", "fp8": "fp8"}[dtype]


def run_select(case, keep_ratio=None, gather=True, query_rows=None):
    """patch_select + token_score_topk on the GPU (the rows variant when
    query_rows is given). Returns host copies."""
    r = case.keep_ratio if keep_ratio is None else keep_ratio
    q, k, v = (to_device(x, case.dtype) for x in (case.q, case.k, case.v))
    logit = torch.from_numpy(case.view_logit).cuda()
    view_keep, token_keep, n_vis = lv.patch_select(logit, case.view_offsets, case.S,
                                                   case.w_lexical, case.threshold)
    out = lv.token_score_topk(q, k, v, token_keep, r, case.V_full, q_scale=case.q_scale,
                              k_scale=case.k_scale, v_scale=case.v_scale, gather=gather,
                              query_rows=query_rows)
    torch.cuda.synchronize()
    cu = out["cu_seqlens"].cpu().numpy()
    res = dict(view_keep=view_keep.cpu().numpy(), token_keep=token_keep.cpu().numpy(),
               n_vis=n_vis.cpu().numpy(), scores=out["scores"].cpu().numpy().astype(np.float64),
               cu=cu, kept_index=out["kept_index"][:cu[-1]].cpu().numpy(), dev=out,
               q=q, k=k, v=v)
    return res


def check_select(case, g, ref, label, exact=False):
    """Selection-stage parity; returns True when every sample's kept set equals
    the oracle's. exact: the kept indices must equal the oracle's bit for bit
    (cases whose exact ties the lower-position rule decides)."""
    vs = oracle.view_scores(case.view_logit, case.view_lexical, case.w_lexical)
    check_view_keep(vs, case.threshold, g["view_keep"])
    # the workloads' view logits lie far from the threshold: the masks are the oracle's
    assert np.array_equal(g["view_keep"], ref["view_keep"]), label
    assert np.array_equal(g["token_keep"], ref["token_keep"]), label
    assert np.array_equal(g["n_vis"], ref["V_b"]), label
    err = score_rel_err(ref["scores"], g["scores"])
    assert err <= SCORE_RTOL, f"{label}: score rel err {err:.3g}"
    assert np.array_equal(g["cu"], ref["cu_seqlens"]), f"{label}: cu_seqlens {g['cu']} vs {ref['cu_seqlens']}"
    identical, bands = True, []
    for b in range(case.B):
        seg = g["kept_index"][g["cu"][b]:g["cu"][b + 1]]
        k_b = int(ref["k_b"][b])
        assert np.array_equal(seg[k_b:], np.arange(case.V_full, case.S)), f"{label}: text tail"
        same, band = check_selection(ref["scores"][b], ref["token_keep"][b], case.V_full, k_b, seg[:k_b])
        identical &= same
        bands.append(band)
    # gathered rows are exact copies of the input rows at the GPU's indices
    for name, src in (("qc", case.q), ("kc", case.k), ("vc", case.v)):
        got = bits_of(g["dev"][name][:g["cu"][-1]])
        want = np.concatenate([src[b, g["kept_index"][g["cu"][b]:g["cu"][b + 1]]] for b in range(case.B)])
        assert np.array_equal(got.reshape(want.shape).view(want.dtype), want), f"{label}: {name} bits"
    if exact:
        assert np.array_equal(g["kept_index"], ref["kept_index"]), f"{label}: kept_index differs"
        identical = True
    log(f"{label}: score rel err {err:.2e}, band sizes {bands}, identical sets {identical}")
    return identical


def attention_on(case, qc, kc, vc, cu, max_len):
    o = lv.prefill_attn(qc, kc, vc, torch.from_numpy(cu).cuda() if isinstance(cu, np.ndarray) else cu,
                        max_len, B=case.B, q_scale=case.q_scale, k_scale=case.k_scale,
                        v_scale=case.v_scale)
    torch.cuda.synchronize()
    return o


# ----------------------------------------------------------------------------- patch select

@pytest.mark.parametrize("cfg", [1, 2, 4])
def test_patch_select_matches_oracle(cfg):
    case = synth.config_case(cfg, Tv=8, T=4, Hq=4, Hkv=2 if cfg > 2 else 4, D=64, dtype="f32")
    log(f"patch_select cfg{cfg}: B={case.B} N={case.N}")
    g = run_select(case, gather=False)
    vs = oracle.view_scores(case.view_logit, None, case.w_lexical)
    check_view_keep(vs, case.threshold, g["view_keep"])
    view_keep = oracle.patch_select(case.view_logit, None, case.w_lexical, case.threshold)
    assert np.array_equal(g["view_keep"], view_keep)
    assert np.array_equal(g["token_keep"], oracle.token_keep_from_views(view_keep, case.view_offsets, case.S))


def test_patch_select_random_logits_lexical_fallback():
    rng = np.random.default_rng(11)
    B, N, S = 16, 6, 64
    off = np.array([0, 5, 9, 20, 21, 40, 50], np.int32)
    logit = rng.normal(0, 2, (B, N)).astype(np.float32)
    lex = rng.random((B, N)).astype(np.float32)
    logit[3] = -20.0                     # nothing passes: fallback
    for w, tau in ((0.0, 0.5), (0.3, 0.6), (1.0, 0.7), (0.5, 0.999)):
        vk, tk, nv = lv.patch_select(torch.from_numpy(logit).cuda(), off, S, w, tau,
                                     view_lexical=torch.from_numpy(lex).cuda())
        torch.cuda.synchronize()
        got = vk.cpu().numpy()
        check_view_keep(oracle.view_scores(logit, lex, w), tau, got)
        # the token mask and counts follow the GPU's own view mask exactly
        assert np.array_equal(tk.cpu().numpy(), oracle.token_keep_from_views(got, off, S))
        assert np.array_equal(nv.cpu().numpy(), oracle.token_keep_from_views(got, off, S)[:, :50].sum(1))
        assert np.array_equal(got, oracle.patch_select(logit, lex, w, tau)), (w, tau)


def test_patch_select_near_threshold():
    """Fused scores within a few ulps of the threshold: views in the 1e-6 band
    may fall either way, every other view and the fallback are exact."""
    rng = np.random.default_rng(12)
    B, N, S = 64, 6, 70
    off = np.array([0, 10, 20, 30, 40, 50, 60], np.int32)
    tau = 0.62
    x0 = math.log(tau / (1 - tau))                 # sigmoid(x0) = tau
    logit = (x0 + rng.integers(-4, 5, (B, N)) * 2e-7 * rng.random((B, N))).astype(np.float32)
    logit[::7] -= 3.0                              # rows where nothing passes: the fallback
    lex = rng.random((B, N)).astype(np.float32)
    total_band = 0
    for w in (0.0, 1e-3):
        vk, tk, nv = lv.patch_select(torch.from_numpy(logit).cuda(), off, S, w, tau,
                                     view_lexical=torch.from_numpy(lex).cuda())
        torch.cuda.synchronize()
        got = vk.cpu().numpy()
        n_band = check_view_keep(oracle.view_scores(logit, lex, w), tau, got)
        assert np.array_equal(tk.cpu().numpy(), oracle.token_keep_from_views(got, off, S))
        assert np.array_equal(nv.cpu().numpy(), oracle.token_keep_from_views(got, off, S)[:, :60].sum(1))
        log(f"near-threshold w={w}: {n_band} of {B * N} views inside the band")
        total_band += n_band
    assert total_band > 0


# ----------------------------------------------------------------------------- attention

ATTN_CASES = [
    # (seqlens, Hq, Hkv, D, dtype, causal, peaked, out_dtype)
    ([80], 4, 4, 64, "f32", True, False, "f32"),
    ([1, 2, 63, 64, 65], 4, 4, 64, "f32", True, True, "f32"),
    ([200, 0, 37], 4, 2, 128, "f32", False, True, "f32"),
    ([320], 16, 16, 128, "bf16", True, False, "bf16"),
    ([1, 127, 128, 129, 300, 0, 257], 8, 2, 128, "bf16", True, True, "bf16"),
    ([500, 3], 8, 1, 128, "bf16", True, True, "f32"),
    ([190, 64], 4, 4, 64, "bf16", True, True, "bf16"),
    ([333], 8, 8, 64, "bf16", False, True, "f32"),
    ([700, 130], 32, 8, 128, "bf16", False, False, "bf16"),
    ([1, 127, 128, 129, 300, 0, 257], 8, 2, 128, "fp8", True, True, "bf16"),
    ([700], 32, 8, 128, "fp8", True, False, "bf16"),
    ([190, 64, 5], 4, 4, 64, "fp8", True, True, "f32"),
    ([333, 64], 8, 4, 128, "fp8", False, True, "f32"),
]


@pytest.mark.parametrize("case_id", range(len(ATTN_CASES)))
def test_attention_matches_oracle(case_id):
    lens, Hq, Hkv, D, dtype, causal, peaked, out_dt = ATTN_CASES[case_id]
    log(f"attention case {case_id}: lens={lens} Hq={Hq} Hkv={Hkv} D={D} {dtype} causal={causal} peaked={peaked}")
    qb, kb, vb, scales, cu = synth.random_attention_inputs(lens, Hq, Hkv, D, dtype, seed=100 + case_id,
                                                           peaked=peaked)
    q, k, v = (to_device(x, dtype) for x in (qb, kb, vb))
    o = lv.prefill_attn(q, k, v, torch.from_numpy(cu).cuda(), max(lens), causal=causal,
                        q_scale=scales[0], k_scale=scales[1], v_scale=scales[2],
                        out_dtype=torch.float32 if out_dt == "f32" else torch.bfloat16)
    torch.cuda.synchronize()
    q64, k64, v64 = (oracle.litevlm.decode_stored(x, dtype, s) for x, s in zip((qb, kb, vb), scales))
    ref = oracle.prefill_attention(q64, k64, v64, cu, Hq, Hkv, 1 / math.sqrt(D), causal=causal)
    stats = check_attention(to_float64(o), ref, attn_kind(dtype), f"case {case_id}")
    log(f"  {stats}")


# ----------------------------------------------------------------------------- selection chain

SELECT_CASES = [
    ("cfg1", dict(cfg=1)),
    ("cfg1-aligned", dict(cfg=1, run=2, plant="aligned")),
    ("cfg2", dict(cfg=2)),
    ("cfg2-peaked", dict(cfg=2, run=1, peaked=True)),
    ("ragged-gqa", dict(cfg=4, Tv=100, T=37, keep_ratio=0.37)),
    ("ragged-gqa-peaked", dict(cfg=4, run=1, Tv=96, T=20, peaked=True, keep_ratio=0.5)),
    ("d64-tail", dict(cfg=2, Tv=50, T=3, Hq=6, Hkv=3, D=64, keep_ratio=0.9)),
    ("fp8-small", dict(cfg=5, Tv=128, T=32)),
    ("k-zero", dict(cfg=2, Tv=16, T=8, keep_ratio=0.01)),
    ("full-keep", dict(cfg=2, Tv=64, T=16, keep_ratio=1.0, n_masked=0)),
    # wide token rows: every gather width (16-byte pieces per thread 4, 5, 9, 32)
    ("gather-w4", dict(cfg=2, Tv=32, T=8, Hq=40, Hkv=8, D=128)),
    ("gather-w5", dict(cfg=2, Tv=32, T=8, Hq=48, Hkv=12, D=128)),
    ("gather-w9", dict(cfg=2, Tv=32, T=8, Hq=48, Hkv=48, D=128)),
    ("gather-w32-f32", dict(cfg=1, Tv=40, T=6, Hq=128, Hkv=64, D=128)),
    # the largest inputs the calls take: LITEVLM_MAX_VISUAL visual tokens (8
    # views of 2048), and LITEVLM_MAX_BATCH samples
    ("max-visual", dict(cfg=2, N=8, Tv=2048, T=16, Hq=8, Hkv=2, D=64, keep_ratio=0.25)),
    ("max-batch", dict(cfg=4, B=256, N=2, Tv=16, T=4, Hq=2, Hkv=1, D=64, n_masked=(0, 1),
                       salient=(0.1, 0.3), keep_ratio=0.5)),
]


@pytest.mark.parametrize("name", [c[0] for c in SELECT_CASES])
def test_select_chain_matches_oracle(name):
    kw = dict(dict(SELECT_CASES)[name])
    cfg = kw.pop("cfg")
    case = synth.config_case(cfg, **kw)
    log(f"select {name}: B={case.B} S={case.S} V={case.V_full} Hq={case.Hq} Hkv={case.Hkv} D={case.D} {case.dtype} r={case.keep_ratio}")
    g = run_select(case)
    ref = oracle.run_path(case, attention=False)
    identical = check_select(case, g, ref, name)
    # attention over the compacted sequence
    cu = g["cu"]
    max_len = int(np.max(np.diff(cu)))
    o = attention_on(case, g["dev"]["qc"], g["dev"]["kc"], g["dev"]["vc"], g["dev"]["cu_seqlens"], max_len)
    if identical:
        ref_o = oracle.run_path(case)["o"]
        stats = check_attention(to_float64(o[:cu[-1]]), ref_o, attn_kind(case.dtype), name)
    else:
        # near-tie sets differ: attention is checked on the oracle's own compacted inputs
        qc = to_device(ref["qc_bits"], case.dtype)
        kc = to_device(ref["kc_bits"], case.dtype)
        vc = to_device(ref["vc_bits"], case.dtype)
        o2 = attention_on(case, qc, kc, vc, ref["cu_seqlens"], max_len)
        ref_o = oracle.run_path(case)["o"]
        stats = check_attention(to_float64(o2), ref_o, attn_kind(case.dtype), name)
    log(f"  attention {stats}")


# ----------------------------------------------------------------------------- in-call patch selection

def run_fused(case, keep_ratio=None, logit=None, lexical=None, w=None, tau=None):
    """litevlm_select_score_topk on the GPU; host copies in run_select's layout."""
    r = case.keep_ratio if keep_ratio is None else keep_ratio
    q, k, v = (to_device(x, case.dtype) for x in (case.q, case.k, case.v))
    lg = torch.from_numpy(case.view_logit if logit is None else logit).cuda()
    lx = None if lexical is None else torch.from_numpy(lexical).cuda()
    out = lv.select_score_topk(lg, case.view_offsets, q, k, v, r, case.V_full,
                               w_lexical=case.w_lexical if w is None else w,
                               threshold=case.threshold if tau is None else tau, view_lexical=lx,
                               q_scale=case.q_scale, k_scale=case.k_scale, v_scale=case.v_scale)
    torch.cuda.synchronize()
    cu = out["cu_seqlens"].cpu().numpy()
    return dict(view_keep=out["view_keep"].cpu().numpy(), token_keep=out["token_keep"].cpu().numpy(),
                n_vis=out["n_visual_kept"].cpu().numpy(), scores=out["scores"].cpu().numpy().astype(np.float64),
                cu=cu, kept_index=out["kept_index"][:cu[-1]].cpu().numpy(), dev=out)


def run_two_calls(case, keep_ratio, logit, lexical, w, tau):
    """patch_select then token_score_topk with explicit selection inputs."""
    q, k, v = (to_device(x, case.dtype) for x in (case.q, case.k, case.v))
    vk, tk, nv = lv.patch_select(torch.from_numpy(logit).cuda(), case.view_offsets, case.S, w, tau,
                                 view_lexical=None if lexical is None else torch.from_numpy(lexical).cuda())
    out = lv.token_score_topk(q, k, v, tk, keep_ratio, case.V_full, q_scale=case.q_scale,
                              k_scale=case.k_scale, v_scale=case.v_scale)
    torch.cuda.synchronize()
    cu = out["cu_seqlens"].cpu().numpy()
    return dict(view_keep=vk.cpu().numpy(), token_keep=tk.cpu().numpy(), n_vis=nv.cpu().numpy(),
                scores=out["scores"].cpu().numpy().astype(np.float64), cu=cu,
                kept_index=out["kept_index"][:cu[-1]].cpu().numpy(), dev=out)


def balanced_split(case):
    """True where the in-call selection splits sweep 1's key tiles unevenly
    over the samples (their live tiles follow the view masks), so that its
    row partials, and the scores' last bits, differ from the two-call path's:
    more than one sample, at most 16, at least two key splits per (sample, KV
    group, row block), at most 256 key tiles of 64."""
    R = (case.Hq // case.Hkv) * (case.S - case.V_full)
    n_rb = -(-R // 512)
    n_kt = -(-case.S // 64)
    ns1 = max(-(-n_kt // 64), min(n_kt, max(1, 256 // (case.B * case.Hkv * n_rb))))
    return 1 < case.B <= 16 and ns1 >= 2 and n_kt <= 256


def assert_same_select(a, b, label, case, exact=True):
    """Two selection runs (a: the in-call selection, b: the two calls) agree.
    exact: every output bit for bit (the packed rows up to cu[B]). Otherwise
    the view decision, the lengths and the text tails bit for bit, the scores
    within SCORE_RTOL of each other, a's kept set by the band rule around b's
    scores, and a's packed rows exact copies of the inputs at a's indices."""
    for key in ("view_keep", "token_keep", "n_vis", "cu"):
        assert np.array_equal(a[key], b[key]), f"{label}: {key}"
    if exact:
        assert np.array_equal(a["kept_index"], b["kept_index"]), f"{label}: kept_index"
        assert np.array_equal(a["scores"].astype(np.float32).view(np.uint32),
                              b["scores"].astype(np.float32).view(np.uint32)), f"{label}: scores"
        rows = int(a["cu"][-1])
        for name in ("qc", "kc", "vc"):
            assert torch.equal(bits_of_t(a["dev"][name][:rows]), bits_of_t(b["dev"][name][:rows])), f"{label}: {name}"
        return
    err = score_rel_err(b["scores"], a["scores"])
    assert err <= SCORE_RTOL, f"{label}: in-call vs two-call score rel err {err:.3g}"
    same = 0
    for bb in range(case.B):
        seg = a["kept_index"][a["cu"][bb]:a["cu"][bb + 1]]
        k_b = seg.shape[0] - (case.S - case.V_full)
        assert np.array_equal(seg[k_b:], np.arange(case.V_full, case.S)), f"{label}: text tail"
        ok, _ = check_selection(b["scores"][bb], b["token_keep"][bb], case.V_full, k_b, seg[:k_b])
        same += int(ok)
    for name, src in (("qc", case.q), ("kc", case.k), ("vc", case.v)):
        got = bits_of(a["dev"][name][:a["cu"][-1]])
        want = np.concatenate([src[bb, a["kept_index"][a["cu"][bb]:a["cu"][bb + 1]]] for bb in range(case.B)])
        assert np.array_equal(got.reshape(want.shape).view(want.dtype), want), f"{label}: {name} bits"
    log(f"{label}: balanced split, scores within {err:.2e} of the two calls, "
        f"{same} of {case.B} kept sets identical")


def bits_of_t(t):
    return t.contiguous().view(torch.uint8)


@pytest.mark.parametrize("cfg,r", [(2, None), (3, 0.5), (3, 0.25), (4, None), (5, None), (1, None)])
def test_fused_select_equals_two_calls(cfg, r):
    """The in-call selection gives the two-call path's results bit for bit, at
    the workload shapes (cfg3-5 full size, cfg4 with masked views, fp8, fp32),
    and the oracle's selection."""
    case = synth.config_case(cfg)
    r = case.keep_ratio if r is None else r
    log(f"fused select cfg{cfg}: B={case.B} S={case.S} N={case.N} {case.dtype} r={r}")
    g = run_fused(case, keep_ratio=r)
    two = run_two_calls(case, r, case.view_logit, None, case.w_lexical, case.threshold)
    exact = not balanced_split(case)
    assert_same_select(g, two, f"cfg{cfg}", case, exact)
    if cfg in (1, 2) or not exact:
        check_select(case, g, oracle.run_path(case, keep_ratio=r, attention=False), f"fused cfg{cfg}")


@pytest.mark.parametrize("name,over", [
    ("3 views of 43 (V_full = 129, not a multiple of 4), one masked, D=64",
     dict(B=3, N=3, Tv=43, T=7, Hq=4, Hkv=2, D=64, n_masked=1, keep_ratio=0.4)),
    ("one view", dict(B=2, N=1, Tv=100, T=9, Hq=8, Hkv=2, D=128, n_masked=0, keep_ratio=0.5)),
    ("8 views of 24, up to 4 masked", dict(B=4, N=8, Tv=24, T=5, Hq=8, Hkv=8, D=128, n_masked=4, keep_ratio=0.7)),
    ("the most visual tokens: 8 views of 2048 (V_full = 16384), D=64",
     dict(B=1, N=8, Tv=2048, T=16, Hq=8, Hkv=2, D=64, n_masked=2, keep_ratio=0.25)),
    ("the most samples: 256 x (2 views of 16 + 4 text), D=64",
     dict(B=256, N=2, Tv=16, T=4, Hq=2, Hkv=1, D=64, n_masked=(0, 1), keep_ratio=0.5)),
])
def test_fused_select_view_layouts(name, over):
    """View boundaries off the 4-key vectors and the 64-key tiles, a single
    view, the most views the in-call selection takes, the most visual tokens
    and samples the calls take: bit for bit the two-call path, and the
    oracle's selection."""
    case = synth.config_case(2, **over)
    log(f"fused select {name}: B={case.B} N={case.N} V_full={case.V_full} S={case.S}")
    g = run_fused(case)
    two = run_two_calls(case, case.keep_ratio, case.view_logit, None, case.w_lexical, case.threshold)
    assert_same_select(g, two, name, case, not balanced_split(case))
    check_select(case, g, oracle.run_path(case, attention=False), name)


@pytest.mark.parametrize("name,over,one_full", [
    ("16 samples, the most the balanced split takes",
     dict(B=16, N=4, Tv=96, T=12, Hq=8, Hkv=2, D=128, n_masked=(0, 3), keep_ratio=0.4), False),
    ("251 key tiles per sample (8 views of 2000 + 16 text), D=64",
     dict(B=2, N=8, Tv=2000, T=16, Hq=4, Hkv=1, D=64, n_masked=(0, 4), keep_ratio=0.3), False),
    ("one sample keeps every view, five keep one",
     dict(B=6, N=6, Tv=200, T=16, Hq=8, Hkv=2, D=128, n_masked=0, keep_ratio=0.5), True),
    ("two 512-row blocks per (sample, KV group): 160 text tokens x 4 heads",
     dict(B=2, N=4, Tv=128, T=160, Hq=8, Hkv=2, D=128, n_masked=(0, 2), keep_ratio=0.5), False),
    ("fp32, 3 samples", dict(cfg=1, B=3, N=3, Tv=64, T=16, n_masked=(0, 1), keep_ratio=0.5), False),
])
def test_fused_select_balanced_split_limits(name, over, one_full):
    """The balanced sweep-1 split at its limits: the most samples it takes, a
    sequence near its 256 key tiles, and a sample that keeps every view beside
    samples that keep one (that sample takes the most splits). Against the
    two-call path by the band rule, and the oracle's selection."""
    over = dict(over)
    case = synth.config_case(over.pop("cfg", 2), **over)
    if one_full:
        logit = np.full((case.B, case.N), -8.0, np.float32)
        logit[0, :] = 8.0
        logit[1:, 0] = 8.0
        case = dataclasses.replace(case, view_logit=logit)
    assert balanced_split(case), name
    log(f"balanced split {name}: B={case.B} N={case.N} V_full={case.V_full} S={case.S}")
    g = run_fused(case)
    two = run_two_calls(case, case.keep_ratio, case.view_logit, None, case.w_lexical, case.threshold)
    assert_same_select(g, two, name, case, exact=False)
    check_select(case, g, oracle.run_path(case, attention=False), name)


def test_fused_select_beyond_balanced_split():
    """17 samples, one past the balanced split's limit: the first sweep splits
    tile ranges evenly again, and the in-call selection equals the two calls
    bit for bit (and the oracle's selection)."""
    case = synth.config_case(2, B=17, N=4, Tv=96, T=12, Hq=8, Hkv=2, D=128, n_masked=(0, 3), keep_ratio=0.4)
    assert not balanced_split(case)
    log(f"beyond the balanced split: B={case.B} N={case.N} V_full={case.V_full} S={case.S}")
    g = run_fused(case)
    two = run_two_calls(case, case.keep_ratio, case.view_logit, None, case.w_lexical, case.threshold)
    assert_same_select(g, two, "B=17", case, exact=True)
    check_select(case, g, oracle.run_path(case, attention=False), "B=17")


def test_fused_select_random_logits_lexical_fallback():
    """Logits near the threshold, lexical scores, and samples where no view
    passes (the best-view fallback): the in-call decision is the patch-select
    kernel's, bit for bit, for several (w, tau)."""
    rng = np.random.default_rng(21)
    case = synth.config_case(2, B=12, N=6, Tv=40, T=16, Hq=8, Hkv=2, D=128)
    tau0 = 0.6
    x0 = math.log(tau0 / (1 - tau0))
    logit = (x0 + rng.normal(0, 1e-3, (case.B, case.N))).astype(np.float32)
    logit[2] = -15.0
    logit[5, :] = x0 - 1.0
    lex = rng.random((case.B, case.N)).astype(np.float32)
    for w, tau, lx in ((0.0, tau0, None), (0.3, 0.55, lex), (1.0, 0.7, lex), (0.0, 0.999, None)):
        g = run_fused(case, logit=logit, lexical=lx, w=w, tau=tau)
        two = run_two_calls(case, case.keep_ratio, logit, lx, w, tau)
        assert_same_select(g, two, f"w={w} tau={tau}", case, not balanced_split(case))
        n_band = check_view_keep(oracle.view_scores(logit, lx, w), tau, g["view_keep"])
        log(f"fused w={w} tau={tau}: views kept {int(g['view_keep'].sum())} of {case.B * case.N}, "
            f"{n_band} in the threshold band")


# scoring from the last n text tokens only (n = 1: the last-token readout)
ROWS_CASES = [
    ("rows1-cfg2", dict(cfg=2), 1),
    ("rows1-ragged-gqa", dict(cfg=4, Tv=100, T=37, keep_ratio=0.37), 1),
    ("rows7-ragged-gqa", dict(cfg=4, run=1, Tv=96, T=37, keep_ratio=0.5), 7),
    ("rows2-d64", dict(cfg=2, Tv=50, T=3, Hq=6, Hkv=3, D=64, keep_ratio=0.9), 2),
    ("rows1-fp8", dict(cfg=5, Tv=128, T=32), 1),
    ("rows1-f32", dict(cfg=1), 1),
    ("rowsT-cfg2", dict(cfg=2, Tv=64, T=16), 16),
]


@pytest.mark.parametrize("name", [c[0] for c in ROWS_CASES])
def test_select_query_rows_matches_oracle(name):
    spec = {c[0]: c for c in ROWS_CASES}[name]
    kw, n = dict(spec[1]), spec[2]
    cfg = kw.pop("cfg")
    case = synth.config_case(cfg, **kw)
    log(f"select {name}: B={case.B} S={case.S} V={case.V_full} Hq={case.Hq} Hkv={case.Hkv} D={case.D} {case.dtype} r={case.keep_ratio} query rows {n}")
    g = run_select(case, query_rows=n)
    ref = oracle.run_path(case, attention=False, query_rows=n)
    check_select(case, g, ref, name)
    if n == case.S - case.V_full:
        # every text row: the same call as litevlm_token_score_topk, bit for bit
        g2 = run_select(case)
        for key in ("scores", "kept_index", "cu"):
            assert np.array_equal(g[key], g2[key]), key


def test_cfg3_full_size_last_token():
    # the last-token readout at the full 6x1024 + 128 shape
    case = synth.config_case(3)
    log("select cfg3 last token: S=6272 r=0.5")
    g = run_select(case, keep_ratio=0.5, query_rows=1)
    ref = oracle.run_path(case, keep_ratio=0.5, attention=False, query_rows=1)
    check_select(case, g, ref, "cfg3-last-token")


def test_chain_is_deterministic():
    case = synth.config_case(4, Tv=128, T=32)
    a = run_select(case)
    b = run_select(case)
    for key in ("scores", "kept_index", "cu"):
        assert np.array_equal(a[key], b[key]), key
    m = int(np.max(np.diff(a["cu"])))
    oa = attention_on(case, a["dev"]["qc"], a["dev"]["kc"], a["dev"]["vc"], a["dev"]["cu_seqlens"], m)
    ob = attention_on(case, b["dev"]["qc"], b["dev"]["kc"], b["dev"]["vc"], b["dev"]["cu_seqlens"], m)
    assert torch.equal(oa[:a["cu"][-1]].view(torch.int16), ob[:a["cu"][-1]].view(torch.int16))


def test_graph_replay_matches_eager():
    """The step's three calls captured in one HIP graph: every replay, with eager
    work (the outputs cleared) and a sync between replays, reproduces the eager
    results bit for bit."""
    case = synth.config_case(4, Tv=128, T=32)
    B, S, Hq, Hkv, D, V = case.B, case.S, case.Hq, case.Hkv, case.D, case.V_full
    q, k, v = (to_device(x, case.dtype) for x in (case.q, case.k, case.v))
    logit = torch.from_numpy(case.view_logit).cuda()
    out = dict(scores=torch.empty((B, V), dtype=torch.float32, device="cuda"),
               kept_index=torch.empty((B * S,), dtype=torch.int32, device="cuda"),
               cu_seqlens=torch.empty((B + 1,), dtype=torch.int32, device="cuda"),
               qc=torch.empty((B * S, Hq, D), dtype=q.dtype, device="cuda"),
               kc=torch.empty((B * S, Hkv, D), dtype=q.dtype, device="cuda"),
               vc=torch.empty((B * S, Hkv, D), dtype=q.dtype, device="cuda"),
               workspace=torch.empty((lv.workspace_bytes(B, S, V, Hq, Hkv, D),), dtype=torch.uint8,
                                     device="cuda"))
    o = torch.empty((B * S, Hq, D), dtype=torch.bfloat16, device="cuda")

    def step():
        _, tk, _ = lv.patch_select(logit, case.view_offsets, S, case.w_lexical, case.threshold)
        lv.token_score_topk(q, k, v, tk, case.keep_ratio, V, q_scale=case.q_scale, k_scale=case.k_scale,
                            v_scale=case.v_scale, out=out)
        lv.prefill_attn(out["qc"], out["kc"], out["vc"], out["cu_seqlens"], S, B=B, q_scale=case.q_scale,
                        k_scale=case.k_scale, v_scale=case.v_scale, out=o)

    step()
    torch.cuda.synchronize()
    total = int(out["cu_seqlens"][-1])
    names = ("scores", "kept_index", "cu_seqlens", "qc", "kc", "vc")
    rows = {"kept_index": total, "qc": total, "kc": total, "vc": total}
    ref = {n: out[n][:rows.get(n, out[n].shape[0])].clone() for n in names}
    ref_o = o[:total].clone()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        step()
    torch.cuda.current_stream().wait_stream(side)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        step()
    for rep in range(3):
        for t in list(out.values()) + [o]:
            t.zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for n in names:
            got = out[n][:rows.get(n, out[n].shape[0])]
            assert torch.equal(got.view(torch.uint8), ref[n].view(torch.uint8)), f"replay {rep}: {n}"
        assert torch.equal(o[:total].view(torch.int16), ref_o.view(torch.int16)), f"replay {rep}: o"
    log(f"graph replays: 3 x bitwise equal to eager ({total} packed rows)")


def test_full_keep_equals_unpruned_attention():
    case = synth.config_case(2, Tv=64, T=16, keep_ratio=1.0, n_masked=0)
    g = run_select(case)
    assert np.array_equal(g["kept_index"], np.arange(case.S))
    o_chain = attention_on(case, g["dev"]["qc"], g["dev"]["kc"], g["dev"]["vc"], g["dev"]["cu_seqlens"], case.S)
    cu = np.array([0, case.S], np.int32)
    o_full = attention_on(case, g["q"].view(case.S, case.Hq, case.D), g["k"].view(case.S, case.Hkv, case.D),
                          g["v"].view(case.S, case.Hkv, case.D), cu, case.S)
    assert torch.equal(o_chain[:case.S].view(torch.int16), o_full.view(torch.int16))


# ----------------------------------------------------------------------------- exact ties

def kept_visual_scores(g, b, V_full):
    return g["scores"][b, :V_full][g["token_keep"][b, :V_full] == 1]


@pytest.mark.parametrize("which", ["cfg2", "cfg3-r0.5"])
def test_exact_ties_zero_queries(which):
    """All queries zero: every attention row is uniform over its visible keys,
    so every kept visual token scores (1/T)*sum_t 1/(V_b+t+1) exactly and all
    of them tie. The GPU scores must be bitwise equal and the kept set must be
    the lowest k_b positions, index for index; the attention over the chain is
    then a prefix mean of V."""
    base = synth.config_case(2) if which == "cfg2" else synth.config_case(3, keep_ratio=0.5)
    case = synth.with_zero_queries(base)
    log(f"zero-query ties {which}: S={case.S} Hq={case.Hq} Hkv={case.Hkv} r={case.keep_ratio}")
    g = run_select(case)
    ref = oracle.run_path(case, attention=False)
    T = case.S - case.V_full
    for b in range(case.B):
        vals = kept_visual_scores(g, b, case.V_full)
        assert np.unique(vals).size == 1, f"sample {b}: {np.unique(vals).size} distinct GPU scores"
        V_b = int(ref["V_b"][b])
        closed = sum(1.0 / (V_b + t + 1) for t in range(T)) / T
        assert abs(vals[0] - closed) <= 1e-6 * closed, (vals[0], closed)
        kept = np.nonzero(ref["token_keep"][b, :case.V_full])[0]
        assert np.array_equal(ref["selected"][b], kept[:int(ref["k_b"][b])])   # the oracle's tie rule
    check_select(case, g, ref, f"zero-query {which}", exact=True)
    cu = g["cu"]
    o = attention_on(case, g["dev"]["qc"], g["dev"]["kc"], g["dev"]["vc"], g["dev"]["cu_seqlens"],
                     int(np.max(np.diff(cu))))
    ref_o = oracle.run_path(case)["o"]
    stats = check_attention(to_float64(o[:cu[-1]]), ref_o, "bf16", which)
    log(f"  attention (prefix means) {stats}")


@pytest.mark.parametrize("which", ["cfg2", "bf16-gqa", "fp8-gqa"])
def test_exact_ties_duplicated_keys_straddle_k(which):
    """Six kept visual tokens share one key row (bitwise), lifted above the
    other tokens; k is chosen so that the group straddles rank k. The members'
    GPU scores must be bitwise equal and exactly the lower-positioned members
    must be kept."""
    if which == "cfg2":
        base = synth.config_case(2)
    elif which == "bf16-gqa":
        base = synth.config_case(4, B=1, Tv=200, T=24, n_masked=1)
    else:
        base = synth.config_case(5, B=1, Tv=256, T=32)
    vk = oracle.patch_select(base.view_logit, None, base.w_lexical, base.threshold)
    tk = oracle.token_keep_from_views(vk, base.view_offsets, base.S)
    cand = np.nonzero(tk[0, :base.V_full])[0]
    n = len(cand)
    members = sorted({int(cand[i]) for i in (n // 3, 7, n // 6, n // 2, (2 * n) // 3, n - 3)})
    case = synth.with_duplicated_keys(base, 0, members, beta=3.0)
    q64, k64, _ = oracle.decode_inputs(case)
    s = oracle.token_scores(q64, k64, tk, case.V_full, case.Hq, case.Hkv, 1 / math.sqrt(case.D))[0]
    sg = s[members[0]]
    assert np.all(s[members] == sg), "oracle: identical keys must score identically"
    others = np.setdiff1d(cand, members)
    assert np.min(np.abs(s[others] - sg)) > 1e-5 * sg, "group not isolated from the other scores"
    above = int(np.sum(s[others] > sg))
    k = above + len(members) // 2
    r = k / n
    assert oracle.keep_count(r, n) == k
    want = np.sort(np.concatenate([others[s[others] > sg], members[:len(members) // 2]]))
    log(f"duplicated keys {which}: V_b={n} members {members} above {above} k={k}")
    g = run_select(case, keep_ratio=r)
    ref = oracle.run_path(case, keep_ratio=r, attention=False)
    assert np.array_equal(ref["selected"][0], want)                       # the oracle's tie rule
    got_s = g["scores"][0, members]
    assert np.unique(got_s).size == 1, f"GPU member scores differ: {got_s}"
    case_r = dataclasses.replace(case, keep_ratio=r)
    check_select(case_r, g, ref, f"duplicated keys {which}", exact=True)
    assert np.array_equal(g["kept_index"][:k], want)


# ----------------------------------------------------------------------------- full sizes

def full_size_chain(case, label, kind, keep_ratio=None):
    """The whole chain at a full workload size: selection against the oracle,
    then attention over every packed row and head. When the kept sets equal
    the oracle's, the attention runs on the chain's own compacted buffers;
    otherwise (near-ties) on the oracle's compacted inputs. The attention grid
    is sized from the host bound floor(r*V_full + 1e-6) + T, as the benchmark
    sizes it."""
    r = case.keep_ratio if keep_ratio is None else keep_ratio
    g = run_select(case, keep_ratio=r)
    ref = oracle.run_path(case, keep_ratio=r, attention=False)
    identical = check_select(case, g, ref, label)
    T = case.S - case.V_full
    bound = oracle.keep_count(r, case.V_full) + T
    cu = ref["cu_seqlens"]
    assert int(np.max(np.diff(cu))) <= bound
    if identical:
        o = attention_on(case, g["dev"]["qc"], g["dev"]["kc"], g["dev"]["vc"], g["dev"]["cu_seqlens"], bound)
    else:
        qc, kc, vc = (to_device(ref[n], case.dtype) for n in ("qc_bits", "kc_bits", "vc_bits"))
        o = attention_on(case, qc, kc, vc, cu, bound)
    q64, k64, v64 = oracle.decode_inputs(case)
    ref_o = oracle.prefill_attention(oracle.gather_rows(q64, ref["kept_index"], cu),
                                     oracle.gather_rows(k64, ref["kept_index"], cu),
                                     oracle.gather_rows(v64, ref["kept_index"], cu),
                                     cu, case.Hq, case.Hkv, 1 / math.sqrt(case.D))
    stats = check_attention(to_float64(o[:cu[-1]]), ref_o, kind, label)
    log(f"  {label}: identical sets {identical}; attention over all {cu[-1]} rows x {case.Hq} heads {stats}")


@pytest.mark.parametrize("r", synth.CFG3_KEEP_SWEEP)
def test_cfg3_full_size(r):
    case = synth.config_case(3, keep_ratio=r)
    log(f"cfg3 full size r={r}: S={case.S} Hq={case.Hq} Hkv={case.Hkv}")
    full_size_chain(case, f"cfg3 r={r}", "bf16")


def test_cfg3_full_size_peaked():
    # Q, K ~ N(0,1): logits of standard deviation ~1 instead of ~1/D
    case = synth.config_case(3, run=1, keep_ratio=0.5, peaked=True)
    log("cfg3 full size peaked r=0.5")
    full_size_chain(case, "cfg3 peaked r=0.5", "bf16")


def test_cfg4_full_size_ragged():
    case = synth.config_case(4)
    log(f"cfg4 full size: B={case.B} masked={[len(m) for m in case.masked_views]}")
    full_size_chain(case, "cfg4", "bf16")


def test_cfg5_full_size_fp8():
    case = synth.config_case(5)
    log(f"cfg5 full size: B={case.B} fp8 e4m3, scales {case.q_scale:.3g} {case.k_scale:.3g} {case.v_scale:.3g}")
    full_size_chain(case, "cfg5", "fp8")


def test_cfg5_full_size_fp8_peaked():
    case = synth.config_case(5, run=1, peaked=True)
    log(f"cfg5 full size peaked: B={case.B} masked={[len(m) for m in case.masked_views]}")
    full_size_chain(case, "cfg5 peaked", "fp8")


@pytest.mark.parametrize("r", synth.CFG3_KEEP_SWEEP)
def test_fp8_batch1_keep_sweep(r):
    """The 6x1024 batch-1 shape in E4M3 across the keep-ratio sweep."""
    case = synth.config_case(3, dtype="fp8", keep_ratio=r)
    log(f"fp8 6x1024 batch 1 r={r}: scales {case.q_scale:.3g} {case.k_scale:.3g} {case.v_scale:.3g}")
    full_size_chain(case, f"fp8 batch1 r={r}", "fp8")


# ----------------------------------------------------------------------------- grid bound

@pytest.mark.parametrize("dtype", ["bf16", "fp8", "f32"])
def test_attention_grid_bound_above_lengths(dtype):
    """max_seqlen only sizes the grid: a bound far above the real lengths (the
    uncompressed S) gives bitwise the output of the tight bound, and both match
    the oracle."""
    lens = [700, 130, 0, 1, 257] if dtype != "f32" else [150, 0, 65, 1]
    Hq, Hkv, D = (32, 8, 128) if dtype != "f32" else (4, 2, 64)
    qb, kb, vb, scales, cu = synth.random_attention_inputs(lens, Hq, Hkv, D, dtype, seed=321, peaked=True)
    q, k, v = (to_device(x, dtype) for x in (qb, kb, vb))
    cu_d = torch.from_numpy(cu).cuda()
    outs = []
    for bound in (max(lens), 6272):
        o = lv.prefill_attn(q, k, v, cu_d, bound, q_scale=scales[0], k_scale=scales[1], v_scale=scales[2])
        torch.cuda.synchronize()
        outs.append(o)
    assert torch.equal(outs[0].view(torch.uint8), outs[1].view(torch.uint8))
    q64, k64, v64 = (oracle.litevlm.decode_stored(x, dtype, sc) for x, sc in zip((qb, kb, vb), scales))
    ref = oracle.prefill_attention(q64, k64, v64, cu, Hq, Hkv, 1 / math.sqrt(D))
    stats = check_attention(to_float64(outs[1]), ref, attn_kind(dtype), f"bound {dtype}")
    log(f"  grid bound 6272 vs {max(lens)}: bitwise equal; {stats}")
