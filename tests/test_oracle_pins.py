"""Pins of the CPU oracle against things other than itself (CPU only).

Each check compares the oracle with a value the paper prints (Table 1), a
closed form, an invariant, a library routine (torch CPU float64 attention,
torch's E4M3 and bf16 casts, Python's sorted) or brute force on tiny inputs.
The mutation tests at the end plant plausible mistakes in copies of oracle
functions and show that at least one pin rejects each of them.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest
import torch

import oracle
from oracle import e4m3
from oracle import litevlm as O
import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ----------------------------------------------------------------------------- helpers

def rand_qk(rng, B, S, Hq, Hkv, D, peaked=True):
    div = 1.0 if peaked else math.sqrt(D)
    q = rng.standard_normal((B, S, Hq, D)) / div
    k = rng.standard_normal((B, S, Hkv, D)) / div
    v = rng.standard_normal((B, S, Hkv, D))
    return q, k, v


def sdpa_scores(q, k, token_keep, V_full, Hq, Hkv, scale, query_rows=None):
    """Importance scores read off torch's CPU float64 causal attention: with
    identity value vectors, the output row of a query IS its probability row.
    query_rows = n sums the rows of the last n text tokens only."""
    B, S = token_keep.shape
    T = S - V_full
    n = T if query_rows is None else query_rows
    G = Hq // Hkv
    out = np.full((B, V_full), -np.inf)
    for b in range(B):
        idx = O.patch_selected_positions(token_keep[b], V_full)
        S_b = idx.shape[0]
        V_b = S_b - T
        qq = torch.from_numpy(q[b, idx].transpose(1, 0, 2).copy())            # [Hq, S_b, D]
        kk = torch.from_numpy(k[b, idx].transpose(1, 0, 2).copy()).repeat_interleave(G, 0)
        eye = torch.eye(S_b, dtype=torch.float64).expand(Hq, S_b, S_b)
        prob = torch.nn.functional.scaled_dot_product_attention(
            qq, kk, eye, is_causal=True, scale=scale)                        # [Hq, S_b, S_b]
        mass = prob[:, V_b + T - n:, :V_b].sum(dim=(0, 1)).numpy() / (Hq * n)
        out[b, idx[:V_b]] = mass
    return out


def sdpa_attention(qc, kc, vc, cu, Hq, Hkv, scale):
    G = Hq // Hkv
    out = np.zeros((qc.shape[0], Hq, vc.shape[2]))
    for b in range(len(cu) - 1):
        lo, hi = cu[b], cu[b + 1]
        if hi == lo:
            continue
        qq = torch.from_numpy(qc[lo:hi].transpose(1, 0, 2).copy())
        kk = torch.from_numpy(kc[lo:hi].transpose(1, 0, 2).copy()).repeat_interleave(G, 0)
        vv = torch.from_numpy(vc[lo:hi].transpose(1, 0, 2).copy()).repeat_interleave(G, 0)
        o = torch.nn.functional.scaled_dot_product_attention(qq, kk, vv, is_causal=True, scale=scale)
        out[lo:hi] = o.numpy().transpose(1, 0, 2)
    return out


def topk_brute(scores_b, keep_b, V_full, k):
    """All k-subsets of the candidates; the valid one has every kept token
    ahead of every dropped one in (score desc, position asc) order."""
    cand = [j for j in range(V_full) if keep_b[j]]
    valid = []
    for sub in itertools.combinations(cand, k):
        s = set(sub)
        ok = all((scores_b[a] > scores_b[c]) or (scores_b[a] == scores_b[c] and a < c)
                 for a in s for c in cand if c not in s)
        if ok:
            valid.append(sorted(sub))
    return valid


def score_pins(score_fn, seed=0):
    """Run the score pins against a candidate implementation; returns the list
    of failed pin names."""
    failed = []
    rng = np.random.default_rng(seed)
    B, N, Tv, T, Hq, Hkv, D = 2, 3, 4, 3, 4, 2, 8
    V_full = N * Tv
    S = V_full + T
    off = np.arange(N + 1) * Tv
    view_keep = np.array([[1, 0, 1], [1, 1, 1]], np.uint8)
    tk = O.token_keep_from_views(view_keep, off, S)
    q, k, _ = rand_qk(rng, B, S, Hq, Hkv, D)
    scale = 1.0 / math.sqrt(D)
    got = score_fn(q, k, tk, V_full, Hq, Hkv, scale)
    # 1. library routine (torch SDPA with identity values)
    ref = sdpa_scores(q, k, tk, V_full, Hq, Hkv, scale)
    fin = np.isfinite(ref)
    if not (np.array_equal(fin, np.isfinite(got)) and np.allclose(got[fin], ref[fin], rtol=1e-12, atol=1e-15)):
        failed.append("sdpa")
    # 2. Q = 0 closed form: every row is uniform over its p_t + 1 keys
    qz = np.zeros_like(q)
    gz = score_fn(qz, k, tk, V_full, Hq, Hkv, scale)
    for b in range(B):
        V_b = int(tk[b, :V_full].sum())
        expect = sum(1.0 / (V_b + t + 1) for t in range(T)) / T
        vis = np.nonzero(tk[b, :V_full])[0]
        if not np.allclose(gz[b, vis], expect, rtol=1e-13):
            failed.append("q0_closed_form")
            break
    # 3. GQA == MHA with the KV heads repeated
    k_rep = np.repeat(k, Hq // Hkv, axis=2)
    g_mha = score_fn(q, k_rep, tk, V_full, Hq, Hq, scale)
    if not np.allclose(g_mha[fin], got[fin], rtol=1e-12):
        failed.append("gqa_equals_repeated_mha")
    # 4. visual query rows and dropped-view keys do not matter
    q2, k2 = q.copy(), k.copy()
    q2[:, :V_full] = rng.standard_normal(q2[:, :V_full].shape)
    k2[0, Tv:2 * Tv] = 100.0 * rng.standard_normal(k2[0, Tv:2 * Tv].shape)  # view 1 of sample 0 is dropped
    g2 = score_fn(q2, k2, tk, V_full, Hq, Hkv, scale)
    if not np.allclose(g2[fin], got[fin], rtol=1e-12):
        failed.append("invariances")
    return failed


# ----------------------------------------------------------------------------- fp8 / bf16 decode

def test_e4m3_table_matches_torch_and_definition():
    codes = torch.arange(256, dtype=torch.int32).to(torch.uint8)
    lib = codes.view(torch.float8_e4m3fn).to(torch.float64).numpy()
    tab = e4m3.DECODE_TABLE
    nan = np.isnan(lib)
    assert np.array_equal(nan, np.isnan(tab))
    assert np.array_equal(lib[~nan], tab[~nan])
    assert set(np.nonzero(nan)[0]) == {0x7F, 0xFF}
    assert tab[0x7E] == 448.0 and tab[0xFE] == -448.0
    assert tab[0x01] == 2.0 ** -9 and tab[0x08] == 2.0 ** -6 and tab[0x38] == 1.0
    assert tab[0x00] == 0.0 and math.copysign(1.0, tab[0x80]) == -1.0


def test_bf16_decode_matches_torch():
    rng = np.random.default_rng(1)
    x = rng.standard_normal(4096).astype(np.float32) * 10
    bits, _ = synth.encode(x, "bf16")
    lib = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(O.decode_stored(bits, "bf16"), lib)


def test_fp8_encode_roundtrip_within_half_ulp():
    rng = np.random.default_rng(2)
    x = rng.standard_normal(10000).astype(np.float32)
    bits, s = synth.encode(x, "fp8")
    back = O.decode_stored(bits, "fp8", s)
    assert np.max(np.abs(back)) <= 448 * s * (1 + 1e-7)
    # |x - q| <= half an E4M3 ulp (2^-4 relative for normals) or half the subnormal step
    err = np.abs(back - x)
    assert np.all(err <= np.maximum(np.abs(x) * 2.0 ** -4, 2.0 ** -10 * s) * (1 + 1e-6))


# ----------------------------------------------------------------------------- patch selection

def test_patch_select_reproduces_seeded_masks():
    for cfg in (2, 4):
        case = synth.config_case(cfg) if cfg == 2 else synth.make_case(
            name="small4", cfg=4, B=8, N=6, Tv=4, T=2, Hq=2, Hkv=1, D=8, dtype="f32",
            keep_ratio=0.3, n_masked=(0, 4), salient=(0.02, 0.1), beta=2.5)
        keep = oracle.patch_select(case.view_logit, None, case.w_lexical, case.threshold)
        for b in range(case.B):
            expect = np.ones(case.N, np.uint8)
            expect[case.masked_views[b]] = 0
            assert np.array_equal(keep[b], expect)


def test_patch_select_closed_forms():
    # w = 1: the lexical score alone; "above" is strict, so lex == tau drops the view
    lex = np.array([[0.5, 0.75, 0.25, 0.5]], np.float32)
    keep = oracle.patch_select(np.zeros((1, 4), np.float32), lex, 1.0, 0.5)
    assert keep.tolist() == [[0, 1, 0, 0]]
    # w = 0.5 mixes: s = 0.5*lex + 0.5*sigmoid(logit), hand values
    logit = np.array([[0.0, 2.0, -2.0]], np.float32)
    lex = np.array([[0.2, 0.0, 1.0]], np.float32)
    s = [0.5 * l + 0.5 / (1 + math.exp(-x)) for l, x in zip(lex[0], logit[0])]
    keep = oracle.patch_select(logit, lex, 0.5, 0.43)
    assert keep[0].tolist() == [int(v > 0.43) for v in s] == [0, 1, 1]
    # nothing passes: the best view is kept, lowest index among ties
    keep = oracle.patch_select(np.array([[-3.0, -1.0, -1.0, -5.0]], np.float32), None, 0.0, 0.9)
    assert keep.tolist() == [[0, 1, 0, 0]]


def test_view_scores_match_expit_in_float64():
    from scipy.special import expit
    rng = np.random.default_rng(5)
    logit = rng.normal(0, 3, (7, 6))
    lex = rng.random((7, 6))
    for w in (0.0, 0.25, 1.0):
        s = oracle.view_scores(logit, lex, w)
        assert s.dtype == np.float64
        assert np.allclose(s, w * lex + (1 - w) * expit(logit), rtol=1e-15, atol=0)
    assert np.allclose(oracle.view_scores(logit, None, 0.3), 0.7 * expit(logit), rtol=1e-15, atol=0)
    # the decision is taken in float64: a score 1e-9 above the threshold is kept
    # (in float32, sigmoid(4e-9) rounds to exactly 0.5 and the view would drop)
    keep = oracle.patch_select(np.array([[4e-9, -4e-9, 0.0]]), None, 0.0, 0.5)
    assert keep.tolist() == [[1, 0, 0]]


def test_patch_select_brute_force_all_masks():
    # for every subset of 6 views, logits +-8 select exactly that subset (or the
    # fallback to view 0 for the empty subset, all scores tie there)
    N = 6
    for bits in range(1 << N):
        want = np.array([(bits >> v) & 1 for v in range(N)], np.uint8)
        logit = np.where(want == 1, 8.0, -8.0).astype(np.float32)[None]
        keep = oracle.patch_select(logit, None, 0.0, 0.5)[0]
        if bits == 0:
            assert keep.tolist() == [1, 0, 0, 0, 0, 0]
        else:
            assert np.array_equal(keep, want)


def test_token_keep_layout_unequal_views():
    off = [0, 3, 8, 10]
    tk = oracle.token_keep_from_views(np.array([[1, 0, 1]], np.uint8), off, 13)
    assert tk[0].tolist() == [1, 1, 1, 0, 0, 0, 0, 0, 1, 1, 1, 1, 1]


# ----------------------------------------------------------------------------- k rule

def test_keep_count_matches_table1():
    with open(os.path.join(GOLDEN, "table1_token_counts.json")) as f:
        g = json.load(f)
    T = g["text_tokens"]
    for row in g["rows"]:
        V = int(round(row["patches"] * g["tokens_per_patch"]))
        assert O.keep_count(row["keep_ratio"], V) + T == row["input_tokens"], row
    # rounding to nearest or up would contradict the table
    assert round(0.3 * 3072) + T != 1063 and math.ceil(0.7 * 3072) + T != 2292


def test_keep_count_edges():
    assert O.keep_count(0.29, 100) == 29        # 28.999999999999996 without the guard
    assert O.keep_count(0.7, 6140) == 4298
    assert O.keep_count(1.0, 6144) == 6144
    assert O.keep_count(0.25, 6144) == 1536
    assert O.keep_count(0.3, 2048) == 614 and O.keep_count(0.3, 6144) == 1843
    assert O.keep_count(0.01, 50) == 0
    assert O.keep_count(1.0, 0) == 0


# ----------------------------------------------------------------------------- scores

def test_scores_pins():
    for seed in range(3):
        assert score_pins(oracle.token_scores, seed) == []


def test_scores_mass_and_permutation():
    rng = np.random.default_rng(5)
    B, N, Tv, T, Hq, Hkv, D = 1, 2, 5, 4, 2, 1, 8
    V_full, S = N * Tv, N * Tv + T
    tk = np.ones((B, S), np.uint8)
    q, k, _ = rand_qk(rng, B, S, Hq, Hkv, D)
    sc = oracle.token_scores(q, k, tk, V_full, Hq, Hkv, 1 / math.sqrt(D))
    # total visual mass is below 1 (text keys take the rest) and positive
    assert 0 < sc.sum() < 1
    # permuting visual keys permutes the scores
    perm = rng.permutation(V_full)
    k2 = k.copy()
    k2[:, :V_full] = k[:, perm]
    sc2 = oracle.token_scores(q, k2, tk, V_full, Hq, Hkv, 1 / math.sqrt(D))
    assert np.allclose(sc2[0], sc[0, perm], rtol=1e-12)


def test_scores_hand_example():
    # one head, D = 4, two visual keys, two text tokens; logits by hand
    q = np.zeros((1, 4, 1, 4))
    k = np.zeros((1, 4, 1, 4))
    q[0, 2, 0] = [1, 0, 0, 0]          # text token 0
    q[0, 3, 0] = [0, 2, 0, 0]          # text token 1
    k[0, 0, 0] = [2, 0, 0, 0]          # visual 0
    k[0, 1, 0] = [0, 1, 0, 0]          # visual 1
    k[0, 2, 0] = [1, 1, 0, 0]          # text 0
    k[0, 3, 0] = [0, 0, 0, 0]          # text 1
    scale = 0.5                         # 1/sqrt(4)
    # text 0 sees keys 0..2 with logits 0.5*(2, 0, 1); text 1 sees 0..3 with 0.5*(0, 2, 2, 0)
    r0 = [math.exp(1.0), math.exp(0.0), math.exp(0.5)]
    r1 = [math.exp(0.0), math.exp(1.0), math.exp(1.0), math.exp(0.0)]
    p0 = [x / sum(r0) for x in r0]
    p1 = [x / sum(r1) for x in r1]
    expect = [(p0[0] + p1[0]) / 2, (p0[1] + p1[1]) / 2]
    got = oracle.token_scores(q, k, np.ones((1, 4), np.uint8), 2, 1, 1, scale)
    assert np.allclose(got[0], expect, rtol=1e-14)


@pytest.mark.parametrize("n", [1, 2, 5])
def test_query_rows_scores_match_sdpa(n):
    # FastV-style readout (the last n text tokens as the only query rows)
    # against torch's float64 causal attention, with a dropped view
    rng = np.random.default_rng(11 + n)
    B, N, Tv, T, Hq, Hkv, D = 2, 3, 6, 5, 4, 2, 8
    V_full, S = N * Tv, N * Tv + T
    tk = np.ones((B, S), np.uint8)
    tk[1, Tv:2 * Tv] = 0
    q, k, _ = rand_qk(rng, B, S, Hq, Hkv, D)
    scale = 1 / math.sqrt(D)
    got = oracle.token_scores(q, k, tk, V_full, Hq, Hkv, scale, query_rows=n)
    ref = sdpa_scores(q, k, tk, V_full, Hq, Hkv, scale, query_rows=n)
    assert np.array_equal(np.isneginf(got), np.isneginf(ref))
    fin = np.isfinite(ref)
    assert np.allclose(got[fin], ref[fin], rtol=1e-12, atol=0)
    if n == T:
        assert np.array_equal(got, oracle.token_scores(q, k, tk, V_full, Hq, Hkv, scale))


def test_query_rows_last_token_closed_form():
    # Q = 0: the last token's row is uniform over its V_b + T visible keys, so
    # every kept visual token scores 1/(V_b + T), and the all-tie selection is
    # the lowest positions
    B, N, Tv, T, Hq, Hkv, D = 1, 4, 8, 6, 4, 2, 8
    V_full, S = N * Tv, N * Tv + T
    tk = np.ones((B, S), np.uint8)
    tk[0, 2 * Tv:3 * Tv] = 0
    V_b = V_full - Tv
    q = np.zeros((B, S, Hq, D))
    k = np.random.default_rng(3).standard_normal((B, S, Hkv, D))
    sc = oracle.token_scores(q, k, tk, V_full, Hq, Hkv, 0.3, query_rows=1)
    kept = tk[0, :V_full] == 1
    assert np.allclose(sc[0, kept], 1.0 / (V_b + T), rtol=1e-14)
    assert np.all(np.isneginf(sc[0, ~kept]))
    sel = O.select_topk(sc[0], tk[0], V_full, 5)
    assert sel.tolist() == [0, 1, 2, 3, 4]
    with pytest.raises(ValueError):
        oracle.token_scores(q, k, tk, V_full, Hq, Hkv, 0.3, query_rows=0)
    with pytest.raises(ValueError):
        oracle.token_scores(q, k, tk, V_full, Hq, Hkv, 0.3, query_rows=T + 1)


@pytest.mark.parametrize("seed", range(6))
def test_aligned_plant_always_selected(seed):
    case = synth.config_case(1, run=seed, plant="aligned")
    res = oracle.run_path(case, attention=False)
    sel = set(res["selected"][0].tolist())
    assert set(case.salient[0].tolist()) <= sel


def test_masked_views_never_selected_even_if_salient():
    case = synth.make_case(name="m", cfg=9, B=3, N=4, Tv=16, T=8, Hq=4, Hkv=2, D=16, dtype="f32",
                           keep_ratio=0.9, n_masked=2, salient=0.3, beta=4.0)
    res = oracle.run_path(case, attention=False)
    for b in range(case.B):
        for v in case.masked_views[b]:
            lo, hi = case.view_offsets[v], case.view_offsets[v + 1]
            assert not np.any((res["selected"][b] >= lo) & (res["selected"][b] < hi))
            assert np.all(np.isneginf(res["scores"][b, lo:hi]))


# ----------------------------------------------------------------------------- top-k

def test_topk_brute_force_with_ties():
    rng = np.random.default_rng(7)
    for trial in range(40):
        V = int(rng.integers(1, 10))
        s = rng.integers(0, 4, V).astype(np.float64) / 4.0        # many exact ties
        keep = (rng.random(V) < 0.8).astype(np.uint8)
        kk = int(rng.integers(0, keep.sum() + 1))
        got = O.select_topk(s, keep, V, kk)
        valid = topk_brute(s, keep, V, kk)
        assert len(valid) == 1 and got.tolist() == valid[0]
        cand = [j for j in range(V) if keep[j]]
        assert got.tolist() == sorted(sorted(cand, key=lambda j: (-s[j], j))[:kk])


def test_topk_all_tie_takes_lowest_indices():
    s = np.full(20, 0.125)
    assert O.select_topk(s, np.ones(20, np.uint8), 20, 7).tolist() == list(range(7))


# ----------------------------------------------------------------------------- compaction

def test_compaction_identity_at_full_keep():
    case = synth.config_case(1, keep_ratio=1.0)
    res = oracle.run_path(case, attention=False)
    assert res["kept_index"].tolist() == list(range(case.S))
    assert res["cu_seqlens"].tolist() == [0, case.S]
    assert np.array_equal(res["qc_bits"], case.q[0])


def test_compaction_layout_and_bits():
    case = synth.config_case(4, Tv=8, T=4, Hq=4, Hkv=2, D=8, dtype="bf16")
    res = oracle.run_path(case, attention=False)
    cu = res["cu_seqlens"]
    for b in range(case.B):
        seg = res["kept_index"][cu[b]:cu[b + 1]]
        assert np.all(np.diff(seg) > 0)
        assert seg[-case.T:].tolist() == list(range(case.V_full, case.S))
        assert cu[b + 1] - cu[b] == res["k_b"][b] + case.T
        assert np.array_equal(res["kc_bits"][cu[b]:cu[b + 1]], case.k[b, seg])


# ----------------------------------------------------------------------------- attention

def attention_pins(attn_fn, seed=0):
    failed = []
    rng = np.random.default_rng(seed)
    Hq, Hkv, D = 4, 2, 8
    lens = [5, 1, 9, 0, 3]
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    tot = int(cu[-1])
    qc = rng.standard_normal((tot, Hq, D))
    kc = rng.standard_normal((tot, Hkv, D))
    vc = rng.standard_normal((tot, Hkv, D))
    sc = 1 / math.sqrt(D)
    got = attn_fn(qc, kc, vc, cu, Hq, Hkv, sc)
    if not np.allclose(got, sdpa_attention(qc, kc, vc, cu, Hq, Hkv, sc), rtol=1e-12, atol=1e-13):
        failed.append("sdpa")
    # Q = 0: prefix means of V
    gz = attn_fn(np.zeros_like(qc), kc, vc, cu, Hq, Hkv, sc)
    for b in range(len(lens)):
        for i in range(lens[b]):
            for h in range(Hq):
                if not np.allclose(gz[cu[b] + i, h], vc[cu[b]:cu[b] + i + 1, h // (Hq // Hkv)].mean(0), rtol=1e-12):
                    failed.append("q0_prefix_mean")
                    return failed
    # a sequence of length 1 returns its value row
    if not np.allclose(got[cu[1], :], vc[cu[1], np.arange(Hq) // (Hq // Hkv)], rtol=1e-14):
        failed.append("len1")
    return failed


def test_attention_pins():
    for seed in range(3):
        assert attention_pins(oracle.prefill_attention, seed) == []


def test_noncausal_attention_matches_torch():
    rng = np.random.default_rng(4)
    cu = np.array([0, 9, 9, 30], np.int32)
    qc, kc, vc = rng.standard_normal((30, 6, 8)), rng.standard_normal((30, 2, 8)), rng.standard_normal((30, 2, 8))
    got = oracle.prefill_attention(qc, kc, vc, cu, 6, 2, 0.4, causal=False)
    for b in range(3):
        lo, hi = cu[b], cu[b + 1]
        if hi == lo:
            continue
        qq = torch.from_numpy(qc[lo:hi].transpose(1, 0, 2).copy())
        kk = torch.from_numpy(kc[lo:hi].transpose(1, 0, 2).copy()).repeat_interleave(3, 0)
        vv = torch.from_numpy(vc[lo:hi].transpose(1, 0, 2).copy()).repeat_interleave(3, 0)
        ref = torch.nn.functional.scaled_dot_product_attention(qq, kk, vv, scale=0.4).numpy()
        assert np.allclose(got[lo:hi], ref.transpose(1, 0, 2), rtol=1e-12, atol=1e-14)


def test_attention_rows_subset_matches_full():
    rng = np.random.default_rng(3)
    cu = np.array([0, 7, 20], np.int32)
    qc, kc, vc = rng.standard_normal((20, 4, 8)), rng.standard_normal((20, 2, 8)), rng.standard_normal((20, 2, 8))
    full = oracle.prefill_attention(qc, kc, vc, cu, 4, 2, 0.3)
    part = oracle.prefill_attention(qc, kc, vc, cu, 4, 2, 0.3, rows=[0, 6, 7, 19])
    assert np.array_equal(part[[0, 6, 7, 19]], full[[0, 6, 7, 19]])
    assert np.isnan(part[1]).all()


def test_compacted_attention_equals_masked_full_attention():
    case = synth.config_case(1, run=3)
    res = oracle.run_path(case)
    q, k, v = oracle.decode_inputs(case)
    kept = res["kept_index"]
    S = case.S
    mask = np.zeros((S, S), bool)                                  # True = may attend
    keep = np.zeros(S, bool)
    keep[kept] = True
    mask[:] = np.tril(np.ones((S, S), bool)) & keep[None, :]
    qq = torch.from_numpy(q[0].transpose(1, 0, 2).copy())
    kk = torch.from_numpy(k[0].transpose(1, 0, 2).copy())
    vv = torch.from_numpy(v[0].transpose(1, 0, 2).copy())
    full = torch.nn.functional.scaled_dot_product_attention(
        qq, kk, vv, attn_mask=torch.from_numpy(mask), scale=1 / math.sqrt(case.D)).numpy()
    assert np.allclose(res["o"], full.transpose(1, 0, 2)[kept], rtol=1e-12, atol=1e-14)


def test_full_keep_reproduces_unpruned_attention():
    case = synth.config_case(2, Tv=16, T=8, Hq=4, Hkv=4, D=16, n_masked=0, keep_ratio=1.0)
    res = oracle.run_path(case)
    q, k, v = oracle.decode_inputs(case)
    cu = np.array([0, case.S], np.int32)
    unpruned = oracle.prefill_attention(q[0], k[0], v[0], cu, case.Hq, case.Hkv, 1 / math.sqrt(case.D))
    assert np.array_equal(res["o"], unpruned)


# ----------------------------------------------------------------------------- mutation checks

def _mutant_scores(kind):
    def fn(q, k, token_keep, V_full, Hq, Hkv, scale):
        B, S = token_keep.shape
        T = S - V_full
        G = Hq // Hkv
        out = np.full((B, V_full), -np.inf)
        for b in range(B):
            idx = O.patch_selected_positions(token_keep[b], V_full)
            if kind == "no_patch_drop":
                idx = np.arange(S)
            V_b = idx.shape[0] - T
            S_b = idx.shape[0]
            acc = np.zeros(V_b)
            off = 1 if kind == "causal_off_by_one" else 0
            p = V_b + np.arange(T) + off
            blocked = np.arange(S_b)[None, :] > p[:, None]
            for h in range(Hq):
                g = h % Hkv if kind == "head_map" else h // G
                if kind == "swap_qk":
                    qt = k[b, V_full + np.arange(T), g, :]
                    kp = q[b, idx, h, :]
                else:
                    qt = q[b, V_full + np.arange(T), h, :]
                    kp = k[b, idx, g, :]
                sc = 1.0 if kind == "no_scale" else scale
                logits = (qt @ kp.T) * sc
                if kind == "drop_mask":
                    pass
                else:
                    logits[blocked] = -np.inf
                logits -= logits.max(axis=1, keepdims=True)
                e = np.exp(logits)
                prob = e / e.sum(axis=1, keepdims=True)
                acc += prob[:, :V_b].sum(axis=0)
            div = Hq if kind == "wrong_norm" else Hq * T
            out[b, idx[:V_b]] = acc / div
        return out
    return fn


@pytest.mark.parametrize("kind", ["head_map", "no_scale", "causal_off_by_one", "drop_mask",
                                  "wrong_norm", "no_patch_drop", "swap_qk"])
def test_score_pins_reject_planted_mistakes(kind):
    assert score_pins(_mutant_scores(kind)) != []


def _mutant_attention(kind):
    def fn(qc, kc, vc, cu, Hq, Hkv, scale):
        G = Hq // Hkv
        out = np.zeros((qc.shape[0], Hq, vc.shape[2]))
        for b in range(len(cu) - 1):
            lo, hi = cu[b], cu[b + 1]
            n = hi - lo
            if n == 0:
                continue
            for h in range(Hq):
                g = h % Hkv if kind == "head_map" else h // G
                L = (qc[lo:hi, h] @ kc[lo:hi, g].T) * (1.0 if kind == "no_scale" else scale)
                if kind != "no_causal":
                    L[np.triu(np.ones((n, n), bool), 1)] = -np.inf
                if kind == "anti_causal":
                    L = L.T.copy()
                L -= L.max(axis=1, keepdims=True)
                P = np.exp(L)
                P /= P.sum(axis=1, keepdims=True)
                out[lo:hi, h] = (P.T if kind == "transpose_p" else P) @ vc[lo:hi, g]
        return out
    return fn


@pytest.mark.parametrize("kind", ["head_map", "no_scale", "no_causal", "transpose_p"])
def test_attention_pins_reject_planted_mistakes(kind):
    assert attention_pins(_mutant_attention(kind)) != []


# ----------------------------------------------------------------------------- decode (extend one)

def decode_pins(fn, seed=0):
    """Pins of extend-one decode attention; returns the names of failed pins."""
    failed = []
    rng = np.random.default_rng(seed)
    Hq, Hkv, D = 6, 2, 8
    G = Hq // Hkv
    lens = [5, 0, 9, 1]
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    B, tot = len(lens), int(cu[-1])
    kc = rng.standard_normal((tot, Hkv, D))
    vc = rng.standard_normal((tot, Hkv, D))
    q1 = rng.standard_normal((B, Hq, D))
    k1 = rng.standard_normal((B, Hkv, D))
    v1 = rng.standard_normal((B, Hkv, D))
    sc = 1 / math.sqrt(D)
    got = fn(q1, k1, v1, kc, vc, cu, Hq, Hkv, sc)
    # torch float64 attention of the one query row over [cache; itself]
    for b in range(B):
        lo, hi = cu[b], cu[b + 1]
        kk = torch.from_numpy(np.concatenate([kc[lo:hi], k1[b][None]], 0).transpose(1, 0, 2).copy())
        vv = torch.from_numpy(np.concatenate([vc[lo:hi], v1[b][None]], 0).transpose(1, 0, 2).copy())
        qq = torch.from_numpy(q1[b][:, None, :].copy())
        ref = torch.nn.functional.scaled_dot_product_attention(
            qq, kk.repeat_interleave(G, 0), vv.repeat_interleave(G, 0), scale=sc)[:, 0].numpy()
        if not np.allclose(got[b], ref, rtol=1e-12, atol=1e-13):
            failed.append("sdpa")
            break
    # the last row of the prefill attention over the sequence with the new token appended
    qs, ks, vs, cu2 = [], [], [], [0]
    for b in range(B):
        lo, hi = cu[b], cu[b + 1]
        qs.append(np.concatenate([np.zeros((hi - lo, Hq, D)), q1[b][None]], 0))
        ks.append(np.concatenate([kc[lo:hi], k1[b][None]], 0))
        vs.append(np.concatenate([vc[lo:hi], v1[b][None]], 0))
        cu2.append(cu2[-1] + hi - lo + 1)
    full = oracle.prefill_attention(np.concatenate(qs), np.concatenate(ks), np.concatenate(vs),
                                    np.asarray(cu2, np.int32), Hq, Hkv, sc, rows=np.asarray(cu2[1:]) - 1)
    if not np.allclose(got, full[np.asarray(cu2[1:]) - 1], rtol=1e-12, atol=1e-13):
        failed.append("prefill_last_row")
    # Q = 0: the mean of every value row, the new one included
    gz = fn(np.zeros_like(q1), k1, v1, kc, vc, cu, Hq, Hkv, sc)
    for b in range(B):
        lo, hi = cu[b], cu[b + 1]
        want = np.concatenate([vc[lo:hi], v1[b][None]], 0).mean(0)[np.arange(Hq) // G]
        if not np.allclose(gz[b], want, rtol=1e-12, atol=1e-14):
            failed.append("q0_mean")
            break
    # an empty cache returns the new value row
    if not np.allclose(got[1], v1[1][np.arange(Hq) // G], rtol=1e-14):
        failed.append("empty_cache")
    return failed


def test_decode_pins():
    for seed in range(3):
        assert decode_pins(oracle.decode_attention, seed) == []


def _mutant_decode(kind):
    def fn(q1, k1, v1, kc, vc, cu, Hq, Hkv, scale):
        B, _, D = q1.shape
        G = Hq // Hkv
        out = np.zeros((B, Hq, D))
        for b in range(B):
            lo, hi = cu[b], cu[b + 1]
            for h in range(Hq):
                g = h % Hkv if kind == "head_map" else h // G
                keys = kc[lo:hi, g] if kind == "no_self" else np.concatenate([kc[lo:hi, g], k1[b, g][None]], 0)
                vals = vc[lo:hi, g] if kind == "no_self" else np.concatenate([vc[lo:hi, g], v1[b, g][None]], 0)
                if keys.shape[0] == 0:
                    continue
                lg = (keys @ q1[b, h]) * (1.0 if kind == "no_scale" else scale)
                lg -= lg.max()
                p = np.exp(lg)
                p /= p.sum()
                out[b, h] = p @ vals
        return out
    return fn


@pytest.mark.parametrize("kind", ["head_map", "no_self", "no_scale"])
def test_decode_pins_reject_planted_mistakes(kind):
    assert decode_pins(_mutant_decode(kind)) != []
