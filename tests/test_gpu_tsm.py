"""GPU parity of the Token Selection Module front end (litevlm_tsm_qk, with
the gain folded by litevlm_tsm_fold_gain) against the oracle's tsm_qk.

The oracle takes the gain and the unfolded weights in float64; the GPU folds
the gain into bf16 weights and rounds its outputs to bf16, so the comparison
allows for bf16 rounding: |got - ref| <= 1e-2 + 2e-2*|ref| elementwise and a
per-(row, head) relative L2 error of at most 1e-2 (bf16 output rounding alone
gives about 2e-3, the folded-weight rounding about as much again).

Key rows are compared for the kept tokens; the kernel leaves the key rows of
dropped tokens untouched, which is checked against a sentinel written before
the call."""
import numpy as np
import pytest
import torch

import oracle
import paper_2506_07416_amd as lv
import synth
from oracle import tsm as OT
from parity_util import log, row_rel_l2, to_device, to_float64

pytestmark = pytest.mark.gpu

EPS, THETA = 1e-5, 1e6
TSM_RTOL, TSM_ATOL, TSM_ROW_L2 = 2e-2, 1e-2, 1e-2
SENTINEL = 0x7FA5  # a bf16 NaN payload no computed key row holds


def run(case, Dm, seed, eps=EPS, theta=THETA, use_keep=True):
    B, S, V, Hq, Hkv, D = case.B, case.S, case.V_full, case.Hq, case.Hkv, case.D
    hid, gamma, wq, wk = synth.tsm_inputs(B, S, Dm, Hq, Hkv, D, seed)
    tk = None
    keep_ref = np.ones((B, S), np.uint8)
    if use_keep:
        _, tk, _ = lv.patch_select(torch.from_numpy(case.view_logit).cuda(), case.view_offsets, S,
                                   case.w_lexical, case.threshold)
        vk_ref = oracle.patch_select(case.view_logit, case.view_lexical, case.w_lexical, case.threshold)
        keep_ref = oracle.token_keep_from_views(vk_ref, case.view_offsets, S)
    g = torch.from_numpy(gamma).cuda()
    wq_f = lv.tsm_fold_gain(to_device(wq, "bf16"), g)
    wk_f = lv.tsm_fold_gain(to_device(wk, "bf16"), g)
    k0 = torch.full((B, S, Hkv, D), SENTINEL, dtype=torch.int16, device="cuda").view(torch.bfloat16)
    q, k = lv.tsm_qk(to_device(hid, "bf16"), tk, V, wq_f, wk_f, Hq, Hkv, D, eps=eps, rope_theta=theta, k=k0)
    torch.cuda.synchronize()
    if tk is not None:
        assert np.array_equal(tk.cpu().numpy(), keep_ref)
    kept = keep_ref.astype(bool)
    kbits = k.cpu().view(torch.int16).numpy()
    assert (kbits[~kept] == SENTINEL).all(), "key rows of dropped tokens were written"
    dec = oracle.litevlm.decode_stored
    qr, kr = OT.tsm_qk(dec(hid, "bf16"), keep_ref, V, gamma.astype(np.float64), dec(wq, "bf16"),
                       dec(wk, "bf16"), Hq, Hkv, D, eps, theta)
    return to_float64(q[:, V:]), to_float64(k.cpu()[torch.from_numpy(kept)]), qr, kr[kept]


def check(got, ref, what):
    err = np.abs(got - ref)
    bad = err > TSM_ATOL + TSM_RTOL * np.abs(ref)
    rl2 = row_rel_l2(got, ref)
    assert not bad.any(), f"{what}: {bad.sum()} elements out of tolerance, max abs {err.max():.3g}"
    assert rl2.max() <= TSM_ROW_L2, f"{what}: row relative L2 {rl2.max():.3g}"
    return float(err.max()), float(rl2.max())


@pytest.mark.parametrize("name,over,Dm", [
    ("3 views x 64 + 32 text, one view dropped, D=128", dict(B=2, N=3, Tv=64, T=32, Hq=4, Hkv=2, D=128,
                                                            n_masked=1), 256),
    ("ragged rows, D=64, GQA 8/2", dict(B=1, N=2, Tv=100, T=37, Hq=8, Hkv=2, D=64, n_masked=0), 192),
    ("MHA 16/16 D=128, 2 of 6 views dropped", dict(B=1, N=6, Tv=40, T=64, Hq=16, Hkv=16, D=128,
                                                   n_masked=2), 512),
    # LITEVLM_MAX_BATCH samples: 256 key row tiles of 256, the tiles dealt by rank
    ("256 samples of 2 views x 48 + 16 text, GQA 4/2", dict(B=256, N=2, Tv=48, T=16, Hq=4, Hkv=2, D=128,
                                                           n_masked=(0, 1)), 256),
])
def test_tsm_matches_oracle(name, over, Dm):
    case = synth.config_case(2, **over)
    q, k, qr, kr = run(case, Dm, seed=4100)
    sq = check(q, qr, name + " q")
    sk = check(k, kr, name + " k")
    log(f"{name}: q max abs {sq[0]:.2e} row L2 {sq[1]:.2e}; k max abs {sk[0]:.2e} row L2 {sk[1]:.2e}")


def test_tsm_without_token_keep_uses_plain_positions():
    case = synth.config_case(2, B=1, N=2, Tv=64, T=16, Hq=4, Hkv=2, D=128, n_masked=0)
    q, k, qr, kr = run(case, 128, seed=4200, use_keep=False)
    check(q, qr, "q")
    check(k, kr, "k")


@pytest.mark.parametrize("cfg,B", [(3, 1), (4, 2), (4, 3)])
def test_tsm_full_size(cfg, B):
    """The 6x1024 + 128 shape with model width Hq*D = 4096 (batch 1, and the
    ragged batch with 0-4 views dropped per sample, cut to 2 and 3 samples to
    keep the float64 oracle within seconds; 3 samples take the 256 x 256 tiles):
    every key row and text query row."""
    case = synth.config_case(cfg) if B == 1 else synth.config_case(cfg, B=B)
    q, k, qr, kr = run(case, case.Hq * case.D, seed=4300 + cfg)
    sq = check(q, qr, f"cfg{cfg} q")
    sk = check(k, kr, f"cfg{cfg} k")
    log(f"cfg{cfg}: q max abs {sq[0]:.2e} row L2 {sq[1]:.2e}; k max abs {sk[0]:.2e} row L2 {sk[1]:.2e}")


@pytest.mark.parametrize("cfg,B", [(2, 1), (4, 3)])
def test_tsm_scoring_chain_and_hidden_gather(cfg, B):
    """The selection path from hidden states: patch select, TSM q/k, scoring with
    no Q/K/V copies, then the hidden states of the kept tokens gathered for the
    LLM. The gathered rows are exact copies at the GPU's kept indices; the
    lengths follow the k rule; the scores agree with the oracle's scores from the
    oracle's own q/k to within the effect of the bf16 q/k rounding."""
    case = synth.config_case(cfg, B=B) if cfg == 4 else synth.config_case(cfg)
    Dm = case.Hq * case.D
    hid, gamma, wq, wk = synth.tsm_inputs(case.B, case.S, Dm, case.Hq, case.Hkv, case.D, seed=4400 + cfg)
    _, tk, nv = lv.patch_select(torch.from_numpy(case.view_logit).cuda(), case.view_offsets, case.S,
                                case.w_lexical, case.threshold)
    g = torch.from_numpy(gamma).cuda()
    x = to_device(hid, "bf16")
    q, k = lv.tsm_qk(x, tk, case.V_full, lv.tsm_fold_gain(to_device(wq, "bf16"), g),
                     lv.tsm_fold_gain(to_device(wk, "bf16"), g), case.Hq, case.Hkv, case.D, eps=EPS,
                     rope_theta=THETA)
    out = lv.token_score_topk(q, k, None, tk, case.keep_ratio, case.V_full, gather=False)
    hc = lv.gather_hidden(x, out["kept_index"], out["cu_seqlens"])
    torch.cuda.synchronize()
    cu = out["cu_seqlens"].cpu().numpy()
    ki = out["kept_index"][:cu[-1]].cpu().numpy()
    got = hc[:cu[-1]].cpu().view(torch.int16).numpy().view(np.uint16)
    want = np.concatenate([hid[b, ki[cu[b]:cu[b + 1]]] for b in range(case.B)])
    assert np.array_equal(got, want), "gathered hidden rows differ from the input rows"
    # lengths: k rule on the oracle's own patch selection
    vk = oracle.patch_select(case.view_logit, case.view_lexical, case.w_lexical, case.threshold)
    tk_ref = oracle.token_keep_from_views(vk, case.view_offsets, case.S)
    V_b = tk_ref[:, :case.V_full].sum(axis=1)
    k_b = [oracle.keep_count(case.keep_ratio, int(v)) for v in V_b]
    assert np.array_equal(np.diff(cu), np.array(k_b) + (case.S - case.V_full))
    # scores against the oracle's scores from its float64 q/k
    dec = oracle.litevlm.decode_stored
    qr, kr = OT.tsm_qk(dec(hid, "bf16"), tk_ref, case.V_full, gamma.astype(np.float64), dec(wq, "bf16"),
                       dec(wk, "bf16"), case.Hq, case.Hkv, case.D, EPS, THETA)
    qfull = np.zeros((case.B, case.S, case.Hq, case.D))
    qfull[:, case.V_full:] = qr
    ref = oracle.token_scores(qfull, kr, tk_ref, case.V_full, case.Hq, case.Hkv, 1.0 / np.sqrt(case.D))
    s = out["scores"].cpu().numpy().astype(np.float64)
    fin = np.isfinite(ref)
    assert np.array_equal(fin, np.isfinite(s))
    rel = np.abs(s[fin] - ref[fin]) / ref[fin]
    log(f"cfg{cfg} B={case.B}: score rel err from bf16 q/k median {np.median(rel):.2e} max {rel.max():.2e}; "
        f"lengths {np.diff(cu).tolist()}")
    assert np.median(rel) < 1e-2 and rel.max() < 1e-1
