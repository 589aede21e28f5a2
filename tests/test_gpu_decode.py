"""GPU parity of the extend-one decode step (litevlm_decode_attn) against the
oracle's decode_attention.

The cache is either random packed rows from the seeded generator, or, at full
size, the compacted K/V that the oracle's own selection chain produces for the
seeded workloads; the new token comes from the seeded generator. No input of
the oracle comes from the GPU.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import paper_2506_07416_amd as lv
import synth
from parity_util import check_attention, log, to_device, to_float64

pytestmark = pytest.mark.gpu


def decode_gpu(q1, k1, v1, kc, vc, cu, max_seqlen, dtype, scales, out_dtype=None):
    o = lv.decode_attn(to_device(q1, dtype), to_device(k1, dtype), to_device(v1, dtype),
                       to_device(kc, dtype), to_device(vc, dtype),
                       torch.from_numpy(np.asarray(cu, np.int32)).cuda(), max_seqlen,
                       q_scale=scales[0], k_scale=scales[1], v_scale=scales[2], out_dtype=out_dtype)
    torch.cuda.synchronize()
    return o


def decode_ref(q1, k1, v1, kc, vc, cu, Hq, Hkv, D, dtype, scales):
    dec = oracle.litevlm.decode_stored
    return oracle.decode_attention(dec(q1, dtype, scales[0]), dec(k1, dtype, scales[1]),
                                   dec(v1, dtype, scales[2]), dec(kc, dtype, scales[1]),
                                   dec(vc, dtype, scales[2]), cu, Hq, Hkv, 1.0 / math.sqrt(D))


def kind_of(dtype):
    return {"f32": "f32", "bf16": "bf16", "fp8": "fp8"}[dtype]


# (name, cache lengths, Hq, Hkv, D, dtype, peaked, extra max_seqlen, out dtype)
CASES = [
    ("f32 MHA D64 edges", [0, 1, 63, 64, 65, 200], 4, 4, 64, "f32", True, 0, None),
    ("bf16 GQA4 D128 short splits", [0, 1, 63, 64, 65, 255, 256, 257, 700], 32, 8, 128, "bf16", True, 37, None),
    ("bf16 GQA4 D128 long splits", [2100, 1999, 0, 512, 513, 1, 2047, 300], 32, 8, 128, "bf16", True, 0, None),
    ("bf16 GQA2 D128 flat", [100, 1000, 31], 16, 8, 128, "bf16", False, 500, None),
    ("bf16 G8 D64", [5, 129, 640], 8, 1, 64, "bf16", True, 0, None),
    ("bf16 G8 D128 long splits", [1100, 50, 1000, 900, 7, 64, 1024, 1099], 64, 8, 128, "bf16", True, 0, None),
    ("bf16 MHA D64 long splits", [600, 2000, 1, 1500], 16, 16, 64, "bf16", True, 0, None),
    ("bf16 in f32 out", [77, 300], 32, 8, 128, "bf16", True, 0, torch.float32),
    ("f32 long splits", [1100, 3, 1024, 900, 1, 64, 1000, 1100], 32, 8, 128, "f32", True, 0, None),
    ("fp8 GQA4 D128", [0, 65, 700, 1500], 32, 8, 128, "fp8", True, 0, None),
    ("fp8 GQA2 D64 long splits", [2100, 10, 2000, 1800, 600, 2100, 5, 2050], 16, 8, 64, "fp8", True, 0, None),
    # LITEVLM_MAX_BATCH samples, cache lengths 0..300 (empty ones included)
    ("bf16 256 samples", [(37 * i) % 301 for i in range(256)], 8, 2, 64, "bf16", True, 0, None),
]


@pytest.mark.parametrize("case_id", range(len(CASES)))
def test_decode_matches_oracle(case_id):
    name, lens, Hq, Hkv, D, dtype, peaked, extra, out_dt = CASES[case_id]
    B = len(lens)
    log(f"decode case {name}: lens {lens}, Hq/Hkv {Hq}/{Hkv}, D {D}, {dtype}")
    _, kc, vc, scales, cu = synth.random_attention_inputs(lens, Hq, Hkv, D, dtype, seed=9100 + case_id,
                                                          peaked=peaked)
    q1, k1, v1, scales = synth.decode_token_inputs(B, Hq, Hkv, D, dtype, seed=9200 + case_id,
                                                   scales=scales, peaked=peaked)
    o = decode_gpu(q1, k1, v1, kc, vc, cu, max(lens) + extra, dtype, scales, out_dt)
    ref = decode_ref(q1, k1, v1, kc, vc, cu, Hq, Hkv, D, dtype, scales)
    kind = "f32" if (dtype == "f32" and o.dtype == torch.float32) else kind_of(dtype)
    st = check_attention(to_float64(o), ref, kind, name)
    log(f"  {st}")


def test_decode_empty_cache_returns_new_value():
    """With no cached token the new token attends only to itself: o = v1."""
    B, Hq, Hkv, D = 3, 8, 2, 128
    _, kc, vc, scales, cu = synth.random_attention_inputs([0, 0, 0], Hq, Hkv, D, "f32", seed=9300)
    kc = np.zeros((1, Hkv, D), np.float32)   # a valid (never read) buffer
    vc = np.zeros((1, Hkv, D), np.float32)
    q1, k1, v1, _ = synth.decode_token_inputs(B, Hq, Hkv, D, "f32", seed=9301)
    o = to_float64(decode_gpu(q1, k1, v1, kc, vc, cu, 0, "f32", (1.0, 1.0, 1.0)))
    want = np.repeat(v1.astype(np.float64), Hq // Hkv, axis=1)
    assert np.array_equal(o, want)


def test_decode_is_deterministic():
    lens = [3000, 17, 1200, 640]
    _, kc, vc, scales, cu = synth.random_attention_inputs(lens, 32, 8, 128, "bf16", seed=9400, peaked=True)
    q1, k1, v1, _ = synth.decode_token_inputs(4, 32, 8, 128, "bf16", seed=9401, peaked=True)
    a = decode_gpu(q1, k1, v1, kc, vc, cu, 3000, "bf16", scales)
    b = decode_gpu(q1, k1, v1, kc, vc, cu, 3000, "bf16", scales)
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))


@pytest.mark.parametrize("cfg,keep", [(3, 0.5), (3, 1.0), (4, None), (5, None)])
def test_decode_full_size_over_oracle_cache(cfg, keep):
    """Full-size workloads: the cache is the oracle's compacted K/V of the seeded
    prompt; every (sample, head) output is checked. max_seqlen is the prompt
    length S, as in the benchmark."""
    case = synth.config_case(cfg)
    ref_chain = oracle.run_path(case, keep_ratio=keep, attention=False)
    cu = ref_chain["cu_seqlens"]
    kc, vc = ref_chain["kc_bits"], ref_chain["vc_bits"]
    scales = (case.q_scale, case.k_scale, case.v_scale)
    q1, k1, v1, scales = synth.decode_token_inputs(case.B, case.Hq, case.Hkv, case.D, case.dtype,
                                                   seed=9500 + cfg, scales=scales)
    log(f"decode full size cfg{cfg} keep {keep}: cache lengths {np.diff(cu).tolist()}")
    o = decode_gpu(q1, k1, v1, kc, vc, cu, case.S, case.dtype, scales)
    ref = decode_ref(q1, k1, v1, kc, vc, cu, case.Hq, case.Hkv, case.D, case.dtype, scales)
    st = check_attention(to_float64(o), ref, kind_of(case.dtype), f"cfg{cfg}")
    log(f"  {st}")


def test_decode_graph_replays_match_eager():
    """The two decode launches captured in a HIP graph: every replay (with other
    GPU work and synchronisations in between) reproduces the eager output bits."""
    lens = [1971, 1356, 1049, 742]
    dtype = "bf16"
    _, kc, vc, scales, cu = synth.random_attention_inputs(lens, 32, 8, 128, dtype, seed=9600, peaked=True)
    q1, k1, v1, _ = synth.decode_token_inputs(4, 32, 8, 128, dtype, seed=9601, peaked=True)
    dq1, dk1, dv1, dkc, dvc = (to_device(x, dtype) for x in (q1, k1, v1, kc, vc))
    dcu = torch.from_numpy(cu).cuda()
    ws = torch.empty((lv.decode_workspace_bytes(torch.bfloat16, 4, 32, 8, 128, 6272),), dtype=torch.uint8,
                     device="cuda")
    out = torch.empty((4, 32, 128), dtype=torch.bfloat16, device="cuda")
    eager = lv.decode_attn(dq1, dk1, dv1, dkc, dvc, dcu, 6272, workspace=ws).clone()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        lv.decode_attn(dq1, dk1, dv1, dkc, dvc, dcu, 6272, out=out, workspace=ws)
    torch.cuda.current_stream().wait_stream(side)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        lv.decode_attn(dq1, dk1, dv1, dkc, dvc, dcu, 6272, out=out, workspace=ws)
    for rep in range(3):
        out.zero_()
        ws.fill_(0x7F)            # the graph must not depend on workspace contents
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16), eager.view(torch.int16)), f"replay {rep}"
