"""The no-alloc scoring entry point (litevlm_token_score_topk_noalloc) against
the workspace entry point (litevlm_token_score_topk): the same inputs must give
bitwise the same scores, indices, lengths and gathered rows, on two calls in a
row (the second on a smaller input, over the scratch the first one left), and
shapes whose workspace exceeds the scratch array are refused on the host."""
import numpy as np
import pytest
import torch

import paper_2506_07416_amd as lv
import synth
from paper_2506_07416_amd import _abi
from parity_util import log, to_device

pytestmark = pytest.mark.gpu


def select(case, noalloc):
    q, k, v = (to_device(x, case.dtype) for x in (case.q, case.k, case.v))
    logit = torch.from_numpy(case.view_logit).cuda()
    _, token_keep, _ = lv.patch_select(logit, case.view_offsets, case.S, case.w_lexical, case.threshold)
    out = lv.token_score_topk(q, k, v, token_keep, case.keep_ratio, case.V_full, q_scale=case.q_scale,
                              k_scale=case.k_scale, v_scale=case.v_scale, noalloc=noalloc)
    torch.cuda.synchronize()
    return out


def assert_same(a, b, label):
    total = int(a["cu_seqlens"][-1])
    assert torch.equal(a["cu_seqlens"], b["cu_seqlens"]), label
    assert torch.equal(a["scores"].view(torch.int32), b["scores"].view(torch.int32)), label
    assert torch.equal(a["kept_index"][:total], b["kept_index"][:total]), label
    for n in ("qc", "kc", "vc"):
        assert torch.equal(a[n][:total].view(torch.uint8), b[n][:total].view(torch.uint8)), f"{label}: {n}"
    return total


def test_noalloc_matches_workspace_call_two_calls():
    # the batch-8 ragged workload at full size, then the smaller 6x256 one
    cases = [synth.config_case(4), synth.config_case(2)]
    for i, case in enumerate(cases):
        need = lv.workspace_bytes(case.B, case.S, case.V_full, case.Hq, case.Hkv, case.D)
        assert need <= _abi.NOALLOC_SCRATCH_BYTES
        log(f"no-alloc call {i}: B={case.B} S={case.S} Hq={case.Hq} Hkv={case.Hkv} workspace {need} bytes")
        ref = select(case, noalloc=False)
        got = select(case, noalloc=True)
        total = assert_same(ref, got, f"call {i}")
        log(f"  bitwise equal over {total} packed rows")


def test_noalloc_refuses_oversized_workspace():
    # B=256 at the 6x1024 shape needs more workspace than the scratch array holds:
    # refused on the host (fake, never-touched device addresses)
    lib = lv.load()
    B, S, V, Hq, Hkv, D = 256, 6272, 6144, 32, 8, 128
    assert lv.workspace_bytes(B, S, V, Hq, Hkv, D) > _abi.NOALLOC_SCRATCH_BYTES
    A = 0x7F0000000000
    st = lib.litevlm_token_score_topk_noalloc(_abi.BF16, B, S, V, Hq, Hkv, D, A, A, A, 0.088, 1.0, 1.0, 1.0,
                                              A, 0.5, A, A, A, A, A, A, None)
    assert st == _abi.ERR_WORKSPACE
