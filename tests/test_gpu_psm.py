"""GPU parity of the Patch Selection Module forward pass (litevlm_psm_forward)
against the oracle's psm_forward.

The GPU rounds every GEMM and attention input to bf16 (fp32 accumulation), so
the logits carry a few parts in a thousand of the activations' scale; the bound
|got - ref| <= 2e-2 + 2e-2*|ref| leaves about 4x headroom over what the bf16
rounding of 4 layers gives. The view decisions of the patch selection made from
the GPU logits must equal the oracle's wherever a logit is not within 0.1 of the
threshold's logit (0 at w_lexical 0, threshold 0.5)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2506_07416_amd as lv
import synth
from oracle import psm as OP
from parity_util import log

pytestmark = pytest.mark.gpu

PSM_RTOL, PSM_ATOL = 2e-2, 2e-2

CASES = [
    ("2 layers, 16 tokens, d 256", dict(B=1, T=16, d=256, H=4, dff=512, N=6, L=2)),
    ("benchmark shape: 4 layers, 128 tokens, d 256, batch 3", dict(B=3, T=128, d=256, H=4, dff=1024, N=6, L=4)),
    ("d 512, head dim 128, ragged 37 tokens", dict(B=2, T=37, d=512, H=4, dff=256, N=3, L=1)),
]


def run(c, seed):
    emb, par = synth.psm_inputs(c["B"], c["T"], c["d"], c["dff"], c["N"], c["L"], seed)
    out = lv.psm_forward(torch.from_numpy(emb).cuda(), torch.from_numpy(par).cuda(), c["H"], c["dff"], c["N"], c["L"])
    torch.cuda.synchronize()
    ref = OP.psm_forward(emb.astype(np.float64), par.astype(np.float64), c["H"], c["dff"], c["N"], c["L"])
    return out, ref


@pytest.mark.parametrize("name,c", CASES)
def test_psm_matches_oracle(name, c):
    out, ref = run(c, seed=5100 + c["T"])
    got = out.cpu().numpy().astype(np.float64)
    err = np.abs(got - ref)
    assert np.all(err <= PSM_ATOL + PSM_RTOL * np.abs(ref)), f"{name}: max err {err.max():.3g}"
    log(f"{name}: logits max abs err {err.max():.2e} (|ref| max {np.abs(ref).max():.2f})")
    # the patch selection made from these logits
    vk, _, _ = lv.patch_select(out, np.arange(c["N"] + 1) * 4, 4 * c["N"] + 1, 0.0, 0.5)
    vk_ref = oracle.patch_select(ref.astype(np.float32), None, 0.0, 0.5)
    clear = np.abs(ref) > 0.1
    assert np.array_equal(vk.cpu().numpy()[clear], vk_ref[clear])


def test_psm_is_deterministic():
    c = CASES[1][1]
    a, _ = run(c, seed=5200)
    b, _ = run(c, seed=5200)
    assert torch.equal(a, b)
