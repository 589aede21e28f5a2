"""C-ABI checks that need no GPU: the library loads, exports every symbol the
header declares, and rejects bad arguments on the host before any HIP call
(fake, never-dereferenced device addresses are passed)."""
import ctypes
import os
import re

import pytest

import paper_2506_07416_amd as lv
from paper_2506_07416_amd import _abi

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "litevlm.h")

A = 0x7F0000000000          # a 256-byte aligned fake device address (never touched)
MIS = A + 8                  # 8-byte aligned only


def header_symbols():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"\b(litevlm_[a-z0-9_]+)\s*\(", text)))


def test_library_exports_every_header_symbol():
    lib = lv.load()
    syms = header_symbols()
    assert set(syms) == set(_abi.SIGNATURES), (syms, sorted(_abi.SIGNATURES))
    for s in syms:
        assert hasattr(lib, s), s


def test_version_and_status_strings():
    lib = lv.load()
    assert lib.litevlm_version() >= 100
    for code in range(8):
        assert lib.litevlm_status_string(code)
    assert lib.litevlm_status_string(99) == b"unknown status"


def test_header_constants_match_binding():
    text = open(HEADER).read()
    assert int(re.search(r"LITEVLM_MAX_VIEWS (\d+)", text).group(1)) == _abi.MAX_VIEWS
    assert int(re.search(r"LITEVLM_MAX_VISUAL (\d+)", text).group(1)) == _abi.MAX_VISUAL
    assert int(re.search(r"LITEVLM_MAX_BATCH (\d+)", text).group(1)) == _abi.MAX_BATCH
    assert int(re.search(r"LITEVLM_MAX_HEADS (\d+)", text).group(1)) == _abi.MAX_HEADS
    assert int(re.search(r"LITEVLM_MAX_FUSED_VIEWS (\d+)", text).group(1)) == _abi.MAX_FUSED_VIEWS


# ----------------------------------------------------------------------------- patch_select

def ps(B=2, N=3, S=20, off=(0, 4, 8, 12), logit=A, lex=None, w=0.0, tau=0.5, vk=A, tk=A, nv=A):
    lib = lv.load()
    offs = None if off is None else (ctypes.c_int32 * len(off))(*off)
    return lib.litevlm_patch_select(B, N, S, offs, logit, lex, w, tau, vk, tk, nv, None)


def test_patch_select_validation():
    assert ps(logit=None) == _abi.ERR_NULL_POINTER
    assert ps(off=None) == _abi.ERR_NULL_POINTER
    assert ps(tk=None) == _abi.ERR_NULL_POINTER
    assert ps(B=0) == _abi.ERR_BAD_SHAPE
    assert ps(N=0) == _abi.ERR_BAD_SHAPE
    assert ps(N=65, off=tuple(range(66))) == _abi.ERR_BAD_SHAPE
    assert ps(off=(1, 4, 8, 12)) == _abi.ERR_BAD_SHAPE          # must start at 0
    assert ps(off=(0, 8, 4, 12)) == _abi.ERR_BAD_SHAPE          # must ascend
    assert ps(off=(0, 4, 8, 21)) == _abi.ERR_BAD_SHAPE          # V_full > S
    assert ps(w=1.5) == _abi.ERR_BAD_VALUE
    assert ps(w=float("nan")) == _abi.ERR_BAD_VALUE
    assert ps(tau=float("inf")) == _abi.ERR_BAD_VALUE
    assert ps(logit=A + 2) == _abi.ERR_MISALIGNED
    assert ps(nv=A + 1) == _abi.ERR_MISALIGNED


# ----------------------------------------------------------------------------- select_score_topk

def sst(N=3, off=(0, 20, 40, 80), logit=A, lex=None, w=0.0, tau=0.5, B=1, S=100, V=80, ws=A, wsb=None,
        q=A, vk=A, tk=A, nv=A):
    lib = lv.load()
    if wsb is None:
        wsb = lib.litevlm_token_score_topk_workspace(B, S, V, 8, 2, 128)
    offs = None if off is None else (ctypes.c_int32 * len(off))(*off)
    return lib.litevlm_select_score_topk(_abi.BF16, B, S, V, 8, 2, 128, N, offs, logit, lex, w, tau, q, A, A,
                                         0.088, 1.0, 1.0, 1.0, 0.5, vk, tk, nv, A, A, A, A, A, A, ws, wsb,
                                         None)


def test_select_score_topk_validation():
    assert sst(logit=None) == _abi.ERR_NULL_POINTER
    assert sst(off=None) == _abi.ERR_NULL_POINTER
    assert sst(q=None) == _abi.ERR_NULL_POINTER
    assert sst(N=0) == _abi.ERR_BAD_SHAPE
    assert sst(off=(1, 20, 40, 80)) == _abi.ERR_BAD_SHAPE       # must start at 0
    assert sst(off=(0, 40, 20, 80)) == _abi.ERR_BAD_SHAPE       # must ascend
    assert sst(off=(0, 20, 40, 70)) == _abi.ERR_BAD_SHAPE       # the views must end at V_full
    assert sst(N=9, off=tuple(range(0, 81, 10))) == _abi.ERR_UNSUPPORTED   # beyond the fused limit
    assert sst(N=65, off=tuple(range(66))) == _abi.ERR_BAD_SHAPE
    assert sst(w=1.5) == _abi.ERR_BAD_VALUE
    assert sst(tau=float("nan")) == _abi.ERR_BAD_VALUE
    assert sst(logit=A + 2) == _abi.ERR_MISALIGNED
    assert sst(nv=A + 1) == _abi.ERR_MISALIGNED
    assert sst(ws=None) == _abi.ERR_WORKSPACE
    assert sst(wsb=16) == _abi.ERR_WORKSPACE
    # the selection outputs are optional
    assert sst(vk=None, tk=None, nv=None, ws=None) == _abi.ERR_WORKSPACE


# ----------------------------------------------------------------------------- token_score_topk

def st(dtype=_abi.BF16, B=1, S=100, V=80, Hq=8, Hkv=2, D=128, q=A, k=A, v=A, sm=0.088,
       qs=1.0, ks=1.0, vs=1.0, keep=A, r=0.5, scores=A, ki=A, cu=A, qc=A, kc=A, vc=A, ws=A,
       wsb=None):
    lib = lv.load()
    if wsb is None:
        wsb = lib.litevlm_token_score_topk_workspace(B, S, V, Hq, Hkv, D)
    return lib.litevlm_token_score_topk(dtype, B, S, V, Hq, Hkv, D, q, k, v, sm, qs, ks, vs, keep, r,
                                        scores, ki, cu, qc, kc, vc, ws, wsb, None)


def test_workspace_size():
    lib = lv.load()
    n = lib.litevlm_token_score_topk_workspace(1, 6272, 6144, 32, 8, 128)
    # per-key-split row stats (at least one split) + fixed-point column sums
    R = 4 * 128
    assert n >= 8 * 8 * 1 * R + 8 * 6144
    assert n % 256 == 0
    # the rows variant with every text row needs exactly as much; fewer rows, less
    assert lib.litevlm_token_score_topk_rows_workspace(1, 6272, 6144, 32, 8, 128, 128) == n
    n1 = lib.litevlm_token_score_topk_rows_workspace(1, 6272, 6144, 32, 8, 128, 1)
    assert 8 * 6144 <= n1 < n
    assert lib.litevlm_token_score_topk_rows_workspace(1, 6272, 6144, 32, 8, 128, 0) == 0
    assert lib.litevlm_token_score_topk_rows_workspace(1, 6272, 6144, 32, 8, 128, 129) == 0
    assert lib.litevlm_token_score_topk_workspace(1, 10, 10, 8, 2, 128) == 0    # no text token
    assert lib.litevlm_token_score_topk_workspace(1, 100, 80, 8, 3, 128) == 0   # Hq % Hkv


def test_token_score_topk_validation():
    assert st(q=None) == _abi.ERR_NULL_POINTER
    assert st(scores=None) == _abi.ERR_NULL_POINTER
    assert st(cu=None) == _abi.ERR_NULL_POINTER
    assert st(v=None) == _abi.ERR_NULL_POINTER                  # vc requested without v
    assert st(dtype=7) == _abi.ERR_UNSUPPORTED
    assert st(Hkv=3) == _abi.ERR_BAD_SHAPE
    assert st(D=96) == _abi.ERR_BAD_SHAPE
    assert st(Hq=256, Hkv=2) == _abi.ERR_BAD_SHAPE               # beyond LITEVLM_MAX_HEADS
    assert st(S=80) == _abi.ERR_BAD_SHAPE                      # T = 0
    assert st(V=20000, S=20010) == _abi.ERR_BAD_SHAPE          # beyond the top-k limit
    assert st(B=0) == _abi.ERR_BAD_SHAPE
    assert st(B=257) == _abi.ERR_BAD_SHAPE
    assert st(r=1.5) == _abi.ERR_BAD_VALUE
    assert st(r=-0.1) == _abi.ERR_BAD_VALUE
    assert st(r=float("nan")) == _abi.ERR_BAD_VALUE
    assert st(sm=0.0) == _abi.ERR_BAD_VALUE
    assert st(qs=2.0) == _abi.ERR_BAD_VALUE                    # scales only for fp8
    assert st(dtype=_abi.FP8_E4M3, qs=float("inf")) == _abi.ERR_BAD_VALUE
    assert st(q=MIS) == _abi.ERR_MISALIGNED
    assert st(qc=MIS) == _abi.ERR_MISALIGNED
    assert st(ws=MIS) == _abi.ERR_MISALIGNED
    assert st(ki=A + 2) == _abi.ERR_MISALIGNED
    assert st(ws=None) == _abi.ERR_WORKSPACE
    assert st(wsb=16) == _abi.ERR_WORKSPACE


def test_token_score_topk_rows_validation():
    lib = lv.load()

    def rows(n, S=100, V=80, wsb=None, q=A):
        if wsb is None:
            wsb = lib.litevlm_token_score_topk_rows_workspace(1, S, V, 8, 2, 128, max(1, min(n, S - V)))
        return lib.litevlm_token_score_topk_rows(_abi.BF16, 1, S, V, 8, 2, 128, n, q, A, A, 0.088, 1.0,
                                                 1.0, 1.0, A, 0.5, A, A, A, A, A, A, A, wsb, None)
    assert rows(0) == _abi.ERR_BAD_VALUE
    assert rows(21) == _abi.ERR_BAD_VALUE                       # T = 20
    assert rows(-3) == _abi.ERR_BAD_VALUE
    assert rows(5, q=None) == _abi.ERR_NULL_POINTER
    assert rows(5, S=80) == _abi.ERR_BAD_SHAPE                  # T = 0
    assert rows(5, wsb=16) == _abi.ERR_WORKSPACE


# ----------------------------------------------------------------------------- prefill_attn

def pa(ind=_abi.BF16, outd=_abi.BF16, B=2, Hq=8, Hkv=2, D=128, q=A, k=A, v=A, cu=A, ml=100,
       sm=0.088, qs=1.0, ks=1.0, vs=1.0, causal=1, o=A):
    lib = lv.load()
    return lib.litevlm_prefill_attn(ind, outd, B, Hq, Hkv, D, q, k, v, cu, ml, sm, qs, ks, vs,
                                    causal, o, None)


def test_prefill_attn_validation():
    assert pa(q=None) == _abi.ERR_NULL_POINTER
    assert pa(cu=None) == _abi.ERR_NULL_POINTER
    assert pa(o=None) == _abi.ERR_NULL_POINTER
    assert pa(ind=5) == _abi.ERR_UNSUPPORTED
    assert pa(outd=_abi.FP8_E4M3) == _abi.ERR_UNSUPPORTED
    assert pa(Hkv=3) == _abi.ERR_BAD_SHAPE
    assert pa(D=256) == _abi.ERR_BAD_SHAPE
    assert pa(B=0) == _abi.ERR_BAD_SHAPE
    assert pa(ml=-1) == _abi.ERR_BAD_SHAPE
    assert pa(causal=2) == _abi.ERR_BAD_VALUE
    assert pa(sm=float("nan")) == _abi.ERR_BAD_VALUE
    assert pa(vs=0.5) == _abi.ERR_BAD_VALUE
    assert pa(ind=_abi.FP8_E4M3, qs=-1.0) == _abi.ERR_BAD_VALUE
    assert pa(o=MIS) == _abi.ERR_MISALIGNED
    assert pa(k=MIS) == _abi.ERR_MISALIGNED
    assert pa(cu=A + 1) == _abi.ERR_MISALIGNED


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(_abi, "_LIB", None)
    monkeypatch.setattr(_abi, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(ImportError):
        _abi.load()


# ----------------------------------------------------------------------------- decode_attn

def da(ind=_abi.BF16, outd=_abi.BF16, B=2, Hq=32, Hkv=8, D=128, q1=A, k1=A, v1=A, kc=A, vc=A, cu=A,
       ml=3200, sm=0.088, qs=1.0, ks=1.0, vs=1.0, o=A, ws=A, wsb=None):
    lib = lv.load()
    if wsb is None:
        wsb = lib.litevlm_decode_attn_workspace(ind, B, Hq, Hkv, D, ml)
    return lib.litevlm_decode_attn(ind, outd, B, Hq, Hkv, D, q1, k1, v1, kc, vc, cu, ml, sm, qs, ks,
                                   vs, o, ws, wsb, None)


def test_decode_workspace_size():
    lib = lv.load()
    # batch 1, 8 KV heads: short splits (64 keys) so the grid fills the chip
    n = lib.litevlm_decode_attn_workspace(_abi.BF16, 1, 32, 8, 128, 3200)
    splits = (3200 + 64) // 64
    assert n >= 32 * splits * (128 * 4 + 8)
    # batch 8: long splits (256 keys) already give enough workgroups
    n8 = lib.litevlm_decode_attn_workspace(_abi.BF16, 8, 32, 8, 128, 6272)
    assert 8 * 32 * ((6272 + 256) // 256) * (128 * 4 + 8) <= n8 < 8 * 32 * ((6272 + 64) // 64) * 520
    assert lib.litevlm_decode_attn_workspace(_abi.BF16, 1, 32, 8, 128, 0) > 0   # new token only
    assert lib.litevlm_decode_attn_workspace(_abi.BF16, 1, 48, 8, 128, 100) == 0  # G = 6
    assert lib.litevlm_decode_attn_workspace(_abi.BF16, 1, 32, 3, 128, 100) == 0  # Hq % Hkv
    assert lib.litevlm_decode_attn_workspace(9, 1, 32, 8, 128, 100) == 0


def test_decode_attn_validation():
    assert da(q1=None) == _abi.ERR_NULL_POINTER
    assert da(k1=None) == _abi.ERR_NULL_POINTER
    assert da(vc=None) == _abi.ERR_NULL_POINTER
    assert da(cu=None) == _abi.ERR_NULL_POINTER
    assert da(o=None) == _abi.ERR_NULL_POINTER
    assert da(ind=5, wsb=1 << 20) == _abi.ERR_UNSUPPORTED
    assert da(outd=_abi.FP8_E4M3) == _abi.ERR_UNSUPPORTED
    assert da(Hq=48, wsb=1 << 20) == _abi.ERR_UNSUPPORTED       # G = 6
    assert da(Hq=256, Hkv=16, wsb=1 << 20) == _abi.ERR_BAD_SHAPE
    assert da(Hkv=3, wsb=1 << 20) == _abi.ERR_BAD_SHAPE
    assert da(D=96, wsb=1 << 20) == _abi.ERR_BAD_SHAPE
    assert da(B=0, wsb=1 << 20) == _abi.ERR_BAD_SHAPE
    assert da(ml=-1, wsb=1 << 20) == _abi.ERR_BAD_SHAPE
    assert da(sm=0.0) == _abi.ERR_BAD_VALUE
    assert da(qs=2.0) == _abi.ERR_BAD_VALUE                    # scales only for fp8
    assert da(ind=_abi.FP8_E4M3, vs=float("nan")) == _abi.ERR_BAD_VALUE
    assert da(kc=MIS) == _abi.ERR_MISALIGNED
    assert da(o=MIS) == _abi.ERR_MISALIGNED
    assert da(ws=MIS) == _abi.ERR_MISALIGNED
    assert da(cu=A + 2) == _abi.ERR_MISALIGNED
    assert da(ws=None) == _abi.ERR_WORKSPACE
    assert da(wsb=64) == _abi.ERR_WORKSPACE


def test_tsm_validation():
    lib = lv.load()

    def tq(B=1, S=100, V=80, Dm=256, Hq=8, Hkv=2, D=128, x=A, keep=A, wq=A, wk=A, eps=1e-5, th=1e6, q=A, k=A):
        return lib.litevlm_tsm_qk(B, S, V, Dm, Hq, Hkv, D, x, keep, wq, wk, eps, th, q, k, None)
    assert tq(x=None) == _abi.ERR_NULL_POINTER
    assert tq(wk=None) == _abi.ERR_NULL_POINTER
    assert tq(q=None) == _abi.ERR_NULL_POINTER
    assert tq(S=80) == _abi.ERR_BAD_SHAPE                     # no text token
    assert tq(Dm=100) == _abi.ERR_BAD_SHAPE                   # not a multiple of 64
    assert tq(Dm=96) == _abi.ERR_BAD_SHAPE
    assert tq(D=96) == _abi.ERR_BAD_SHAPE
    assert tq(Hkv=3) == _abi.ERR_BAD_SHAPE
    assert tq(Hq=2, Hkv=1, D=64) == _abi.ERR_UNSUPPORTED       # Hkv*D = 64 < 128
    assert tq(eps=0.0) == _abi.ERR_BAD_VALUE
    assert tq(th=1.0) == _abi.ERR_BAD_VALUE
    assert tq(th=float("inf")) == _abi.ERR_BAD_VALUE
    assert tq(x=MIS) == _abi.ERR_MISALIGNED
    assert tq(k=MIS) == _abi.ERR_MISALIGNED
    assert lib.litevlm_tsm_fold_gain(4, 8, None, A, A, None) == _abi.ERR_NULL_POINTER
    assert lib.litevlm_tsm_fold_gain(0, 8, A, A, A, None) == _abi.ERR_BAD_SHAPE
    assert lib.litevlm_tsm_fold_gain(4, 8, A, A + 2, A, None) == _abi.ERR_MISALIGNED


def test_gather_hidden_validation():
    lib = lv.load()

    def gh(B=2, S=100, rb=8192, h=A, ki=A, cu=A, o=A):
        return lib.litevlm_gather_hidden(B, S, rb, h, ki, cu, o, None)
    assert gh(h=None) == _abi.ERR_NULL_POINTER
    assert gh(cu=None) == _abi.ERR_NULL_POINTER
    assert gh(B=0) == _abi.ERR_BAD_SHAPE
    assert gh(rb=8) == _abi.ERR_BAD_SHAPE
    assert gh(rb=8200) == _abi.ERR_BAD_SHAPE
    assert gh(rb=48 * 256 * 16 + 16) == _abi.ERR_BAD_SHAPE
    assert gh(h=MIS) == _abi.ERR_MISALIGNED
    assert gh(ki=A + 2) == _abi.ERR_MISALIGNED


def test_psm_validation():
    lib = lv.load()
    n = lib.litevlm_psm_param_count(256, 1024, 6, 4)
    per_layer = 4 * 256 + 3 * 256 * 256 + 3 * 256 + 256 * 256 + 256 + 1024 * 256 + 1024 + 256 * 1024 + 256
    assert n == 4 * per_layer + 2 * 256 + 6 * 256 + 3 * (256 * 256 + 256) + 6 * 256 + 6
    assert lib.litevlm_psm_workspace(1, 128, 256, 4, 1024) > 0
    assert lib.litevlm_psm_workspace(1, 128, 200, 4, 1024) == 0

    def pf(B=1, T=128, d=256, H=4, dff=1024, N=6, L=4, e=A, p=A, npar=None, o=A, ws=A, wsb=None):
        npar = lib.litevlm_psm_param_count(d, dff, N, L) if npar is None else npar
        wsb = lib.litevlm_psm_workspace(B, T, d, H, dff) if wsb is None else wsb
        return lib.litevlm_psm_forward(B, T, d, H, dff, N, L, e, p, npar, o, ws, wsb, None)
    assert pf(e=None) == _abi.ERR_NULL_POINTER
    assert pf(o=None) == _abi.ERR_NULL_POINTER
    assert pf(d=128, wsb=1 << 30) == _abi.ERR_BAD_SHAPE
    assert pf(H=8) == _abi.ERR_UNSUPPORTED                     # head dim 32
    assert pf(dff=1000, wsb=1 << 30) == _abi.ERR_BAD_SHAPE
    assert pf(N=0) == _abi.ERR_BAD_SHAPE
    assert pf(npar=5) == _abi.ERR_BAD_SHAPE
    assert pf(p=A + 4) == _abi.ERR_MISALIGNED
    assert pf(ws=None) == _abi.ERR_WORKSPACE
    assert pf(wsb=100) == _abi.ERR_WORKSPACE
