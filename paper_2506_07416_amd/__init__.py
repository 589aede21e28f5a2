"""LiteVLM select + prefill hot path on MI355X (gfx950).

Thin Python binding over the C ABI of liblitevlm.so: it checks tensor
placement and shapes, allocates outputs with PyTorch (device memory and the
current stream are all PyTorch provides) and passes raw pointers. Every step of
the path runs in the library's HIP kernels:

    psm_forward(...)       the Patch Selection Module's view logits from the query embeddings
    patch_select(...)      view selection and per-view patch masking
    token_score_topk(...)  visual-token scoring, top-k and gather compaction
    prefill_attn(...)      causal GQA prefill attention over the packed sequence
    decode_attn(...)       extend-one decode attention over the compacted KV cache
    tsm_qk(...)            the Token Selection Module's scoring q and k from hidden states
"""
from __future__ import annotations

import ctypes
import math
from typing import Optional, Sequence

import torch

from . import _abi
from ._abi import LiteVLMError, load  # noqa: F401

__all__ = ["patch_select", "token_score_topk", "select_score_topk", "prefill_attn", "decode_attn", "tsm_qk", "tsm_fold_gain",
           "gather_hidden", "psm_forward",
           "dtype_code",
           "workspace_bytes", "decode_workspace_bytes", "LiteVLMError", "load"]


def dtype_code(t: torch.dtype) -> int:
    if t == torch.float32:
        return _abi.F32
    if t == torch.bfloat16:
        return _abi.BF16
    if t in (torch.float8_e4m3fn, torch.uint8):
        return _abi.FP8_E4M3
    raise TypeError(f"unsupported dtype {t}")


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("tensors must live on the GPU")
    if not t.is_contiguous():
        raise ValueError("tensors must be contiguous")
    return t.data_ptr()


def _stream(device) -> int:
    return torch.cuda.current_stream(device).cuda_stream


def patch_select(view_logit: torch.Tensor, view_offsets: Sequence[int], S: int,
                 w_lexical: float = 0.0, threshold: float = 0.5,
                 view_lexical: Optional[torch.Tensor] = None):
    """View selection + patch mask. view_logit: fp32 [B, N] on the GPU.
    Returns (view_keep uint8 [B,N], token_keep uint8 [B,S], n_visual_kept int32 [B])."""
    lib = load()
    B, N = view_logit.shape
    dev = view_logit.device
    view_keep = torch.empty((B, N), dtype=torch.uint8, device=dev)
    token_keep = torch.empty((B, S), dtype=torch.uint8, device=dev)
    n_vis = torch.empty((B,), dtype=torch.int32, device=dev)
    off = (ctypes.c_int32 * (N + 1))(*[int(x) for x in view_offsets])
    st = lib.litevlm_patch_select(B, N, S, off, _ptr(view_logit), _ptr(view_lexical),
                                  float(w_lexical), float(threshold), _ptr(view_keep),
                                  _ptr(token_keep), _ptr(n_vis), _stream(dev))
    _abi.check(st, "litevlm_patch_select")
    return view_keep, token_keep, n_vis


def workspace_bytes(B: int, S: int, V_full: int, Hq: int, Hkv: int, D: int,
                    query_rows: Optional[int] = None) -> int:
    if query_rows is None:
        return int(load().litevlm_token_score_topk_workspace(B, S, V_full, Hq, Hkv, D))
    return int(load().litevlm_token_score_topk_rows_workspace(B, S, V_full, Hq, Hkv, D, int(query_rows)))


def token_score_topk(q: torch.Tensor, k: torch.Tensor, v: Optional[torch.Tensor],
                     token_keep: Optional[torch.Tensor], keep_ratio: float, V_full: int,
                     softmax_scale: Optional[float] = None, q_scale: float = 1.0,
                     k_scale: float = 1.0, v_scale: float = 1.0, gather: bool = True,
                     workspace: Optional[torch.Tensor] = None, out: Optional[dict] = None,
                     query_rows: Optional[int] = None, noalloc: bool = False) -> dict:
    """Scores, top-k and compaction. q: [B,S,Hq,D], k/v: [B,S,Hkv,D] (fp32, bf16 or
    E4M3 bytes). Returns a dict of device tensors: scores [B,V_full] fp32,
    kept_index [B*S] int32 (packed, valid up to cu_seqlens[B]), cu_seqlens [B+1],
    and when gather is set qc [B*S,Hq,D], kc/vc [B*S,Hkv,D] (valid rows likewise).
    ``out`` may supply preallocated tensors under the same keys (plus "workspace").
    query_rows = n scores with the last n text tokens as the only query rows
    (litevlm_token_score_topk_rows); None uses every text token. noalloc calls
    litevlm_token_score_topk_noalloc, whose workspace is the library's own
    device array (no workspace tensor is made or passed)."""
    lib = load()
    B, S, Hq, D = q.shape
    Hkv = k.shape[2]
    dev = q.device
    if softmax_scale is None:
        softmax_scale = 1.0 / math.sqrt(D)
    o = dict(out or {})
    o.setdefault("scores", torch.empty((B, V_full), dtype=torch.float32, device=dev))
    o.setdefault("kept_index", torch.empty((B * S,), dtype=torch.int32, device=dev))
    o.setdefault("cu_seqlens", torch.empty((B + 1,), dtype=torch.int32, device=dev))
    if gather:
        o.setdefault("qc", torch.empty((B * S, Hq, D), dtype=q.dtype, device=dev))
        o.setdefault("kc", torch.empty((B * S, Hkv, D), dtype=k.dtype, device=dev))
        o.setdefault("vc", torch.empty((B * S, Hkv, D), dtype=v.dtype, device=dev))
    if noalloc:
        if query_rows is not None or workspace is not None:
            raise ValueError("the no-alloc call scores every text row and takes no workspace")
        st = lib.litevlm_token_score_topk_noalloc(
            dtype_code(q.dtype), B, S, V_full, Hq, Hkv, D, _ptr(q), _ptr(k), _ptr(v), float(softmax_scale),
            float(q_scale), float(k_scale), float(v_scale), _ptr(token_keep), float(keep_ratio),
            _ptr(o["scores"]), _ptr(o["kept_index"]), _ptr(o["cu_seqlens"]), _ptr(o.get("qc")),
            _ptr(o.get("kc")), _ptr(o.get("vc")), _stream(dev))
        _abi.check(st, "litevlm_token_score_topk_noalloc")
        return o
    nbytes = workspace_bytes(B, S, V_full, Hq, Hkv, D, query_rows)
    ws = workspace if workspace is not None else o.get("workspace")
    if ws is None:
        ws = torch.empty((max(nbytes, 1),), dtype=torch.uint8, device=dev)
    o["workspace"] = ws
    common = (_ptr(q), _ptr(k), _ptr(v), float(softmax_scale), float(q_scale), float(k_scale),
              float(v_scale), _ptr(token_keep), float(keep_ratio), _ptr(o["scores"]),
              _ptr(o["kept_index"]), _ptr(o["cu_seqlens"]), _ptr(o.get("qc")), _ptr(o.get("kc")),
              _ptr(o.get("vc")), _ptr(ws), ws.numel() * ws.element_size(), _stream(dev))
    if query_rows is None:
        st = lib.litevlm_token_score_topk(dtype_code(q.dtype), B, S, V_full, Hq, Hkv, D, *common)
        _abi.check(st, "litevlm_token_score_topk")
    else:
        st = lib.litevlm_token_score_topk_rows(dtype_code(q.dtype), B, S, V_full, Hq, Hkv, D,
                                               int(query_rows), *common)
        _abi.check(st, "litevlm_token_score_topk_rows")
    return o


def select_score_topk(view_logit: torch.Tensor, view_offsets: Sequence[int], q: torch.Tensor,
                      k: torch.Tensor, v: Optional[torch.Tensor], keep_ratio: float, V_full: int,
                      w_lexical: float = 0.0, threshold: float = 0.5,
                      view_lexical: Optional[torch.Tensor] = None, softmax_scale: Optional[float] = None,
                      q_scale: float = 1.0, k_scale: float = 1.0, v_scale: float = 1.0, gather: bool = True,
                      token_keep: bool = True, workspace: Optional[torch.Tensor] = None,
                      out: Optional[dict] = None) -> dict:
    """patch_select and token_score_topk in one call (litevlm_select_score_topk):
    the returned dict holds token_score_topk's tensors plus view_keep [B,N],
    n_visual_kept [B] and, when token_keep is set, the token mask [B,S]."""
    lib = load()
    B, S, Hq, D = q.shape
    Hkv = k.shape[2]
    N = view_logit.shape[1]
    dev = q.device
    if softmax_scale is None:
        softmax_scale = 1.0 / math.sqrt(D)
    o = dict(out or {})
    o.setdefault("scores", torch.empty((B, V_full), dtype=torch.float32, device=dev))
    o.setdefault("kept_index", torch.empty((B * S,), dtype=torch.int32, device=dev))
    o.setdefault("cu_seqlens", torch.empty((B + 1,), dtype=torch.int32, device=dev))
    o.setdefault("view_keep", torch.empty((B, N), dtype=torch.uint8, device=dev))
    o.setdefault("n_visual_kept", torch.empty((B,), dtype=torch.int32, device=dev))
    if token_keep:
        o.setdefault("token_keep", torch.empty((B, S), dtype=torch.uint8, device=dev))
    if gather:
        o.setdefault("qc", torch.empty((B * S, Hq, D), dtype=q.dtype, device=dev))
        o.setdefault("kc", torch.empty((B * S, Hkv, D), dtype=k.dtype, device=dev))
        o.setdefault("vc", torch.empty((B * S, Hkv, D), dtype=v.dtype, device=dev))
    nbytes = workspace_bytes(B, S, V_full, Hq, Hkv, D)
    ws = workspace if workspace is not None else o.get("workspace")
    if ws is None:
        ws = torch.empty((max(nbytes, 1),), dtype=torch.uint8, device=dev)
    o["workspace"] = ws
    off = (ctypes.c_int32 * (N + 1))(*[int(x) for x in view_offsets])
    st = lib.litevlm_select_score_topk(
        dtype_code(q.dtype), B, S, V_full, Hq, Hkv, D, N, off, _ptr(view_logit), _ptr(view_lexical),
        float(w_lexical), float(threshold), _ptr(q), _ptr(k), _ptr(v), float(softmax_scale), float(q_scale),
        float(k_scale), float(v_scale), float(keep_ratio), _ptr(o["view_keep"]), _ptr(o.get("token_keep")),
        _ptr(o["n_visual_kept"]), _ptr(o["scores"]), _ptr(o["kept_index"]), _ptr(o["cu_seqlens"]),
        _ptr(o.get("qc")), _ptr(o.get("kc")), _ptr(o.get("vc")), _ptr(ws), ws.numel() * ws.element_size(),
        _stream(dev))
    _abi.check(st, "litevlm_select_score_topk")
    return o


def prefill_attn(qc: torch.Tensor, kc: torch.Tensor, vc: torch.Tensor, cu_seqlens: torch.Tensor,
                 max_seqlen: int, B: Optional[int] = None, causal: bool = True,
                 softmax_scale: Optional[float] = None, q_scale: float = 1.0, k_scale: float = 1.0,
                 v_scale: float = 1.0, out_dtype: Optional[torch.dtype] = None,
                 out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Causal GQA attention over packed sequences. qc: [rows,Hq,D], kc/vc: [rows,Hkv,D]
    with rows >= cu_seqlens[B]. Output [rows,Hq,D] in out_dtype (bf16 by default,
    fp32 for fp32 input); rows past cu_seqlens[B] are left untouched."""
    lib = load()
    rows, Hq, D = qc.shape
    Hkv = kc.shape[1]
    if B is None:
        B = cu_seqlens.numel() - 1
    if softmax_scale is None:
        softmax_scale = 1.0 / math.sqrt(D)
    if out_dtype is None:
        out_dtype = torch.float32 if qc.dtype == torch.float32 else torch.bfloat16
    o = out if out is not None else torch.empty((rows, Hq, D), dtype=out_dtype, device=qc.device)
    st = lib.litevlm_prefill_attn(
        dtype_code(qc.dtype), dtype_code(o.dtype), B, Hq, Hkv, D, _ptr(qc), _ptr(kc), _ptr(vc),
        _ptr(cu_seqlens), int(max_seqlen), float(softmax_scale), float(q_scale), float(k_scale),
        float(v_scale), 1 if causal else 0, _ptr(o), _stream(qc.device))
    _abi.check(st, "litevlm_prefill_attn")
    return o


def decode_workspace_bytes(in_dtype: torch.dtype, B: int, Hq: int, Hkv: int, D: int,
                           max_seqlen: int) -> int:
    return int(load().litevlm_decode_attn_workspace(dtype_code(in_dtype), B, Hq, Hkv, D, int(max_seqlen)))


def decode_attn(q1: torch.Tensor, k1: torch.Tensor, v1: torch.Tensor, kc: torch.Tensor,
                vc: torch.Tensor, cu_seqlens: torch.Tensor, max_seqlen: int,
                softmax_scale: Optional[float] = None, q_scale: float = 1.0, k_scale: float = 1.0,
                v_scale: float = 1.0, out_dtype: Optional[torch.dtype] = None,
                out: Optional[torch.Tensor] = None,
                workspace: Optional[torch.Tensor] = None) -> torch.Tensor:
    """One decode step per sample over the compacted cache. q1: [B,Hq,D], k1/v1:
    [B,Hkv,D] (the new token), kc/vc: [rows,Hkv,D] with rows >= cu_seqlens[B].
    Returns [B,Hq,D] in out_dtype (bf16 by default, fp32 for fp32 input)."""
    lib = load()
    B, Hq, D = q1.shape
    Hkv = k1.shape[1]
    if softmax_scale is None:
        softmax_scale = 1.0 / math.sqrt(D)
    if out_dtype is None:
        out_dtype = torch.float32 if q1.dtype == torch.float32 else torch.bfloat16
    o = out if out is not None else torch.empty((B, Hq, D), dtype=out_dtype, device=q1.device)
    nbytes = decode_workspace_bytes(q1.dtype, B, Hq, Hkv, D, max_seqlen)
    ws = workspace if workspace is not None else torch.empty((max(nbytes, 1),), dtype=torch.uint8,
                                                             device=q1.device)
    st = lib.litevlm_decode_attn(
        dtype_code(q1.dtype), dtype_code(o.dtype), B, Hq, Hkv, D, _ptr(q1), _ptr(k1), _ptr(v1),
        _ptr(kc), _ptr(vc), _ptr(cu_seqlens), int(max_seqlen), float(softmax_scale), float(q_scale),
        float(k_scale), float(v_scale), _ptr(o), _ptr(ws), ws.numel() * ws.element_size(),
        _stream(q1.device))
    _abi.check(st, "litevlm_decode_attn")
    return o


def tsm_fold_gain(w: torch.Tensor, gamma: torch.Tensor, out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """bf16 w [rows, cols] times the fp32 gain gamma [cols] per column, rounded to bf16."""
    rows, cols = w.shape
    o = out if out is not None else torch.empty_like(w)
    st = load().litevlm_tsm_fold_gain(rows, cols, _ptr(w), _ptr(gamma), _ptr(o), _stream(w.device))
    _abi.check(st, "litevlm_tsm_fold_gain")
    return o


def tsm_qk(hidden: torch.Tensor, token_keep: Optional[torch.Tensor], V_full: int, w_q: torch.Tensor,
           w_k: torch.Tensor, Hq: int, Hkv: int, D: int, eps: float = 1e-5, rope_theta: float = 1e6,
           q: Optional[torch.Tensor] = None, k: Optional[torch.Tensor] = None):
    """Scoring queries (text rows) and keys (kept rows) of the Token Selection
    Module from bf16 hidden states [B,S,Dm]; w_q/w_k carry the folded RMS gain.
    Returns (q [B,S,Hq,D], k [B,S,Hkv,D]) in bf16; q's visual rows and the key
    rows of dropped tokens are untouched."""
    B, S, Dm = hidden.shape
    dev = hidden.device
    q = q if q is not None else torch.empty((B, S, Hq, D), dtype=torch.bfloat16, device=dev)
    k = k if k is not None else torch.empty((B, S, Hkv, D), dtype=torch.bfloat16, device=dev)
    st = load().litevlm_tsm_qk(B, S, V_full, Dm, Hq, Hkv, D, _ptr(hidden), _ptr(token_keep), _ptr(w_q),
                               _ptr(w_k), float(eps), float(rope_theta), _ptr(q), _ptr(k), _stream(dev))
    _abi.check(st, "litevlm_tsm_qk")
    return q, k


def gather_hidden(hidden: torch.Tensor, kept_index: torch.Tensor, cu_seqlens: torch.Tensor,
                  out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """Packed copies of the kept rows of hidden [B,S,...] (rows cu_seqlens[b].. of the
    result for sample b): out [B*S, ...] with rows past cu_seqlens[B] untouched."""
    B, S = hidden.shape[0], hidden.shape[1]
    row_bytes = hidden[0, 0].numel() * hidden.element_size()
    o = out if out is not None else torch.empty((B * S,) + tuple(hidden.shape[2:]), dtype=hidden.dtype,
                                                device=hidden.device)
    st = load().litevlm_gather_hidden(B, S, row_bytes, _ptr(hidden), _ptr(kept_index), _ptr(cu_seqlens),
                                      _ptr(o), _stream(hidden.device))
    _abi.check(st, "litevlm_gather_hidden")
    return o


def psm_forward(emb: torch.Tensor, params: torch.Tensor, n_heads: int, d_ff: int, n_views: int,
                n_layers: int, out: Optional[torch.Tensor] = None,
                workspace: Optional[torch.Tensor] = None) -> torch.Tensor:
    """View logits [B, n_views] fp32 from fp32 token embeddings [B, T, d] and the
    flat fp32 parameter vector (order documented in include/litevlm.h)."""
    lib = load()
    B, T, d = emb.shape
    dev = emb.device
    o = out if out is not None else torch.empty((B, n_views), dtype=torch.float32, device=dev)
    if workspace is None:
        nbytes = int(lib.litevlm_psm_workspace(B, T, d, n_heads, d_ff))
        workspace = torch.empty((max(nbytes, 1),), dtype=torch.uint8, device=dev)
    st = lib.litevlm_psm_forward(B, T, d, n_heads, d_ff, n_views, n_layers, _ptr(emb), _ptr(params),
                                 params.numel(), _ptr(o), _ptr(workspace),
                                 workspace.numel() * workspace.element_size(), _stream(dev))
    _abi.check(st, "litevlm_psm_forward")
    return o
