"""CPU oracle for the LiteVLM select + prefill path.

TEST INFRASTRUCTURE ONLY. A plain, slow, float64 NumPy implementation of what
the path computes, written from the paper's definitions. Only ``tests/``,
``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` may
import it; the product path (the HIP library and its Python binding) never
does, and shares no code with it.

Every function here is pinned by ``-m "not gpu"`` tests against values the
paper fixes (Table 1 token counts), closed forms, invariants, library routines
and brute force. No function is "parity unpinned".
"""
from .litevlm import (  # noqa: F401
    decode_inputs,
    view_scores,
    patch_select,
    token_keep_from_views,
    patch_selected_positions,
    token_scores,
    keep_count,
    select_topk,
    compact,
    gather_rows,
    prefill_attention,
    decode_attention,
    run_path,
)
from . import tsm  # noqa: F401,E402  (the Token Selection Module front end)
from . import psm  # noqa: F401,E402  (the Patch Selection Module forward pass)
