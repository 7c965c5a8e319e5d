"""CateKV hybrid-KV decode path for MI355X (gfx950).

The compute lives in ``libcatekv.so`` (HIP kernels behind the C ABI of
``include/catekv.h``); this package is its Python binding.
"""
from ._lib import CateKVError, LIB_PATH, lib  # noqa: F401
from .binding import (  # noqa: F401
    DecodePlan,
    adaptive_budget,
    append_kv,
    classify_heads,
    compact_kv,
    decode_attn,
    decode_plan,
    decode_workspace,
    kv_table,
    page_bounds,
    retrieve_pages,
    score_heads,
    score_heads_workspace,
    select_critical,
    select_workspace,
    workspace,
)
