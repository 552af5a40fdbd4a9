"""CPU oracle (test infrastructure only).

Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may
import this package. It imports nothing from the product package and the
product never imports it.
"""
from .attention import (  # noqa: F401
    bf16_bits_to_f64,
    kv_views,
    decode,
    merge,
    decode_split,
    gather_rows,
    mla_absorb_query,
    mla_explicit,
)
from . import planner  # noqa: F401,E402
