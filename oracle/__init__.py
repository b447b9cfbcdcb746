"""fp64 CPU oracle for owner-local paged MLA decode attention.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the CPU
baseline leg of the benchmark may import this package.  The library and its
Python binding never call it, and it shares no code with them: it decodes the
storage formats from their definitions, walks the block table itself and
evaluates softmax attention directly in float64 with numpy.

What it computes (the owner's attention step): each owner attends all H query
heads of its own query rows over the complete causal prefix of each request's
history, with one head-shared latent row per token serving as key
(``[latent | rope]``, width d_c + d_r) and, through its first d_c entries, as
value (Sec. 3 "DOP: Computation"; Sec. 3 "Cost", d_q = d_c + d_r, d_z = d_c;
Sec. 1 on MLA keeping one head-shared latent per token).  ``s`` counts the
current chunk, ``1 <= q <= s`` (App. B), and every query reads its complete
causal prefix (Sec. 4.1 "Handoff").

Parity pins: every function here is checked by the CPU tests against values
that do not come from this package (brute force on dense un-paged inputs,
torch's float64 scaled-dot-product attention, closed forms, invariants, a
hand-worked example, and the format definitions cross-checked with numpy and
torch dtypes).
"""
from . import dop
from .formats import DS_ROW_BYTES, bf16_bits_to_f64, ds_rows_to_f64, e4m3_bits_to_f64
from .mla import (gather_history, mla_attention, mla_attention_sampled,
                  merge_partials, attention_rows, gather_positions, mla_attention_topk)

__all__ = ["dop", "bf16_bits_to_f64", "e4m3_bits_to_f64", "ds_rows_to_f64", "DS_ROW_BYTES", "gather_history", "gather_positions",
           "mla_attention_topk",
           "mla_attention", "mla_attention_sampled", "merge_partials",
           "attention_rows"]
