"""CPU oracle for prefix-cached paged extend attention -- TEST INFRASTRUCTURE.

This package is the plain, slow reference that the GPU library is checked
against.  It is test infrastructure only: the test suite, the smoke check and
the benchmark's CPU-baseline leg may import it; the library and its Python
binding never do, and this package imports nothing from them.  It has its own
bf16/fp8 decoding, its own page gather and scatter, and computes attention in
float64 by its plain definition.

What it computes (the paper, CacheWise, states the premise: Sec. 2 persists
KV prefixes in fixed-size blocks that later requests extending the same prefix
reuse; Sec. 3 observes that every agent turn reuses and extends a growing
prefix; Sec. 6.1 serves GQA models with chunked prefill).  The attention itself
is not written in the paper; the oracle takes the standard definition of
causal softmax attention with the readings listed in the design notes:

* suffix row i of sequence b sits at absolute position Lp_b + i and sees keys
  0 .. Lp_b + i (bottom-right causal alignment);
* query head h uses kv head h // G;
* keys < Lp_b come from the page pool through the block table, keys >= Lp_b
  from the new K/V inputs.

Modules
  codecs           bf16 and OCP fp8-e4m3fn decoding/encoding from their definitions
  paged_attention  page gather/scatter, row-wise and blocked attention
  page_swap        whole-page copies between the page pool and a host block pool
                   (the offloading configuration of Sec. 6.4)
  cachewise_policy the KV-block policy (prefix-aware dispatch, predictive / LRU /
                   Belady eviction) simulated plainly over agent sessions
"""
from .codecs import bf16_bits_to_f64, e4m3fn_decode, e4m3fn_encode_rne  # noqa: F401
from .paged_attention import (  # noqa: F401
    PagedInputs,
    decode_attention,
    extend_attention_blocked,
    extend_attention_rows,
    extend_attention_rowwise,
    extend_attention_token_blocks,
    gather_sequence_kv,
    write_pages,
)
from .page_swap import swap_in, swap_out  # noqa: F401
from . import cachewise_policy  # noqa: F401

PARITY_UNPINNED = ()  # every function above has at least one independent pin
