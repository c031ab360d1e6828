"""fp64 CPU oracle for chunk-streamed speculative-verification attention.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports, links or
calls this package: only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` use it.  It shares no code with the HIP
library (no kernels, headers, helpers or tables); both sides only read the
same seeded inputs.

Contents
--------
``attention.verify_attention``
    The definition the method reaches (Sec. 4.2, Eq. 12 with the causal
    candidate mask; Eq. 17 states that the chunked reduction equals it in
    real arithmetic): masked softmax attention of each candidate query over
    the committed history plus the visible candidates, in float64.
``attention.verify_attention_chunked``
    The paper's own procedure (Sec. 4.2, Eq. 13 chunk-local state, Eq. 14
    merge, initial state (-inf, 0, 0), GPU-resident masked pass, O = a/l),
    over any partition and order of the history; used for the invariance
    claims.
``bruteforce.verify_attention_decimal``
    The same definition written out element by element in 50-digit decimal
    arithmetic, for tiny inputs.

Pins (see ``tests/test_oracle_*.py``): decimal brute force, torch's
``scaled_dot_product_attention`` in float64 (a library routine that gives
masked GQA softmax attention), chunk count/order invariance, single-token
decode at k = 0, mask invariance, weight normalisation, closed forms and
hand-derived golden cases, plus planted-mistake tests showing each pin
catches a plausible error.
"""
from .attention import (  # noqa: F401
    bf16_bits_to_f64,
    candidate_visible,
    kv_head_of,
    verify_attention,
    verify_attention_chunked,
    attend_heads,
)
from .bruteforce import verify_attention_decimal  # noqa: F401
