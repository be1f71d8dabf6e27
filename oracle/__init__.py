"""Plain fp64 CPU oracle for Intermittent Semi-working Mask (ISM) attention.

TEST INFRASTRUCTURE ONLY. Nothing on the product path may import, call or
execute anything in this package: only the test suite, the smoke check of the
entry-point module and the CPU-baseline leg of the benchmark do. It shares no
code with the HIP library or its Python binding, and imports neither.

Every function here is written from the paper (arXiv 2408.00539,
"Intermittent Semi-working Mask: A New Masking Paradigm for LLMs"):
the visibility bound f(j) of Eq. 5, the masked attention update of Eq. 4 in
its softmax form (Sec. 2.3, on integrating the mask), the KV-cache reuse
procedure of Sec. 2.3, and ChatGLM-style 2-D rotary positions (the
prefix-backbone adaptation of Sec. 2.3, module ``rope2d``).
"""

from .ism_oracle import (  # noqa: F401
    lim,
    seq_index,
    mask_dense,
    mask_eq5,
    fwd,
    fwd_rows,
    bwd,
    prefill_cached,
    decode_step,
    brute_force_fwd,
    visible_pairs,
    seer,
    uniform_fwd,
    uniform_bwd,
)
from .rope2d import positions_2d, rope2d  # noqa: F401,E402
