"""Plain fp64 CPU oracle for the low-bit substitute-layer linear (SubSpec, Sec. 4.1)
and for the draft-tree expansion step with probability sharpening (Sec. 4.2, App. D)
and the draft model's tree attention over the shared KV cache (Sec. 4.1), and for the
quantizer with an HQQ-style optimised zero-point (Sec. 4.1, Sec. 5.1).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or call anything in this package.
The product path (``paper_2509_18344_amd``) never imports it, and this package
imports nothing from the product: it is written from the paper's definition of a
substitute layer and from the packed-layout specification in ``include/subspec.h``.

Every function is slow and obviously correct on purpose: NumPy in float64, no
blocking, fusion or reordering beyond what the definition states.
"""
from .qlinear import (  # noqa: F401
    fp16_round,
    bf16_round_bits,
    bf16_bits_to_f64,
    quantize_minmax,
    dequant,
    dequant_f32,
    dequant_bf16_bits,
    unpack,
    qlinear_ref,
    qlinear_ref_cols,
)
from .tree import (  # noqa: F401
    log_softmax_rows,
    expand_scores,
    tree_expand,
    kth_gap,
)
from .tree_attn import (  # noqa: F401
    append_kv,
    tree_attention,
    weighted_abs_v,
)
from .hqq import (  # noqa: F401
    quantize_hqq,
)
