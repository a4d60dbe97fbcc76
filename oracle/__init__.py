"""CPU oracle for the LegoLink link step (EPIC, arXiv 2410.15332).

TEST INFRASTRUCTURE ONLY.  Nothing in the product path imports, calls or links
this package: only the tests, the smoke check and the benchmark's CPU-baseline
leg use it.  It shares no code with the GPU library; the only shared module is
``synth`` (seeded random inputs, no link-step arithmetic).

Everything is plain NumPy in float64.  Library matmuls serve as steps; there is
no blocking or fusion beyond processing independent query rows in groups.

Contents
  link.py   -- token selection (Sec. 4.2), KV expansion (Sec. 4.2, third step),
               masked attention (Eq. 1), attention-level link step, decode
               after it (new tokens over the linked sequence), the rotary
               embedding and the cached-K re-rotation variant.
  model.py  -- Llama-style decoder layer for the selected rows, the compile step
               (Sec. 2.2), the full-model link step, and the layer's row-set
               projections on their own.

Pins (tests/test_oracle_pins.py) tie each function to something other than
itself: library causal attention (FR = full prefill, Sec. 2.3), the Naive
special case (k = 0), closed forms (one-hot and constant V, zero queries,
position 0), a worked selection example, the HuggingFace Llama forward, and
brute-force sums for the projections.
"""
from .link import (  # noqa: F401
    chunk_offsets,
    legolink_positions,
    expand_kv,
    masked_attention,
    link_attention,
    decode_attention,
    rerotate_cached,
)
from .model import (  # noqa: F401
    projection,
    rmsnorm,
    rope,
    compile_chunk,
    decoder_layer,
    link_model,
)
