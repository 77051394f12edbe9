"""fp64 CPU oracle of Attuner suffix prefill over a frozen artifact cache.

TEST INFRASTRUCTURE, NOT PART OF THE PRODUCT.  Only the test suite, the smoke
check and the benchmark's CPU-baseline leg may import or call anything in this
package.  It shares no code with the HIP path and imports nothing from it; its
only inputs are the seeded draws of :mod:`synthdata` (bf16 bit patterns, decoded
here exactly) and plain integers.

Every function is the paper's definition written out in float64, step by step,
with no blocking, fusion or reordering beyond what the definition states.
"""

from .attuner_ref import (  # noqa: F401
    decode_bf16,
    page_valid_counts,
    block_table,
    assemble,
    qproj_lora,
    rms_norm_heads,
    rope,
    attention,
    attention_probs,
    suffix_layer,
    full_prefill,
    silu,
    linear,
    swiglu,
    decoder_layer,
    first_token,
    interleaved_layer,
    block_table_segments,
    merge_lora,
)
