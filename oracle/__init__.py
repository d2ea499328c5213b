"""CPU oracle for one decoder-layer step over a paged-KV token batch.

TEST INFRASTRUCTURE ONLY.  This package is the slow, plain reference that the
HIP path is checked against.  Only the test-suite, the package smoke check and
the benchmark's CPU-baseline leg may import it; the product path never does.
It shares no code with the HIP path and imports nothing from it.
"""
from .layer import (  # noqa: F401
    bf16_bits_to_f32,
    f32_to_bf16_bits,
    rmsnorm,
    rope,
    silu,
    gather_positions,
    attend_one,
    paged_attention_row,
    layer_step,
    stack_step,
    prepare_weights,
    LayerCfg,
)
from . import fp8  # noqa: F401,E402  (E4M3 cache codes)
from . import moe  # noqa: F401,E402  (mixture-of-experts block)
