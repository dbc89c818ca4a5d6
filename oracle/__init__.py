"""CPU oracle for the per-hit classifier (test infrastructure only).

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s
``cpu_baseline`` leg may import this package; the HIP product path never does.
"""

from .pointid_oracle import *  # noqa: F401,F403
from .pointid_oracle import (  # noqa: F401
    gather_patches, gather_patches_planes, to_bf16_rne, bf16_bits, conv_relu,
    flatten_hwc, dense_relu, softmax, sigmoid, heads, forward, logits,
    classify_patches, classify, classify_planes, to_fp16_rne, fp16_bits, round16,
    quantize_16bit_model, forward_16bit_emulated, forward_bf16_emulated,
    classify_16bit_emulated,
)
