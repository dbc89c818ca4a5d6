"""CPU oracle for the per-hit classifier (test infrastructure only).

Only ``tests/``, ``__graft_entry__.smoke()`` and ``bench.py``'s
``cpu_baseline`` leg may import this package; the HIP product path never does.
"""

from .pointid_oracle import *  # noqa: F401,F403
from .pointid_oracle import (  # noqa: F401
    gather_patches, gather_patches_planes, to_bf16_rne, bf16_bits, conv_relu,
    flatten_hwc, dense_relu, softmax, sigmoid, heads, forward, logits,
    classify_patches, classify, classify_planes, quantize_bf16_model,
    forward_bf16_emulated,
)
