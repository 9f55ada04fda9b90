"""Oracle for the step-pruned video-DiT denoise step.

TEST INFRASTRUCTURE.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this package.  The product path
(the HIP library and its Python binding) never imports, calls or links it,
and this package imports nothing from the product path.

It is a plain, slow, obviously-correct numpy forward, in float64 unless the
caller asks for float32, of exactly what the GPU path computes: the dense
DiT block stack with the keep masks applied by zeroing the pruned rows and
columns of dense weights (the paper's gating equation, Sec. 3.2, exported to
a dense network).  See oracle/dit.py for the per-function citations and the
readings taken where the paper is silent.
"""
from .dit import (  # noqa: F401
    sinusoid, silu, gelu_tanh, layer_norm, rms_norm, rope_split, rope_angles,
    apply_rope, softmax_rows, attention, apply_keep, time_embedding, block,
    step, euler, denoise, sigmas, predict_clean, renoise, rollout,
)
from .gates import hard_gates, ffn_channel_norms, ffn_reorder  # noqa: F401
