"""CPU fp64 oracle of the video-attention hot path -- TEST INFRASTRUCTURE ONLY.

This package is the plain, slow, obviously-correct definition of what the HIP
path computes: 3D rotary position embedding of query/key tokens over their
(time, height, width) latent coordinates, followed by non-causal scaled
dot-product attention with a per-batch valid-key prefix.  The paper (Section 2,
"3D RoPE, 3D VAEs, and flash attention") dispatches this to flash-attention
kernels, which reorganise the same exact computation so that the query-key
score matrix is never materialised; the oracle therefore is the definition
itself, evaluated in float64 with a two-pass (max, then exp/sum) softmax.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  It shares no code with the HIP path:
the only common code is the seeded input generator, which holds none of the
method's arithmetic.

``qk_norm_ref`` is the query/key prologue that precedes the rotation in the
served models (per-head RMS normalisation with a learned gain);
``attn_bwd_ref`` is the gradient of the attention (for post-training),
``rope_transpose_ref`` carries a gradient back through the rotation, and
``na3d_ref`` is the 3D neighbourhood (windowed) attention of a VAE decoder,
and ``qkv_proj_ref`` the Q/K/V projection followed by the Q/K prologue.
"""

from .bf16 import bf16_bits_to_f64, f64_to_bf16_bits
from .rope3d import RopeSpec, rope3d_ref, rope_angles
from .attention import attn_ref, attn_ref_rows
from .qknorm import qk_norm_ref
from .attention_bwd import attn_bwd_ref, attn_bwd_ref_rows, rope_transpose_ref
from .na3d import na3d_ref
from .qkv import qkv_proj_ref

__all__ = [
    "bf16_bits_to_f64",
    "f64_to_bf16_bits",
    "RopeSpec",
    "rope3d_ref",
    "rope_angles",
    "attn_ref",
    "attn_ref_rows",
    "qk_norm_ref",
    "attn_bwd_ref",
    "attn_bwd_ref_rows",
    "rope_transpose_ref",
    "na3d_ref",
    "qkv_proj_ref",
]
