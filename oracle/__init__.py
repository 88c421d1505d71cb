"""CPU oracle for the Thinker decoder layer.

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, by the smoke check and by the
bench's CPU-baseline leg, never by the HIP product path.  It shares no code
with the HIP path; both receive their inputs from the seeded generators in
``synth``.

* ``oracle.layer`` -- the plain vectorised definition (float64 by default,
  float32 on request).
* ``oracle.brute`` -- a naive scalar float64 brute force for tiny shapes that
  pins ``oracle.layer``.
"""
from .layer import (attention, kvcache_append, layer_forward, moe_ffn, moe_route, project, rmsnorm,
                    rope, rope_angles, rope_angles_sections, round_bf16, silu, softmax, swiglu, topk_lower_index)
from .brute import layer_brute

__all__ = ["attention", "kvcache_append", "layer_forward", "moe_ffn", "moe_route", "project", "rmsnorm",
           "rope", "rope_angles", "rope_angles_sections", "round_bf16", "silu", "softmax", "swiglu", "topk_lower_index", "layer_brute"]
