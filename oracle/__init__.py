"""Plain, slow, fp64 CPU oracle for the action-expert per-tick forward.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  The product path
(the HIP library and its Python binding) never imports, calls or links it, and
this package imports nothing from the product path.

What it computes (the expert of Sec. 3.1, "Action Expert with Per-Layer Cache
Attention", run once per control tick as in Sec. 3.3):

* ``expert.py``  -- RMSNorm, rotary encoding, the joint attention of Eq. (1)
  over [cached backbone K/V ; the expert's own K/V], the output projection, the
  SwiGLU block, the mean-pool + linear waypoint head, and the paper's
  two-layer head over the waypoint-query tokens; the staleness-augmented training
  form (Sec. 3.2): every frame's expert block of a clip in one forward, one
  attention over the whole clip with per-block masks.
* ``backbone.py`` -- the backbone's incremental forward (Sec. 3.3): the n new
  tokens of a frame through LLaMA decoder layers over the cache, giving the
  rows to append.
* ``fp8.py``     -- decoding of OCP FP8 E4M3 (e4m3fn) codes (the diagnostic
  reference for the fp8-stored cache) and their encoding against a scale
  (the reference of the quantising append).

Every function is the plain definition evaluated in float64 on the exact values
the GPU receives (inputs are rounded to the stored dtype first, then upcast).
Readings of points the paper leaves open are listed at the top of each module.
Parity status: every function is pinned by the ``-m "not gpu"`` tests in
``tests/test_oracle_pins.py``; no function is "parity unpinned" except the
end-to-end composition, which has no printed worked example in the paper and is
pinned only through its pinned parts and invariants (see those tests).
"""

from .expert import (  # noqa: F401
    ExpertShape,
    rmsnorm,
    rope_cos_sin,
    apply_rope,
    joint_attention,
    swiglu_ffn,
    expert_layer,
    waypoint_head,
    gelu,
    query_head,
    apply_head,
    expert_forward,
    staleness_visible_rows,
    masked_multiblock_forward,
)
from .fp8 import e4m3fn_decode, e4m3fn_encode  # noqa: F401
from .backbone import (  # noqa: F401
    BackboneShape,
    causal_cache_attention,
    backbone_layer,
    backbone_incremental_forward,
)
