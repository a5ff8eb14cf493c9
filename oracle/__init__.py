"""Plain fp64 CPU oracle of the HeteroFold transfer-time path.

This package is TEST INFRASTRUCTURE.  Only the test-suite, the smoke check in
``__graft_entry__.smoke`` and the ``cpu_baseline`` leg of ``bench.py`` may
import or execute it.  The product path (the HIP library and its Python
binding) never calls into it, and it shares no code with that path.

Everything here is written to be checked against the paper by eye:

* ``alignment``  -- Token Alignment (Sec. 3.1 "Token Alignment"; App. B.1) and
  the overlap-weighted span alignment, both as a CSR span table.
* ``layer_map``  -- two-nearest-layer linear interpolation of sender layers for
  each receiver layer, and the paper's proportional-depth neighbourhood (Eq. 1).
* ``rope``       -- rotate-half rotary position embedding, rotation and
  un-rotation in fp64.
* ``transfer``   -- the folded affine K/V map of Eq. 9 applied to the aligned,
  layer-interpolated sender cache, with RoPE un-rotation of post-RoPE sender
  keys and re-rotation at receiver positions.
* ``recolor``    -- the offline construction of those maps: sender RMS (Eq. 3),
  weighted moments, whitening + Procrustes (Eq. 4), Recolor (Eq. 5), and the
  low-rank correction folded into the map (Eq. 9).

Integer results are exact.  Floating-point results are fp64 computed from the
exact stored input values (bf16 or fp32 widened to fp64).
"""

from . import alignment, layer_map, recolor, rope, transfer  # noqa: F401
