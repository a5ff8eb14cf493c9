"""HeteroFold transfer-time path for AMD MI355X (gfx950).

* ``heterofold`` -- Python binding of the C ABI in ``include/heterofold.h``
  (``hf_build_alignment``, ``hf_build_layer_map``, ``hf_pack_maps``,
  ``hf_transfer_kv`` and helpers), backed by ``libheterofold.so``.
* ``synth``      -- seeded synthetic workloads.
* ``build``      -- builds ``libheterofold.so`` in-tree.

Importing the package loads nothing; the library is loaded on first call.
"""

__all__ = ["heterofold", "synth", "build"]
