"""Oracle: a plain, slow, obviously correct CPU implementation of the Winograd
convolution layer, used only as test infrastructure.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import anything here.  The HIP product path never imports this
package and shares no code, header, table or constant generator with it.

* :mod:`oracle.direct` -- fp64 direct 3x3 stride-1 correlation (the definition
  that Eq. 1 reaches exactly), built from ``direct_conv.c``.
* :mod:`oracle.cooktoom` -- exact rational Cook-Toom matrices derived from their
  interpolation points, Eq. 1 / Listing 1 evaluated over the rationals, and fp64
  references of each stage (filter, input and output transform, the per-position
  GEMMs) in the paper's order.
* :mod:`oracle.nn` -- fp64 ReLU and 2x2 max-pool for layer stacks.
"""
