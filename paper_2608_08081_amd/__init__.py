"""IsoQuant compressed-space decode attention for AMD Instinct MI355X.

* ``paper_2608_08081_amd.api``   - PyTorch binding of the C ABI
  (include/isoquant.h): iq_make_rotation, iq_compress_kv, iq_append_token,
  iq_decode_attention, iq_decode_step, ...
* ``paper_2608_08081_amd.synth`` - seeded synthetic workloads.
* ``paper_2608_08081_amd.build`` - builds libisoquant.so for gfx950.

Submodules are imported explicitly so that importing the package does not
load torch or the shared library.
"""
