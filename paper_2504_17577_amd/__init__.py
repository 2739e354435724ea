"""MI355X-native fused attention forward (libtileattn) and its Python binding.

  paper_2504_17577_amd.tileattn  binding of the C ABI in include/tileattn.h
  paper_2504_17577_amd.gen       seeded bf16 inputs shared by tests and bench
  paper_2504_17577_amd.build     hipcc build of libtileattn.so for gfx950
"""
