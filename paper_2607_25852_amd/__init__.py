"""MI355X-native draft-verify round: verify attention, speculative acceptance and
D-cut budget allocation as hand-written gfx950 HIP kernels behind the C ABI of
libspecverify (declared in include/specverify.h).

Submodules:
  binding -- ctypes binding of libspecverify (loads the built library lazily and
             fails loudly if it is missing)
  synth   -- seeded synthetic inputs (drafter, target model, scheduler stand-ins)
  build   -- builds libspecverify.so for gfx950 with hipcc
"""
__all__ = ["binding", "synth", "build"]
