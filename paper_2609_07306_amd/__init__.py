"""MI355X-native route-maintenance hot path of RouteRelay (arXiv 2609.07306).

Modules:
  ``routerelay`` -- the ctypes binding of ``librouterelay.so`` (the C ABI
                    declared in ``include/routerelay.h``); importing it loads
                    the library and fails loudly if it is not built.
  ``synth``      -- seeded synthetic chunk representations (inputs only).
  ``build``      -- compiles the HIP library for gfx950.
"""
__version__ = "0.1.0"
