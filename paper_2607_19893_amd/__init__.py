"""MI355X-native (gfx950) 3D Gaussian Splatting training-view hot path.

Submodules:
  gsmi      ctypes binding of libgsmi (include/gsmi.h), same names as the C ABI
  pipeline  ViewTrainer: device buffers of one primitive pool + phase-ordered calls
  scenes    seeded synthetic workloads (inputs only)
  build     in-tree hipcc build of libgsmi.so for gfx950

Importing the package itself loads nothing; importing `gsmi` or `pipeline`
loads libgsmi.so and raises if it has not been built.
"""
