"""MI355X-native hot path of parallel NeRF inversion for pose estimation.

`synth` draws seeded synthetic workloads; `pnerf` binds the HIP library
(libpnerf.so, C ABI declared in include/pnerf.h).
"""
