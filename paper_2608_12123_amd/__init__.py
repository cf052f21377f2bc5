"""MI355X-native batched ready-cohort control transition.

``rc_cohort``  -- binding of the HIP library (librc_cohort.so, C ABI in
                  include/rc_cohort.h); every step runs in hand-written gfx950
                  kernels, with no CPU fallback.
``workload``   -- seeded synthetic inputs of the benchmark workloads.
``build``      -- in-tree hipcc build of the library.
"""
