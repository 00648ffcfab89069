"""MI355X-native trace pipeline of Chopper (arXiv 2512.08242).

align -> attribute -> overlap -> aggregate (+ derived ratios and the
re-keyed views with their medians) over per-kernel
records of a multi-GPU training run, in hand-written HIP for gfx950 behind the
C ABI of include/chopper.h.  This package holds the HIP sources (csrc/), the
build step (build.py) and the ctypes binding (binding.py).
"""
from .binding import (DeviceTrace, Pipeline, RowsBuffer, Views, Filter,
                      make_filter,
                      kernel_names, time_kernel, lib, LIB_PATH, NONE,
                      LEVEL_GPU, LEVEL_WORKLOAD, LEVEL_ALL, ST_BAD_GPU,
                      ST_BAD_CLASS, ST_NEG_DURATION, ST_MARKER_OVERLAP,
                      ST_RANGE, ST_ROWS_OVERFLOW, ST_BAD_LEVEL,
                      ST_PATH_CONFLICT)

__all__ = ["DeviceTrace", "Pipeline", "RowsBuffer", "Views", "Filter",
           "make_filter",
           "kernel_names", "time_kernel", "lib", "LIB_PATH", "NONE",
           "LEVEL_GPU", "LEVEL_WORKLOAD", "LEVEL_ALL"]
