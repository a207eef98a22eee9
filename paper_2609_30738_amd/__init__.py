"""MI355X-native diversity-aware, layer-wise KV-cache eviction scoring.

The computation lives in libkvevict.so (hand-written gfx950 HIP kernels behind the C ABI declared
in include/kvevict.h).  `_lib` is its ctypes binding, `api` the device plumbing that runs a whole
pass, `workloads` the seeded synthetic inputs.  Importing the package loads nothing; the library is
opened on first use and its absence is an error.
"""

__all__ = ["_lib", "api", "workloads", "build"]
