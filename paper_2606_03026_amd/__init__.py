"""MI355X-native spike-gated INT8 projection.

The compute path is the HIP library libspike_proj.so (C ABI in
include/spike_proj.h); `_binding` wraps its entry points under the same
names.  `workloads` draws the seeded synthetic inputs.
"""
__all__ = ["workloads", "build"]
