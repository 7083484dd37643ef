"""MI355X-native H2O chunk step: SDPA over [KV cache || chunk] with summed
attention weights, H2O score accumulation, bottom-k eviction and K/V insert.

The compute path is the HIP library ``libh2o.so`` (sources in ``csrc/``,
C ABI in ``include/h2o.h``); ``h2o`` is its thin ctypes binding. Importing this
package does not load the library; the first call into ``h2o`` does, and it
raises if the library is missing.
"""
__all__ = ["h2o", "workloads"]
