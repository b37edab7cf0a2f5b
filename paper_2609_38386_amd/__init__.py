"""MI355X-native hot path of Decode-Latency Feedback Prefill (DLFP).

* ``dlfp``     -- Python binding of libdlfp (C ABI in ``include/dlfp.h``).
* ``runtime``  -- device KV pools, per-iteration batches and workspace.
* ``workload`` -- seeded synthetic inputs (no method arithmetic).
* ``replay``   -- closed-loop continuous-batching replay driven by the controller.
* ``build``    -- compiles ``libdlfp.so`` for gfx950.

Submodules are imported on demand so that the input generator works without
the compiled library.
"""

__all__ = ["dlfp", "runtime", "workload", "replay", "build"]
