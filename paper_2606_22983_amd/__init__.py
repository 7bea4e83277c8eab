"""MI355X-native paged-KV attention and KV-block restore/stash for LiveServe-style
interactive multi-turn serving (arXiv 2606.22983).

Submodules are imported lazily so that the seeded workload generators
(:mod:`paper_2606_22983_amd.workloads`) stay importable without the HIP library:

* :mod:`paper_2606_22983_amd.kv`        — the Python binding of the C-ABI library
  (``kv_pool_create``, ``paged_attn_decode``, ``paged_attn_prefill``,
  ``kv_blocks_restore``, ``kv_blocks_stash``).  Importing it loads
  ``libliveserve_kv.so`` and raises if the library has not been built.
* :mod:`paper_2606_22983_amd.workloads` — seeded synthetic sessions (inputs only).
* :mod:`paper_2606_22983_amd.build`     — compiles the HIP library for gfx950.
"""
__all__ = ["kv", "workloads", "build"]
