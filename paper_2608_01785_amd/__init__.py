"""MI355X (gfx950) shared-stage hot path: HIP kernels behind a C ABI.

Submodules are imported on demand:

* ``workloads`` - seeded synthetic inputs (no layer arithmetic).
* ``binding``   - ctypes binding of ``libhorizon.so`` (argument marshalling only).
* ``build``     - compiles the HIP library for gfx950.
"""
