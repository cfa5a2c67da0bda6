"""SMetric request -> KV-holder matching and routing on MI355X (gfx950).

The compute path lives in the HIP library ``libsmetric.so`` (C ABI, ``include/smetric.h``);
``paper_2607_08565_amd.smetric`` is its thin ctypes binding.  ``workload`` draws the
seeded synthetic inputs.  Importing the package does not load the library.
"""
