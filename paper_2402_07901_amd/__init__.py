"""MI355X-native Fastmax attention (arXiv 2402.07901) behind a C ABI.

The compute path is the HIP library ``libfastmax.so`` (built by
``paper_2402_07901_amd.build``); ``paper_2402_07901_amd.fastmax`` is its thin
ctypes binding.  ``inputs`` holds the seeded synthetic workloads.
"""
__all__ = ["fastmax", "inputs", "build"]
