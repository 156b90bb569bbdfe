"""MI355X-native hot path of the Advanced Model Server image-embedding step.

The compute lives in ``libams.so`` (hand-written HIP for gfx950, C ABI declared
in ``include/ams.h``); ``paper_1711_06505_amd.ams`` is the thin ctypes binding
and ``paper_1711_06505_amd.synth`` draws seeded synthetic inputs.  Importing the
package itself loads nothing.
"""
__version__ = "0.1.0"
