"""GIST sub-GCN training step on AMD MI355X (gfx950).

The compute lives in ``libgist.so`` (hand-written HIP kernels behind the C ABI
of ``include/gist.h``).  ``paper_2102_10424_amd.gist`` is the ctypes binding
(same names as the ABI); ``paper_2102_10424_amd.step`` sequences those calls
into a sub-GCN step and a GIST round.  Importing either module without a
built library raises ImportError -- there is no fallback implementation.
"""

__all__ = ["gist", "step", "build"]
