"""MI355X (gfx950) attention hot path of a prefill/decode-disaggregated LLM server.

The compute lives in ``libdopd_attn.so`` (hand-written HIP kernels behind a
C ABI, declared in ``include/dopd_attn.h``).  ``paper_2511_20982_amd.attn``
is a thin ctypes binding with the same entry-point names; it loads the
library on first use and raises if it is missing.  ``inputs`` draws the
seeded synthetic workloads.
"""
__all__ = ["attn", "inputs"]
