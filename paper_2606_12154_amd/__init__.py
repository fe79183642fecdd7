"""MI355X (gfx950) runtime for the mouth model of the Horsehair runtime path:
prompt prefill and greedy decode of a Llama-style decoder against a paged KV
cache, in hand-written HIP kernels behind the C ABI of include/hh.h.

``paper_2606_12154_amd.hh`` is the ctypes binding; ``build.py`` compiles
``csrc/`` into ``libhh.so``.
"""
from . import hh  # noqa: F401
