"""MI355X (gfx950) token-tree verification for LLMCad-style generate-then-verify
decoding (arXiv 2309.04255, §3.2).

The compute lives in libllmcad.so (hand-written HIP, C ABI in include/llmcad.h);
`binding` is its ctypes binding.  Build with `python -m paper_2309_04255_amd.build`.
"""

import os

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libllmcad.so")


def load():
    """Import and return the binding module (raises ImportError if the library is not built)."""
    from . import binding

    return binding
