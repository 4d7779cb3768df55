"""Fine-grained ViT encoder-layer kernels for MI355X (gfx950).

The encoder layer's forward and backward are a chain of separately
launchable HIP kernels behind the C ABI in include/optimus_enc.h, so that a
scheduler can place each kernel into a short idle period of an LLM pipeline
(Optimus, arXiv 2408.03505).  `binding` is the ctypes binding; `build`
compiles the library in-tree.
"""

from . import binding  # noqa: F401
from .binding import EncError  # noqa: F401

__all__ = ["binding", "EncError"]
