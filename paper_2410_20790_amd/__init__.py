"""MI355X (gfx950) diff-computation encoder: SparseTem's per-layer sparse
delta convolution as hand-written HIP behind a C ABI (include/sparsetem.h).

``binding`` wraps the C entry points one to one; ``net.SparseTemNet`` keeps
weights and workspace in torch device memory.  Importing this package loads
``libsparsetem.so`` and raises ImportError if it has not been built.
"""

from . import binding
from .binding import StError
from .net import SparseTemNet, layer_desc

__all__ = ["binding", "StError", "SparseTemNet", "layer_desc"]
