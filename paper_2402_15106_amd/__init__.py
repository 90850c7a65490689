"""MI355X (gfx950) hot path of DS-MPNN (arXiv 2402.15106).

Node sampling, radius-graph construction, the edge-conditioned
message-passing layer (forward and backward) and the encoder, decoder and
loss of the hop loop as hand-written HIP kernels behind a C ABI
(include/dsmpnn.h); this package is the thin Python binding.
"""

from ._lib import (  # noqa: F401
    Dsmp, DsmpError, Graph, LayerDesc, layer_desc, load_library, LIB_PATH, EXPORTED, KERNEL_CLASSES,
    CAP_KNN, CAP_RANDOM, F32, BF16, ACT_IDENTITY, ACT_RELU, ATTR_CONCAT, ATTR_DIFF,
    GRAD_ACCUMULATE, GRAD_X_ACCUMULATE, MlpDesc, EDGE_AUTO, EDGE_PER_EDGE, EDGE_AGGREGATE, OK, INVALID_ARG, CAPACITY, HIP_ERROR, UNSUPPORTED, WORKSPACE_TOO_SMALL,
)
from .hop import HopShapes, HopStep  # noqa: F401,E402
from .infer import SubdomainInference  # noqa: F401,E402
