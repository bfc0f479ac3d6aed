"""PinSage hot path for one MI355X (gfx950).

Importance neighbourhoods by Philox random walks and layer-wise K-layer
CONVOLVE (Ying et al., KDD 2018, Secs. 3.2 and 3.4), implemented as HIP
kernels in libpinsage.so behind the C ABI of include/pinsage.h. This package
is the thin Python binding; it needs the built library and a GPU.
"""

from ._lib import PinsageError, lib  # noqa: F401
from .api import (  # noqa: F401
    DeviceGraph,
    DeviceLayer,
    DeviceMLP,
    EmbedAll,
    EmbedAllBipartite,
    Minibatch,
    Neighborhoods,
    Schedule,
    build_graph_neighborhoods,
    build_neighborhoods,
    convolve_layer,
    convolve_workspace_size,
    embed_all,
    embed_all_workspace_size,
    hard_negatives,
    max_margin_loss,
    output_mlp,
    profile_enable,
    profile_read,
)
