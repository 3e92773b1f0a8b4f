"""PnP-Nystra window attention on MI355X (gfx950).

The compute path is the HIP library ``libnystra.so`` (sources in ``csrc/``,
C ABI in ``include/nystra.h``); ``binding`` marshals torch tensors into it.
``workloads`` draws the seeded synthetic inputs.
"""
from . import binding  # noqa: F401  (loads nothing until first use)
from .binding import (  # noqa: F401
    NystraError,
    nystra_attn_forward,
    nystra_attn_forward_ex,
    nystra_attn_forward_ws,
    nystra_attn_workspace_size,
    nystra_block_forward,
    nystra_block_workspace_size,
    nystra_exact_attn_forward,
    nystra_landmark_pool,
    nystra_landmark_map,
    nystra_select_variant,
    nystra_status_str,
    nystra_default_opts,
    make_opts,
)
