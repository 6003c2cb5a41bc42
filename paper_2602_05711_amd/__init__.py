"""MI355X (gfx950) implementation of the OmniMoE atomic-expert layer forward pass.

The computation lives in libomnimoe.so (HIP kernels behind the C ABI of include/omnimoe.h);
``binding`` exposes the same entry points to Python for torch tensors.
"""
from .binding import (  # noqa: F401
    EXPORTED, KERNEL_NAMES, OmnimoeError, OmnimoeLayerDesc, Timer, load_library, make_desc,
    omnimoe_expert_backward, omnimoe_expert_forward, omnimoe_expert_forward_grouped,
    omnimoe_expert_forward_group_rows, omnimoe_expert_forward_scatter,
    omnimoe_expert_forward_token_centric,
    omnimoe_layer_forward, omnimoe_layer_forward_noalloc, omnimoe_layer_path,
    omnimoe_route, omnimoe_route_backward, omnimoe_route_dense, omnimoe_schedule, omnimoe_select, omnimoe_select_dense,
    omnimoe_shared_mlp, omnimoe_shared_mlp_workspace_size, omnimoe_workspace_size, workspace,
)
