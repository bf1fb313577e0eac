"""MI355X (gfx950) mixed-precision MoE expert-FFN kernels: the inference hot
path of DynaMo (arXiv 2503.21135) -- top-k routing and token permutation,
per-expert 2/3/4/6/8-bit packed weights with fp16 scale/zero, the channel-level
switch to resident 8-bit copies, the fused dequant + MFMA grouped SiLU-GLU
FFN, and un-permute/combine -- behind the C ABI of include/moe_quant.h.

The compute lives in libmoe_quant.so (built by ``build.build()``); the
modules here only marshal torch tensors into it.
"""
from ._lib import EXPORTS, LIB_PATH, MoEError, load  # noqa: F401
from .api import (moe_code_row_words, moe_expert_ffn_mixed, moe_expert_ffn_mixed_ev,  # noqa: F401
                  moe_ffn_plan, moe_quant_pack, moe_route_permute, moe_route_workspace_bytes, moe_set_channel_switch,
                  moe_unpermute_combine)
from .layer import MoELayer  # noqa: F401
