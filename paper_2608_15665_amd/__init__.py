"""SubZero+ hot path on AMD Instinct MI355X (gfx950).

The computation lives in libzo.so (hand-written HIP kernels behind the C ABI
of include/zo.h); this package only binds it.  Entry points:

    subspace_refresh       Haar factors of Gaussian panels (Eq. 11, Alg. 1);
                           subspace_refresh_noalloc the same for callers that cannot
                           allocate (the library's static per-GPU scratch)
    perturbed_linear       X_b (W +- eps U Z_j V^T)^T for all query blocks (Eq. 4);
                           PerturbedLinear.apply takes a fused ReLU or residual epilogue;
                           prepare_group prepares a layer's q, k, v in one pass over X
    lora_perturbed_linear  the same for a LoRA-adapted layer: both adapter factors
                           perturbed in their own subspaces
    layernorm, causal_attention, DecoderLayer
                           the network a query evaluates (the forward of Eq. 5): a
                           pre-LN decoder layer with all six matrices perturbed
    rmsnorm, rope, LlamaLayer
                           the same for a LLaMA-family layer (RMS norms, rotary
                           positions, SwiGLU MLP) with all seven matrices perturbed
    LlamaLoraLayer         the LoRA scheme's layer (grouped key/value heads, frozen
                           base, perturbed adapters on q and v)
    subspace_adam_update   subspace Adam and W <- W - lr U S V^T (Eqs. 6-10)
    subspace_sgd_update    plain subspace SGD, W <- W - lr U Zbar V^T
    sq_loss, combine_central, combine_forward   loss and estimate helpers (central
                           difference, or forward difference against a baseline block)
"""
from ._lib import (ZO_BF16, ZO_EPI_NONE, ZO_EPI_RELU, ZO_EPI_RESIDUAL, ZO_EPI_SILU_MUL, ZO_F16, ZO_F32, ZO_MAX_BLOCKS,
                   ZO_MAX_QR_RANK, ZO_MAX_RANK, ZO_NOALLOC_SCRATCH_BYTES, ABI_SYMBOLS, LIB_PATH, DecoderLayer, LlamaLayer,
                   LlamaLoraLayer, LoraPerturbedLinear, PerturbedLinear, Workspace, ZoError, abi_version, causal_attention, combine_central,
                   combine_forward, layernorm, lib, lora_perturbed_linear, perturbed_linear, prepare_group, rmsnorm, rope,
                   sq_loss, subspace_adam_update, subspace_refresh, subspace_refresh_noalloc,
                   subspace_sgd_update)

__all__ = ["ZO_BF16", "ZO_EPI_NONE", "ZO_EPI_RELU", "ZO_EPI_RESIDUAL", "ZO_EPI_SILU_MUL", "ZO_F16", "ZO_F32", "ZO_MAX_BLOCKS",
           "ZO_MAX_QR_RANK", "ZO_MAX_RANK", "ZO_NOALLOC_SCRATCH_BYTES", "ABI_SYMBOLS", "LIB_PATH", "DecoderLayer", "LlamaLayer", "LlamaLoraLayer", "LoraPerturbedLinear",
           "PerturbedLinear", "Workspace", "ZoError", "abi_version", "causal_attention", "combine_central",
           "combine_forward", "layernorm", "lib", "lora_perturbed_linear", "perturbed_linear", "prepare_group", "rmsnorm", "rope", "sq_loss",
           "subspace_adam_update", "subspace_refresh", "subspace_refresh_noalloc", "subspace_sgd_update"]
