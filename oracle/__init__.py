"""CPU float64 oracle of the PCPP per-patch hot path.

TEST INFRASTRUCTURE ONLY: imported by the test suite, the smoke check and the
benchmark's CPU-baseline leg, never by the library or its Python binding.
"""

from .pcpp_oracle import (  # noqa: F401
    CTX_EPS,
    as_f64,
    assemble_context,
    boundary_messages,
    context_rows,
    context_rows_multihop,
    context_token_ids,
    from_bf16_bits,
    gelu,
    geglu,
    group_norm,
    group_norm_synchronized,
    group_stats,
    layer_norm,
    linear,
    mha,
    multihop_message,
    multihop_message_rows,
    partial_attention,
    partial_attention_multihop,
    place_boundary_messages,
    place_multihop_message,
    transformer_block,
    transformer_module,
    MODULE_BLOCK_KEYS,
)
from .unet_oracle import (  # noqa: F401
    RESNET_GN_EPS,
    conv3x3_band,
    conv3x3_band_mode,
    edge_rows,
    guided_noise,
    pad_band,
    resnet_block,
    resnet_weight_shapes,
    reverse_step_ddim,
    reverse_step_ddpm,
    scaled_linear_alphabar,
    silu,
    unet_band_step,
    image_step,
)
