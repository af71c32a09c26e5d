// Placeholder: the transformer-block entry points are added with the GEMM,
// normalisation and cross-attention kernels.
#include "../../include/pcpp.h"

#define PCPP_EXPORT extern "C" __attribute__((visibility("default")))

PCPP_EXPORT size_t pcpp_transformer_block_workspace_size(const pcpp_geom_t*, const pcpp_block_weights_t*,
                                                         int32_t, int32_t) {
    return 0;
}

PCPP_EXPORT int pcpp_transformer_block(const pcpp_geom_t*, const pcpp_block_weights_t*, const void*,
                                       const void*, int32_t, int32_t, const void*, const void*,
                                       const void*, const void*, void*, void*, void*, void*, size_t,
                                       void*) {
    return PCPP_ENOTSUP;
}
