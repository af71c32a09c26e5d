// Host-side helpers shared by the C ABI translation units.
#pragma once

#include <stdint.h>

#include "../../include/pcpp.h"
#include "kernels.h"

namespace pcpp {

// Eq. 1 geometry of one validated call.
struct Geo {
    int32_t h;      // band height H / n
    int32_t up;     // context rows from the band above
    int32_t dn;     // context rows from the band below
    int32_t nq;     // queries per image: h * W
    int32_t n_kv;   // context keys per image: (up + h + dn) * W
    int32_t C;      // heads * head_dim
    int32_t esize;  // bytes per element
};

int validate_geom(const pcpp_geom_t* g, Geo* out);
int validate_geom_hops(const pcpp_geom_t* g, bool multi_hop, Geo* out);
KvSource make_kv_source(const pcpp_geom_t* g, const Geo& r, const void* k_fresh, const void* v_fresh,
                        const void* k_up, const void* v_up, const void* k_dn, const void* v_dn);
AttnParams make_attn_params(const pcpp_geom_t* g, const Geo& r, const void* q, void* out,
                            const KvSource& kv);
// Argument checks of pcpp_partial_attention (geometry, dtype, head_dim,
// pointers, 16-byte alignment); PCPP_OK or the status to return.
int check_attention(const pcpp_geom_t* g, Geo* r, const void* q, const void* k_fresh, const void* v_fresh,
                    const void* k_up, const void* v_up, const void* k_dn, const void* v_dn, const void* out);

}  // namespace pcpp
