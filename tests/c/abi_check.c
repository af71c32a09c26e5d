/* A plain C99 client of the C ABI: compiles against include/pcpp.h alone
 * and calls the host-side entry points (geometry, validation, sizes), which
 * need no GPU.  Exit status 0 when every check holds, else the number of the
 * first failed check. */
#include <stdio.h>
#include <string.h>

#include "pcpp.h"

int main(void) {
    pcpp_geom_t g;
    int32_t h = 0, up = 0, dn = 0, n_kv = 0;
    memset(&g, 0, sizeof g);
    g.H = 128; g.W = 128; g.n_patches = 8; g.patch_idx = 3; g.partial = 0.25;
    g.heads = 10; g.head_dim = 64; g.batch = 1; g.step = 0; g.dtype = PCPP_DTYPE_BF16;

    if (pcpp_version() != PCPP_VERSION) return 1;
    if (pcpp_context_rows(&g, &h, &up, &dn, &n_kv) != PCPP_OK) return 2;
    if (h != 16 || up != 4 || dn != 4 || n_kv != 3072) return 3;   /* Eq. 1 at the 2048 px level-1 band */
    if (pcpp_boundary_bytes(&g) != (size_t)2 * 4 * 128 * 640 * 2) return 4;
    if (pcpp_strerror(PCPP_EINVAL) == NULL || pcpp_strerror(12345) == NULL) return 5;

    g.partial = 1.5;   /* beyond the neighbours: only the multi-hop form takes it */
    if (pcpp_context_rows(&g, NULL, NULL, NULL, NULL) != PCPP_EINVAL) return 6;
    if (pcpp_partial_attention_workspace_size(&g) != 0) return 7;
    if (pcpp_partial_attention_multihop_workspace_size(&g) == 0) return 8;

    g.partial = 0.25;
    g.patch_idx = 8;   /* out of range */
    if (pcpp_context_rows(&g, &h, &up, &dn, &n_kv) != PCPP_EINVAL) return 9;
    /* validation fails before any launch: no device is touched */
    if (pcpp_partial_attention(&g, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, NULL, 0, NULL) != PCPP_EINVAL)
        return 10;
    printf("C ABI checks passed: h=16 up=4 dn=4 n_kv=3072\n");
    return 0;
}
