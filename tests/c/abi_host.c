/* A plain C99 caller of the library's C ABI: host-only calls (no GPU needed).
 * Prints one line per check; the Python test compares them. */
#include <stdio.h>
#include <string.h>

#include "rettention.h"

int main(void) {
    rt_pattern p;
    int32_t nnz = -1;
    rt_status st;
    memset(&p, 0, sizeof p);
    p.kind = RT_PAT_LOCAL2D;
    p.grid_h = 32;
    p.grid_w = 32;
    p.keep = 1;
    st = rt_index_size(&p, 1024, 32, &nnz); /* PixArt-alpha-512: 32 blocks, diagonal only */
    printf("local2d %d %s %d\n", (int)st, rt_status_str(st), (int)nnz);
    st = rt_index_size(&p, 1024, 48, &nnz); /* unsupported block size */
    printf("block48 %d %s\n", (int)st, strstr(rt_last_error(), "block") != NULL ? "named" : "unnamed");
    {
        const uint8_t mask[4] = {1, 0, 0, 1}; /* 2 x 2 blocks, diagonal */
        const uint8_t empty[4] = {1, 1, 0, 0}; /* second row keeps nothing */
        rt_pattern e;
        memset(&e, 0, sizeof e);
        e.kind = RT_PAT_EXPLICIT;
        e.host_mask = mask;
        st = rt_index_size(&e, 128, 64, &nnz);
        printf("explicit %d %d\n", (int)st, (int)nnz);
        e.host_mask = empty;
        st = rt_index_size(&e, 128, 64, &nnz);
        printf("empty_row %d %s\n", (int)st, rt_status_str(st));
    }
    {
        rt_dims d = {2, 30, 17776, 64};
        int64_t bytes = -1;
        st = rt_dynamic_index_workspace(d, 64, 9, &bytes); /* 2 * B*H*278*64 floats */
        printf("workspace %d %lld\n", (int)st, (long long)bytes);
    }
    return 0;
}
