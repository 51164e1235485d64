/* A plain C99 consumer of the library: compiles against include/nuna.h, links libnuna.so and
 * exercises the calls that need no device memory.  Every collective call here is rejected by the
 * host checks (or is a count-0 no-op) before any launch, so no kernel ever runs on the fake
 * addresses.  Prints "ok" and returns 0 when every status is the documented one. */
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "nuna.h"

static int failures = 0;

static void expect(int cond, const char* what) {
    if (!cond) {
        printf("FAIL %s (last error: %s)\n", what, nuna_last_error_string());
        ++failures;
    }
}

int main(void) {
    const void* in[8];
    void* out[8];
    int r;
    for (r = 0; r < 8; ++r) {
        in[r] = (const void*)(uintptr_t)(0x100000000ull + (uint64_t)r * 0x100000ull);
        out[r] = (void*)(uintptr_t)(0x200000000ull + (uint64_t)r * 0x100000ull);
    }
    expect(nuna_version() > 0, "version");

    expect(nuna_allreduce(in, out, 0, 64, NUNA_BF16, NUNA_ALGO_AUTO, NUNA_PLACE_XCD, NULL) == NUNA_ERR_INVALID_ARG,
           "P = 0 rejected");
    expect(strlen(nuna_last_error_string()) > 0, "error text set");
    expect(nuna_allreduce(in, out, 8, 0, NUNA_BF16, NUNA_ALGO_AUTO, NUNA_PLACE_XCD, NULL) == NUNA_OK,
           "count 0 is a no-op");
    expect(strlen(nuna_last_error_string()) == 0, "error text cleared on success");
    out[3] = (void*)((uintptr_t)out[3] + 8);
    expect(nuna_allreduce(in, out, 8, 64, NUNA_BF16, NUNA_ALGO_AUTO, NUNA_PLACE_XCD, NULL) == NUNA_ERR_MISALIGNED,
           "misaligned output rejected");
    out[3] = out[2];
    expect(nuna_allreduce(in, out, 8, 64, NUNA_BF16, NUNA_ALGO_AUTO, NUNA_PLACE_XCD, NULL) == NUNA_ERR_OVERLAP,
           "overlapping outputs rejected");
    expect(nuna_reduce_scatter(in, out, 8, 64, (nuna_dtype_t)7, NUNA_PLACE_XCD, NULL) == NUNA_ERR_UNSUPPORTED,
           "unknown dtype rejected");
    expect(nuna_all_gather(in, NULL, 8, 64, NUNA_F32, NUNA_PLACE_LINEAR, NULL) == NUNA_ERR_INVALID_ARG,
           "NULL output array rejected");

    {
        int64_t v = -1;
        expect(nuna_set_tunable("NUNA_VPT", 8) == NUNA_OK, "set tunable");
        expect(nuna_get_tunable("NUNA_VPT", &v) == NUNA_OK && v == 8, "get tunable");
        expect(nuna_set_tunable("NUNA_VPT", 3) == NUNA_ERR_INVALID_ARG, "tunable value outside its set");
        expect(nuna_set_tunable("NUNA_VPT", 0) == NUNA_OK, "reset tunable");
    }
    {
        /* Algorithm 1 on three threadblocks: 0 and 1 share chunk 1, 2 touches chunk 3 alone. */
        nuna_nap_topology_t topo;
        const int64_t offsets[4] = {0, 2, 4, 5};
        const int64_t chunks[5] = {0, 1, 1, 2, 3};
        const int64_t bytes[3] = {4096, 4096, 4096};
        int64_t group[3], ngroups = 0;
        int32_t domain[3], cu[3], stack[5];
        expect(nuna_nap_topology_mi355x(&topo) == NUNA_OK && topo.num_domains == 8, "topology");
        expect(nuna_nap_plan(&topo, 8, 3, offsets, chunks, bytes, NULL, group, domain, cu, stack, &ngroups) ==
                   NUNA_OK,
               "plan");
        expect(ngroups == 2 && group[0] == 0 && group[1] == 0 && group[2] == 1, "logical groups");
        expect(domain[0] == 0 && domain[1] == 0 && domain[2] == 1, "groups dealt to domains");
        expect(stack[1] == stack[2], "a shared chunk has one stack");
    }
    {
        int64_t g = 0;
        expect(nuna_placement_grid(NUNA_PLACE_XCD, 10, 4, &g) == NUNA_OK && g == 64, "XCD grid of 10 groups of 4");
    }
    if (failures == 0) printf("ok\n");
    return failures == 0 ? 0 : 1;
}
