/* A plain C11 program against include/rsc.h and librsc.so: the header must
 * compile as C and the host-only entry points must work without a GPU.
 * Built and run by tests/test_abi.py. */
#include <stdio.h>
#include <string.h>

#include "rsc.h"

int main(void) {
    if (rsc_abi_version() != RSC_ABI_VERSION) return 1;
    if (strcmp(rsc_status_string(RSC_ERR_CAPACITY), "RSC_ERR_CAPACITY") != 0) return 2;
    /* budget -> k as a column fraction: floor(n p / 100) */
    if (rsc_k_from_fraction(2449029, 30, 100) != 734708) return 3;
    rsc_csr_t A;
    memset(&A, 0, sizeof A);
    A.n_rows = -1;
    if (rsc_spmm_workspace_bytes(&A) != 0) return 4;
    /* greedy allocation on two layers of four pairs, one block per pair */
    const uint64_t k0[4] = {9ull << 52, 7ull << 52, 5ull << 52, 3ull << 52};
    const uint64_t k1[4] = {8ull << 52, 6ull << 52, 4ull << 52, 2ull << 52};
    const uint64_t *keys[2] = {k0, k1};
    const int32_t colnnz[4] = {3, 1, 2, 4};
    const int32_t d[2] = {4, 2};
    const double fro_b2[2] = {1.0, 1.0};
    int32_t k_out[2] = {-1, -1};
    int64_t bud = -1;
    if (rsc_greedy_allocate(2, 4, 10, keys, colnnz, d, 1.0, fro_b2, 1, 2, 1, 4, k_out, &bud) != RSC_OK) return 5;
    /* the budget ends at or below half of the full 10 * (4 + 2) */
    if (bud * 2 > 60 || k_out[0] < 0 || k_out[0] > 4 || k_out[1] < 0 || k_out[1] > 4) return 6;
    if (rsc_greedy_allocate(0, 4, 10, keys, colnnz, d, 1.0, fro_b2, 1, 2, 1, 4, k_out, &bud) !=
        RSC_ERR_INVALID_ARGUMENT)
        return 7;
    printf("%d %d %lld\n", k_out[0], k_out[1], (long long)bud);
    return 0;
}
