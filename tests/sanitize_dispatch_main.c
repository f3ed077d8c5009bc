/*
 * Test driver: runs the oracle's counting-sort dispatch (oracle/dispatch.c)
 * once, built with AddressSanitizer and UndefinedBehaviorSanitizer by
 * tests/test_oracle_sanitizers_cpu.py.  CPU-only test infrastructure.
 *
 * stdin:  int32 T, k, E, e0, E_loc, then T*k int32 ids.
 * stdout: int32 N_loc, n_bad, counts[E], offsets[E_loc + 1],
 *         slot_of_row[N_loc], row_of_slot[T*k].
 * Every buffer is allocated at exactly the size the definition needs, so an
 * access past any of them is reported by the sanitizer.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

int32_t oracle_dispatch(int32_t T, int32_t k, int32_t E, int32_t e0, int32_t E_loc,
                        const int32_t *ids, int32_t *counts, int32_t *offsets,
                        int32_t *slot_of_row, int32_t *row_of_slot, int32_t *n_bad);

static int read_all(void *dst, size_t bytes)
{
    return fread(dst, 1, bytes, stdin) == bytes ? 0 : -1;
}

int main(void)
{
    int32_t hdr[5];
    if (read_all(hdr, sizeof hdr)) return 2;
    const int32_t T = hdr[0], k = hdr[1], E = hdr[2], e0 = hdr[3], E_loc = hdr[4];
    const size_t n = (size_t)T * (size_t)k;
    int32_t *ids = malloc(n ? n * 4 : 1);
    int32_t *counts = malloc((size_t)E * 4);
    int32_t *offsets = malloc(((size_t)E_loc + 1) * 4);
    int32_t *row_of_slot = malloc(n ? n * 4 : 1);
    if (!ids || !counts || !offsets || !row_of_slot || read_all(ids, n * 4)) return 2;
    /* first pass for the exact size of slot_of_row: the local slots */
    size_t n_loc = 0;
    for (size_t s = 0; s < n; ++s)
        if (ids[s] >= e0 && ids[s] < e0 + E_loc && ids[s] < E) ++n_loc;
    int32_t *slot_of_row = malloc(n_loc ? n_loc * 4 : 1);
    if (!slot_of_row) return 2;
    int32_t bad = -1;
    const int32_t r = oracle_dispatch(T, k, E, e0, E_loc, ids, counts, offsets, slot_of_row,
                                      row_of_slot, &bad);
    if (r < 0 || (size_t)r != n_loc) return 3;
    fwrite(&r, 4, 1, stdout);
    fwrite(&bad, 4, 1, stdout);
    fwrite(counts, 4, (size_t)E, stdout);
    fwrite(offsets, 4, (size_t)E_loc + 1, stdout);
    fwrite(slot_of_row, 4, n_loc, stdout);
    fwrite(row_of_slot, 4, n, stdout);
    free(ids);
    free(counts);
    free(offsets);
    free(row_of_slot);
    free(slot_of_row);
    return 0;
}
