/*
 * Oracle: counting-sort dispatch of top-k routed token slots.
 *
 * TEST INFRASTRUCTURE ONLY.  This file belongs to the CPU oracle that checks
 * the HIP expert stage; nothing in the product path links or calls it.
 *
 * What it computes (the paper's MoE-side token metadata is a count of tokens
 * per expert, and the payload is grouped by expert; section "Asynchronous
 * Dispatch", Table 2 MoE rows):
 *   slot s = t*k + j holds expert id ids[s]; ids[s] == -1 marks a masked slot.
 *   counts[e]      = number of slots whose id is e, for every e in [0, E)
 *   offsets[i]     = sum of counts[e0 + i'] for i' < i  (i in [0, E_loc])
 *   slot_of_row[r] = the local slots listed by ascending (expert id, s)
 *   row_of_slot[s] = position of s in that list, or -1 if s is not local
 * Ids outside [-1, E) are invalid: they are treated as masked and counted in
 * *n_bad.  The return value is N_loc, the number of local slots.
 *
 * This is the textbook counting sort: one pass to count, a prefix sum, and a
 * second pass in ascending s that places each slot at its expert's next free
 * row, which makes the order within an expert ascending in s (stable).
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

int32_t oracle_dispatch(int32_t T, int32_t k, int32_t E, int32_t e0, int32_t E_loc,
                        const int32_t *ids, int32_t *counts, int32_t *offsets,
                        int32_t *slot_of_row, int32_t *row_of_slot, int32_t *n_bad)
{
    int64_t n_slots = (int64_t)T * (int64_t)k;
    int32_t bad = 0;
    memset(counts, 0, sizeof(int32_t) * (size_t)E);
    for (int64_t s = 0; s < n_slots; ++s) {
        int32_t e = ids[s];
        if (e == -1) continue;
        if (e < -1 || e >= E) { ++bad; continue; }
        counts[e] += 1;
    }
    offsets[0] = 0;
    for (int32_t i = 0; i < E_loc; ++i)
        offsets[i + 1] = offsets[i] + counts[e0 + i];

    int32_t *next = (int32_t *)malloc(sizeof(int32_t) * (size_t)(E_loc > 0 ? E_loc : 1));
    if (!next) return -1;
    for (int32_t i = 0; i < E_loc; ++i) next[i] = offsets[i];
    for (int64_t s = 0; s < n_slots; ++s) {
        int32_t e = ids[s];
        int32_t i = e - e0;
        if (e >= 0 && e < E && i >= 0 && i < E_loc) {
            int32_t r = next[i]++;
            slot_of_row[r] = (int32_t)s;
            row_of_slot[s] = r;
        } else {
            row_of_slot[s] = -1;
        }
    }
    free(next);
    if (n_bad) *n_bad = bad;
    return offsets[E_loc];
}
