// Host-side check of the work-schedule arithmetic shared by the partial kernel, the
// merge kernel and fka_plan_slots (sched_ratio / worker_start / worker_range in
// internal.h).  For random item sizes and grids it verifies: the workers of the items
// tile [0, E) with E = NV - 1 or NV;
// every non-empty item owns at least one worker and empty items none; the slice ranges
// of an item's workers tile the item; the (virtual block, item) slots are distinct and
// below (virtual blocks + items); and the slots the merge enumerates for an item are
// exactly those the blocks write.  Prints "ok <cases>" or the first failure.
#include <cstdio>
#include <cstdlib>
#include <random>
#include <set>
#include <vector>

#include "internal.h"

using namespace fka;

static int fail(const char *what, int c)
{
    std::printf("FAIL case %d: %s\n", c, what);
    return 1;
}

int main(int argc, char **argv)
{
    const int cases = argc > 1 ? std::atoi(argv[1]) : 2000;
    std::mt19937_64 rng(12345);
    // sched_ratio against the plain 64-bit division: edge values and random pairs over the range
    {
        const int64_t edge[] = {0, 1, 2, 3, 31, 32, 33, 1000, 65535, 65536, 1 << 20, (1 << 30) - 1, 1 << 30,
                                (int64_t(1) << 31) - 2, (int64_t(1) << 31) - 1};
        auto ref = [](int64_t A, int64_t T) { return ((uint64_t)A << 32) / (uint64_t)T; };
        for (int64_t A : edge)
            for (int64_t T : edge)
                if (T > 0 && sched_ratio(A, T) != ref(A, T)) return fail("sched_ratio differs (edge)", (int)A);
        for (int k = 0; k < 2000000; ++k) {
            const int shift_a = (int)(rng() % 32), shift_t = (int)(rng() % 32);
            const int64_t A = (int64_t)(rng() & ((uint64_t(1) << shift_a) - 1));
            const int64_t T = 1 + (int64_t)(rng() & ((uint64_t(1) << shift_t) - 1));
            if (A >= (int64_t(1) << 31) || T >= (int64_t(1) << 31)) continue;
            if (sched_ratio(A, T) != ref(A, T)) return fail("sched_ratio differs", k);
        }
    }
    for (int c = 0; c < cases; ++c) {
        const int n_items = 1 + (int)(rng() % 300);
        const int NW = (rng() % 2) ? 8 : 4;
        const int NB = 1 + (int)(rng() % 300);
        std::vector<int64_t> size(n_items);
        int64_t T = 0, NNE = 0;
        for (int i = 0; i < n_items; ++i) {
            const int kind = (int)(rng() % 4);
            size[i] = kind == 0 ? 0 : kind == 1 ? 1 + (int64_t)(rng() % 4) : (int64_t)(rng() % 5000);
            T += size[i];
            NNE += size[i] > 0;
        }
        const int rounds = std::max<int64_t>(1, (2 * n_items + (int64_t)NB * NW - 1) / ((int64_t)NB * NW));
        const int64_t NV = (int64_t)NB * rounds * NW;
        const int64_t A = NV - NNE;
        if (T == 0) continue;
        if (A < NV / 2) return fail("A below NV/2", c);
        const uint64_t R = sched_ratio(A, T);
        std::vector<int> owner(NV, -1);
        std::set<int64_t> written;  // (virtual block, item) slots written
        int64_t C = 0, K = 0;
        int64_t prev_end = 0;
        for (int i = 0; i < n_items; ++i) {
            const int32_t ws0 = worker_start(C, K, R);
            const int32_t ws1 = size[i] > 0 ? worker_start(C + size[i], K + 1, R) : ws0;
            if (ws0 != prev_end) return fail("worker ranges are not contiguous", c);
            if (size[i] == 0 && ws1 != ws0) return fail("empty item owns workers", c);
            if (size[i] > 0 && ws1 <= ws0) return fail("non-empty item owns no worker", c);
            int32_t next = 0;
            for (int32_t gw = ws0; gw < ws1; ++gw) {
                int32_t lo, hi;
                worker_range(gw - ws0, ws1 - ws0, (int32_t)size[i], lo, hi);
                if (lo != next || hi < lo) return fail("slice ranges do not tile the item", c);
                next = hi;
                owner[gw] = i;
                written.insert((int64_t)(gw / NW) * 1000000 + i);
            }
            if (size[i] > 0 && next != size[i]) return fail("slice ranges miss the item's end", c);
            // what the merge enumerates for item i
            if (size[i] > 0) {
                for (int32_t vb = ws0 / NW; vb <= (ws1 - 1) / NW; ++vb)
                    if (!written.count((int64_t)vb * 1000000 + i)) return fail("merge reads an unwritten slot", c);
            }
            prev_end = ws1;
            C += size[i];
            K += size[i] > 0;
        }
        if (prev_end != NV && prev_end != NV - 1) return fail("the items do not end at NV - 1 or NV", c);
        for (int64_t gw = 0; gw < prev_end; ++gw)
            if (owner[gw] < 0) return fail("a worker inside the items has no item", c);
        std::set<int64_t> slots;
        for (int64_t key : written) {
            const int64_t vb = key / 1000000, i = key % 1000000;
            const int64_t slot = vb + i;
            if (!slots.insert(slot).second) return fail("two partials share a slot", c);
            if (slot >= (int64_t)NB * rounds + n_items) return fail("slot out of range", c);
        }
    }
    std::printf("ok %d\n", cases);
    return 0;
}
