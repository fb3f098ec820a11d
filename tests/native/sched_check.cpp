// Host-side check of the work-schedule arithmetic shared by the partial kernel, the merge
// kernel and fka_plan_slots (internal.h).  Verifies:
//   * sched_ratio against the plain 64-bit division;
//   * mul_div against the plain 64-bit division;
//   * the static split: static_item inverts static_start, the items tile [0, NV) and each
//     owns floor or ceil of NV / Hkv workers;
//   * the proportional split: the workers of the items tile [0, E) with E = NV - 1 or NV,
//     every non-empty item owns at least one worker and empty items none;
//   * the split within an item: pre_split and suf_split are non-decreasing from 0 to P and
//     to S, and each worker's total differs from the even share by less than one slice when
//     S >= W (by less than two otherwise);
//   * the (virtual block, item) slots are distinct and below (virtual blocks + items), and
//     the slots the merge reads for an item are exactly those its blocks write.
// Prints "ok <cases>" or the first failure.
#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <random>
#include <set>
#include <vector>

#include "internal.h"

using namespace fka;

static int fail(const char *what, long c)
{
    std::printf("FAIL case %ld: %s\n", c, what);
    return 1;
}

// Checks the split of P prefix and S suffix slices over W workers.
static bool split_ok(int32_t W, int32_t P, int32_t S)
{
    int32_t lo = 0, hi = 0;
    for (int32_t j = 0; j < W; ++j) {
        const int32_t a0 = pre_split(j, W, P), a1 = pre_split(j + 1, W, P);
        const int32_t b0 = suf_split(j, W, P, S), b1 = suf_split(j + 1, W, P, S);
        if (a1 < a0 || b1 < b0) return false;
        const int32_t n = (a1 - a0) + (b1 - b0);
        if (j == 0) lo = hi = n;
        lo = std::min(lo, n);
        hi = std::max(hi, n);
    }
    if (pre_split(0, W, P) != 0 || pre_split(W, W, P) != P) return false;
    if (suf_split(0, W, P, S) != 0 || suf_split(W, W, P, S) != S) return false;
    return hi - lo <= (S >= W ? 1 : 2);
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
                if (T > 0 && sched_ratio(A, T) != ref(A, T)) return fail("sched_ratio differs (edge)", (long)A);
        for (int k = 0; k < 2000000; ++k) {
            const int shift_a = (int)(rng() % 32), shift_t = (int)(rng() % 32);
            const int64_t A = (int64_t)(rng() & ((uint64_t(1) << shift_a) - 1));
            const int64_t T = 1 + (int64_t)(rng() & ((uint64_t(1) << shift_t) - 1));
            if (A >= (int64_t(1) << 31) || T >= (int64_t(1) << 31)) continue;
            if (sched_ratio(A, T) != ref(A, T)) return fail("sched_ratio differs", k);
        }
    }
    // mul_div against the 64-bit division, both sides of the 32-bit product boundary
    for (int k = 0; k < 2000000; ++k) {
        const int32_t c = 1 + (int32_t)(rng() % ((k & 1) ? 4096 : 0x7fffffff));
        const int32_t a = (int32_t)(rng() % ((uint64_t)c + 1));
        const int32_t b = (int32_t)(rng() % ((k & 2) ? 0x7fffffffULL : 1u << 24));
        if (mul_div(a, b, c) != (int32_t)((int64_t)a * b / c)) return fail("mul_div differs", k);
    }
    // the split within an item: exhaustive over small sizes, random over large ones
    for (int32_t W = 1; W <= 40; ++W)
        for (int32_t P = 0; P <= 100; ++P)
            for (int32_t S = 0; S <= 100; ++S)
                if (!split_ok(W, P, S)) return fail("item split", (long)W * 1000000 + P * 1000 + S);
    for (int k = 0; k < 20000; ++k) {
        const int32_t W = 1 + (int32_t)(rng() % 1024);
        const int32_t P = (int32_t)(rng() % (1 << 22)), S = (int32_t)(rng() % (1 << ((k % 3) ? 12 : 22)));
        if (!split_ok(W, P, S)) return fail("item split (random)", k);
    }
    // static split
    for (int k = 0; k < 20000; ++k) {
        const int32_t Hkv = 1 + (int32_t)(rng() % 16);
        const int32_t NV = Hkv + (int32_t)(rng() % 4096);
        int32_t prev = 0;
        for (int32_t g = 0; g < Hkv; ++g) {
            const int32_t ws0 = static_start(g, NV, Hkv), ws1 = static_start(g + 1, NV, Hkv);
            if (ws0 != prev || ws1 - ws0 < NV / Hkv || ws1 - ws0 > (NV + Hkv - 1) / Hkv)
                return fail("static split does not tile evenly", k);
            for (int32_t w = ws0; w < ws1; ++w)
                if (static_item(w, NV, Hkv) != g) return fail("static_item is not the inverse", k);
            prev = ws1;
        }
        if (prev != NV) return fail("static split misses workers", k);
    }
    // proportional split and slots
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
            for (int32_t gw = ws0; gw < ws1; ++gw) {
                owner[gw] = i;
                written.insert((int64_t)(gw / NW) * 1000000 + i);
            }
            // what the merge reads for item i: blocks ws0 / NW .. (ws1 - 1) / NW
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
        // the same for a static split over Hkv = n_items % 16 + 1 items
        const int32_t Hkv = n_items % 16 + 1;
        std::set<int64_t> sslots;
        for (int32_t g = 0; g < Hkv && Hkv <= NV; ++g) {
            const int32_t ws0 = static_start(g, (int32_t)NV, Hkv), ws1 = static_start(g + 1, (int32_t)NV, Hkv);
            for (int32_t vb = ws0 / NW; vb <= (ws1 - 1) / NW; ++vb) {
                const int64_t slot = vb + g;
                if (!sslots.insert(slot).second) return fail("two static partials share a slot", c);
                if (slot >= (int64_t)NB * rounds + Hkv) return fail("static slot out of range", c);
            }
        }
    }
    std::printf("ok %d\n", cases);
    return 0;
}
