// Internal interface between the C ABI layer (api.hip) and the kernels (kernels.hip, partials.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

namespace fka {

constexpr int kSlice = 32;      // tokens a wave scores per step; work is balanced in whole slices
constexpr int kPageSize = 16;
constexpr int kMaxRows = 64;    // query rows (sequences x G) per KV head that one item can hold
constexpr int kMaxSeqs = 512;   // sequences per plan (per-sequence schedule tables live in LDS)

// ---------------------------------------------------------------------------------------
// Work schedule shared by the partial kernel, the merge kernel and the host.
//
// A unit is a run of sequences that share one prefix (the whole fork when the prefix is
// shared, else a single sequence).  Item i = u * Hkv + g holds every key of unit u and KV head
// g: first the unit's prefix slices (read by all the unit's query rows, nseq * G of them, so
// each prefix byte is fetched once for all branches), then the suffix slices of the unit's
// sequences in order (each read by its own sequence's G rows only).  With P prefix slices and
// S suffix slices (S follows the suffix lengths on the device), the item's work list has
// P + S slices.
//
// The launch has NV workers (waves), NV = waves per block x virtual blocks.
//   * One unit (static split): item g owns workers [floor(g NV / Hkv), floor((g+1) NV / Hkv)).
//     All items have the same keys, so this is balanced whatever the lengths, and the merge
//     finds every row's partials without reading anything.
//   * Several units (proportional split): with T = total slices, A = NV - (non-empty items)
//     and the 32.32 fixed-point ratio R = floor(A * 2^32 / T), item i owns workers
//     [WS(i), WS(i+1)), WS(i) = floor(C_i * R / 2^32) + K_i, where C_i counts the slices of the
//     items before i and K_i the non-empty items before it: an empty item owns none, every
//     other item at least one and about size_i * A / T of them.
// Within an item of W workers, worker j owns prefix slices [pre_split(j), pre_split(j+1)) and
// suffix slices [suf_split(j), suf_split(j+1)): the prefix part of each worker depends only on
// the plan (so the first prefix loads need no lengths), and when S >= W the suffix part makes
// each worker's total floor((j+1)(P+S)/W) - floor(j(P+S)/W), the balance of one joint split.
//
// The waves of block vb are workers [vb*NW, (vb+1)*NW).  Those on the same item form a group:
// its prefix range and suffix range are the unions of its workers' ranges, and its waves deal
// the slices of [prefix range ; suffix range] in turn.  The group writes one partial (o, lse)
// per row of the item to slot vb + i: along the order of work each step advances vb, i or
// both, so slots are distinct and fewer than (blocks + items).  Every block of a static split
// writes its slot, empty or not; under a proportional split the block holding an item's first
// worker records, for each row of the item, where its partials start and how many there are.
// ---------------------------------------------------------------------------------------
struct UnitRec {  // four int32 fields, read field by field on the device
    int32_t seq0;       // first sequence of the unit
    int32_t nseq;       // sequences of the unit (rows = nseq * G)
    int32_t plen;       // prefix length of the unit
    int32_t ps_before;  // prefix slices of the units before this one
};

constexpr int kRowRec = 2;  // merge record of a row under a proportional split: first part offset, count

__host__ __device__ inline int32_t slices_of(int32_t tokens) { return (tokens + kSlice - 1) / kSlice; }

// floor(a * b / c) for 0 <= a <= c, b >= 0, c > 0: 32-bit arithmetic whenever the product fits
// (the common case, far cheaper on the GPU than a 64-bit division).
__host__ __device__ inline int32_t mul_div(int32_t a, int32_t b, int32_t c)
{
    const uint64_t p = (uint64_t)(uint32_t)a * (uint32_t)b;
    if (p < ((uint64_t)1 << 32)) return (int32_t)((uint32_t)p / (uint32_t)c);
    return (int32_t)(p / (uint64_t)c);
}

// Fixed-point ratio workers per slice, R = floor(A * 2^32 / T) (0 <= A < 2^31, 0 < T < 2^31).
// Exact, without a 64-bit integer division (a long software sequence on the GPU): a double
// quotient is within 2^10 + 1 of R, a second one on the remainder brings it within 1, and the
// last remainder fixes it.  Products and remainders stay below 2^63.
__host__ __device__ inline uint64_t sched_ratio(int64_t A, int64_t T)
{
    const uint64_t num = (uint64_t)A << 32, t = (uint64_t)T;
    uint64_t q = (uint64_t)((double)num / (double)T);
    int64_t rem = (int64_t)(num - q * t);
    q = (uint64_t)((int64_t)q + (int64_t)floor((double)rem / (double)T));
    rem = (int64_t)(num - q * t);
    if (rem < 0)
        --q;
    else if (rem >= T)
        ++q;
    return q;
}

// First worker of an item that starts at slice C (C <= T, so C * R < 2^63) with K
// non-empty items before it (proportional split).
__host__ __device__ inline int32_t worker_start(int64_t C, int64_t K, uint64_t R)
{
    return (int32_t)(((uint64_t)C * R) >> 32) + (int32_t)K;
}

// First worker of item g under the static split of NV workers over Hkv items.
__host__ __device__ inline int32_t static_start(int32_t g, int32_t NV, int32_t Hkv) { return mul_div(g, NV, Hkv); }

// Item of worker w under the static split.
__host__ __device__ inline int32_t static_item(int32_t w, int32_t NV, int32_t Hkv)
{
    int32_t g = mul_div(w, Hkv, NV);
    if (g + 1 < Hkv && static_start(g + 1, NV, Hkv) <= w) ++g;
    return g;
}

// First prefix slice of worker j (0 <= j <= W) of an item with P prefix slices.
__host__ __device__ inline int32_t pre_split(int32_t j, int32_t W, int32_t P) { return mul_div(j, P, W); }

// First suffix slice of worker j (0 <= j <= W) of an item with P prefix and S suffix slices.
// Non-decreasing in j from 0 to S: for S >= W, floor(T/W) >= ceil(P/W), so each worker's joint
// count floor((j+1)T/W) - floor(jT/W) covers its prefix count.
__host__ __device__ inline int32_t suf_split(int32_t j, int32_t W, int32_t P, int32_t S)
{
    if (S >= W) return mul_div(j, P + S, W) - mul_div(j, P, W);
    return mul_div(j, S, W);
}

struct AttnArgs {
    const UnitRec *units;  // [n_units]
    int32_t n_units;
    int32_t static_split;  // 1: one unit, items split statically
    int32_t ps_total;      // prefix slices of all units
    const int32_t *seq_prefix_len;  // [S] prefix length of each sequence's unit (paged page offsets)
    int32_t *rowrec;        // proportional split: [S * Hq][kRowRec], written by this launch
    int32_t *lens;          // [S] clamped suffix lengths of this launch, for the merge (block 0)
    const uint16_t *q;  // [S][Hq][d]
    // contiguous layout
    const uint16_t *prefix_k, *prefix_v;  // [Hkv][Lp][d]
    const uint16_t *suffix_k, *suffix_v;  // [S][Hkv][cap][d]
    int32_t prefix_len;
    int32_t suffix_cap;
    // paged layout
    const uint16_t *k_pool, *v_pool;  // [pages][Hkv][16][d]
    const int32_t *page_table;        // [S][max_pages]
    int32_t max_pages;
    int32_t n_pool_pages;
    int32_t paged;
    const int32_t *suffix_len;  // [S]
    int32_t max_suffix_len;
    int32_t n_seqs;
    int32_t n_q_heads;
    int32_t n_kv_heads;
    int32_t group;
    float scale_log2;  // softmax scale * log2(e)
    float *part_o;     // [slots][slot_rows][d]
    float *part_lse;   // [slots][slot_rows]
    int32_t slot_rows;
    int32_t n_slots;
    int32_t *err;
    // instruction prefill (the prefill kernel only): sequence s = b n + t is instruction token t of
    // branch b, reading b's suffix buffer up to position suffix_len[b] + t (n = prefill_n)
    int32_t prefill_n;
    int32_t prefill_groups;  // instruction prefill: units per block, each taken by NW / groups waves
};

struct MergeArgs {
    const float *part_o;    // explicit mode [n_parts][rows][d]; plan mode [slots][slot_rows][d]
    const float *part_lse;  // explicit mode [n_parts][rows];    plan mode [slots][slot_rows]
    float *out;             // [rows][d]
    float *out_lse;         // [rows] or null
    int32_t rows;
    int32_t n_q_heads;       // rows of one sequence (plan mode)
    // explicit mode (plan == 0): every row merges parts 0..n_parts-1
    int32_t n_parts;
    // plan mode: row (s, h) merges the partials of its item (see the work schedule above)
    int32_t plan;
    int32_t static_split;      // 1: slots from the static split; 0: from rowrec
    const int32_t *rowrec;     // proportional split: written by this launch's partial kernel
    const int32_t *lens;       // this launch's clamped suffix lengths
    int32_t slot_rows;
    int32_t n_slots;           // records pointing outside [0, n_slots * slot_rows) are not followed
    int32_t *err;
    int32_t waves;      // NW: workers per virtual block
    int32_t n_workers;  // NV
    // fused step: the token in k_new / v_new (not yet in the cache) joins each row as one
    // more part; block (s, head 0) then stores it and advances suffix_len[s]
    int32_t step_mode;
    int32_t *suffix_len;  // written only by a fused step
    int32_t max_suffix_len;
    const uint16_t *q;  // [S][Hq][d]
    float scale;        // softmax scale (natural-log units)
    int32_t group;      // G = Hq / Hkv
    const uint16_t *k_new, *v_new;  // [S][Hkv][d]
    uint16_t *k_dst, *v_dst;        // suffix buffers or pools
    const int32_t *page_table;
    const int32_t *seq_prefix_len;
    int32_t suffix_cap;
    int32_t max_pages;
    int32_t n_pool_pages;
    int32_t n_kv_heads;
    int32_t paged;
};

struct AppendArgs {
    const uint16_t *k_new, *v_new;  // [S][Hkv][d]
    uint16_t *k_dst, *v_dst;        // contiguous suffix buffers or paged pools
    const int32_t *page_table;      // paged only
    const int32_t *seq_prefix_len;  // paged only: prefix length of each sequence's group
    int32_t *suffix_len;
    int32_t suffix_cap;  // contiguous
    int32_t max_pages;   // paged
    int32_t n_pool_pages;  // paged
    int32_t max_suffix_len;
    int32_t n_kv_heads;
    int32_t head_dim;
    int32_t paged;
    int32_t *err;
};

struct GatherArgs {
    const uint16_t *k_pool, *v_pool;
    const int32_t *page_table;
    uint16_t *k_out, *v_out;  // [Hkv][out_len - begin][d]
    int32_t seq;
    int32_t prefix_len;
    int32_t begin;            // first logical position copied
    int32_t out_len;          // one past the last
    int32_t max_pages;
    int32_t n_pool_pages;
    int32_t n_kv_heads;
    int32_t head_dim;
    int32_t *err;
};

struct ScatterArgs {
    const uint16_t *k_src, *v_src;  // positions [from, len): [Hkv][len - from][d]
    const int32_t *page_row;        // dense layout: position p at page_row[p / 16], slot p % 16
    uint16_t *k_pool, *v_pool;
    int32_t len;
    int32_t from;
    int32_t n_pool_pages;
    int32_t n_kv_heads;
    int32_t head_dim;
    int32_t *err;                   // nullable
};

// Instruction prefill as a tiled multi-query kernel (prefill.hip, head_dim 128).  Rows of KV head g
// are cut into units of 32 (row i: query head g G + i mod G of virtual sequence i / G, where
// sequence s = b n + t is instruction token t of branch b); block vb takes KV head vb mod Hkv,
// unit group k = (vb / Hkv) mod unit_groups (units [floor(k U / UG), floor((k + 1) U / UG)), at
// most eight, one per wave) and prefix range
// vb / (Hkv unit_groups) of `ranges`, range r covering prefix tiles (64 keys) [floor(r T / R),
// floor((r + 1) T / R)) of T = prefix_tiles + tail_reserve, clamped to the whole tiles; the last
// range also reads the prefix keys past them (Lp mod 64) and the suffix keys.  Part r of output row (s, h) is written at
// part_o[(r S Hq + s Hq + h) d] and part_lse[r S Hq + s Hq + h].
struct PrefillArgs {
    const uint16_t *q;                    // [S][Hq][d]
    const uint16_t *prefix_k, *prefix_v;  // contiguous: [Hkv][Lp][d]
    const uint16_t *suffix_k, *suffix_v;  // contiguous: [N][Hkv][cap][d]
    const uint16_t *k_pool, *v_pool;      // paged: [pages][Hkv][16][d]
    const int32_t *page_table;            // paged: [N][max_pages]
    const int32_t *suffix_len;            // [N], each branch's suffix before the instruction
    float *part_o;                        // [ranges][S Hq][d]
    float *part_lse;                      // [ranges][S Hq]
    int32_t *err;
    int32_t n_branches, n_tokens;  // N, n
    int32_t prefix_len, suffix_cap, max_suffix_len;
    int32_t max_pages, n_pool_pages;
    int32_t paged;
    int32_t n_q_heads, n_kv_heads, group;
    int32_t n_units;       // 32-row units per KV head
    int32_t unit_groups;   // ceil(n_units / 8)
    int32_t ranges;        // R
    int32_t prefix_tiles;  // floor(Lp / 64): whole 64-key tiles
    int32_t tail_reserve;  // tiles of the balance given to the last range's per-wave keys
    float scale_log2;      // softmax scale * log2(e)
};

// error-flag bits (device)
constexpr int32_t kErrSuffixClamped = 1;
constexpr int32_t kErrAppendNoRoom = 2;
constexpr int32_t kErrBadPage = 4;
constexpr int32_t kErrBadSchedule = 8;

hipError_t launch_partials(const AttnArgs &a, int n_blocks, int head_dim, int row_tiles, hipStream_t s);
// Resident blocks per compute unit of the partial kernel for this shape (0 on error).
int partials_blocks_per_cu(int head_dim, int row_tiles, bool paged);
// Waves per block of the partial kernel for this shape.
int partials_waves_per_block(int head_dim, int row_tiles, bool paged);
int prefill_waves_per_block(int head_dim, int row_tiles, bool paged);
// Query rows (tokens x G) per unit of the instruction prefill: 32 for d = 128 (two tiles, two
// waves per SIMD) when a unit of 32 rows holds a token, else kMaxRows.
int prefill_max_rows(int head_dim, int group);
// Instruction prefill: the partial kernel over virtual sequences (AttnArgs::prefill_n) with the
// cyclic placement over block sets, contiguous suffix buffers or (AttnArgs::paged) the page pool,
// where a virtual sequence reads its branch's page-table row.
hipError_t launch_prefill(const AttnArgs &a, int n_blocks, int head_dim, int row_tiles, hipStream_t s);
int prefill_blocks_per_cu(int head_dim, int row_tiles, bool paged);
hipError_t launch_merge(const MergeArgs &a, int head_dim, hipStream_t s);
// The tiled instruction prefill (head_dim 128): query rows per unit (one wave each), waves (and
// so units) per block, resident blocks per compute unit, and the launch.
int prefill_tiles_unit_rows();
int prefill_tiles_waves();
int prefill_tiles_blocks_per_cu(bool paged);
hipError_t launch_prefill_tiles(const PrefillArgs &a, int n_blocks, hipStream_t s);
hipError_t launch_append(const AppendArgs &a, int n_seqs, hipStream_t s);
hipError_t launch_gather(const GatherArgs &a, hipStream_t s);
hipError_t launch_scatter(const ScatterArgs &a, hipStream_t s);
hipError_t launch_read_probe(const void *buf, size_t bytes, int blocks, int threads, int unroll, uint32_t *sink,
                             hipStream_t s);

}  // namespace fka
