// Internal interface between the C ABI layer (api.hip) and the kernels (kernels.hip).
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
// The keys are cut into items, in this fixed order:
//   prefix items  i = u * Hkv + g            (u = prefix unit: a sequence group when the
//                                              prefix is shared, else one sequence)
//   suffix items  i = n_pre + s * Hkv + g    (sequence s, KV head g)
// Item i holds size_i = ceil(tokens_i / kSlice) slices; C_i is the number of slices of the
// items before it and K_i the number of non-empty items before it.  Suffix sizes follow
// the suffix lengths on the device, so the schedule is rebuilt by every launch.
//
// The launch has NV workers (waves), NV = waves per block x virtual blocks.  With
// T = total slices, A = NV - (non-empty items) and the 32.32 fixed-point ratio
// R = floor(A * 2^32 / T), item i owns workers [WS(i), WS(i+1)) with
// WS(i) = floor(C_i * R / 2^32) + K_i: an empty item owns none, every other item at least
// one and about size_i * A / T of them; the items end at WS(n_items), NV - 1 or NV, and a
// worker past that end has no work.  Worker j of an item with w workers scores slices
// [floor(j*size/w), floor((j+1)*size/w)).
//
// The waves of block vb are workers [vb*NW, (vb+1)*NW).  They combine their
// results per item, and the partial of (vb, item i) goes to slot vb + i: along the
// order of work each step advances vb, i or both, so slots are distinct and fewer than
// (blocks + items).  The merge reads, for an item, the slots of every block that owns
// one of its workers; each of those blocks writes its slot, empty or not.
// ---------------------------------------------------------------------------------------
struct PrefixItem {  // eight int32 fields, read field by field on the device
    int32_t seq0;     // first sequence of the item's rows
    int32_t nseq;     // sequences of the item's rows (rows = nseq * G)
    int32_t kv_head;
    int32_t n_tok;    // prefix length of the unit
    int32_t c0;       // slices of the prefix items before this one
    int32_t k0;       // non-empty prefix items before this one
    int32_t pad0, pad1;
};

// Schedule cache.  The schedule depends only on the plan and on the clamped suffix lengths.  The
// merge kernel of each launch builds, into the other half of a ping-pong pair, the schedule for
// two candidates of the next launch's lengths: candidate 0 = this launch's lengths (the next
// call of a multi-layer model, or a decode without append) and, after a fused step, candidate 1
// = the lengths after the append (the same layer's next step).  Per candidate:
//   table  [workers][kTabWords]: what the partial kernel's placement puts in LDS for each
//          worker (its item, the item's rows and keys, and its group in the block);
//   key    [S]: the clamped suffix lengths the table is for (-1 at [0]: none);
//   rowrec [S * Hq][kRowRec]: for merge row (s, h) the offset (slot * slot_rows + row within the
//          slot) of its first prefix part and the count of prefix parts, then the same for its
//          suffix item; parts of one item sit in consecutive slots.
// A launch reads half `cur` (the host alternates it after each merge).  The partial kernel
// takes the first candidate whose key equals the clamped lengths it reads; if none does, it
// builds the schedule itself and writes its slot records to a separate live buffer.  Block 0
// records the choice (sel: 0, 1, or 2 for the live records) and the clamped lengths (lens) for
// the merge.  Only the merge writes a candidate, so a key always describes its table and records.
constexpr int kTabWords = 9;
constexpr int kRowRec = 4;

__host__ __device__ inline int32_t slices_of(int32_t tokens) { return (tokens + kSlice - 1) / kSlice; }

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
// non-empty items before it.
__host__ __device__ inline int32_t worker_start(int64_t C, int64_t K, uint64_t R)
{
    return (int32_t)(((uint64_t)C * R) >> 32) + (int32_t)K;
}

// Slice range [lo, hi) of worker j of an item with `size` slices and w workers (exact floor
// divisions; 32-bit arithmetic whenever w * size fits, which gives the same result cheaper).
__host__ __device__ inline void worker_range(int32_t j, int32_t w, int32_t size, int32_t &lo, int32_t &hi)
{
    if ((uint64_t)w * (uint64_t)size < ((uint64_t)1 << 32)) {
        lo = (int32_t)((uint32_t)j * (uint32_t)size / (uint32_t)w);
        hi = (int32_t)((uint32_t)(j + 1) * (uint32_t)size / (uint32_t)w);
    } else {
        lo = (int32_t)((int64_t)j * size / w);
        hi = (int32_t)((int64_t)(j + 1) * size / w);
    }
}

// The group of virtual block vb on an item with workers [ws0, ws1) and `size` slices: the
// block's workers [lo, hi) of the item and the union [glo, ghi) of their slice ranges.
__host__ __device__ inline void block_group(int32_t vb, int32_t nw, int32_t ws0, int32_t ws1, int32_t size,
                                            int32_t &lo, int32_t &hi, int32_t &glo, int32_t &ghi)
{
    lo = ws0 > vb * nw ? ws0 : vb * nw;
    hi = ws1 < (vb + 1) * nw ? ws1 : (vb + 1) * nw;
    int32_t dummy;
    worker_range(lo - ws0, ws1 - ws0, size, glo, dummy);
    worker_range(hi - 1 - ws0, ws1 - ws0, size, dummy, ghi);
}

// Slot records (kRowRec) of the rows of item i, whose parts are `count` consecutive slots from
// slot vb0 + i: a prefix item's rows are (s, g*G + r) for s in [seq0, seq0 + nseq), a suffix
// item's (seq0, g*G + r); the record's row within the slot is (s - seq0) * G + r.
__host__ __device__ inline void write_rowrecs(int32_t *rowrec, int32_t i, int32_t n_pre, int32_t seq0, int32_t nseq,
                                              int32_t g, int32_t G, int32_t Hq, int32_t slot_rows, int32_t vb0,
                                              int32_t count)
{
    const int32_t field = i < n_pre ? 0 : 2;
    for (int32_t s = 0; s < nseq; ++s)
        for (int32_t r = 0; r < G; ++r) {
            int32_t *rr = rowrec + ((size_t)(seq0 + s) * Hq + g * G + r) * kRowRec + field;
            rr[0] = (vb0 + i) * slot_rows + s * G + r;
            rr[1] = count;
        }
}

struct AttnArgs {
    const PrefixItem *pre_items;  // [n_pre]
    int32_t n_pre;
    int32_t pre_slices;   // sum of the prefix items' slices
    int32_t pre_nonempty; // non-empty prefix items
    const int32_t *seq_prefix_len;  // [S] prefix length of each sequence's unit (paged page offsets)
    const int32_t *tab[2];  // schedule cache of this launch: candidate tables and keys
    const int32_t *key[2];
    int32_t *rowrec_live;   // slot records written when no candidate is taken
    int32_t *sel;           // block 0 writes the choice: candidate 0 / 1, or 2 (live records)
    int32_t *lens;          // [S] clamped suffix lengths of this launch, for the merge
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
};

struct MergeArgs {
    const float *part_o;    // explicit mode [n_parts][rows][d]; plan mode [slots][slot_rows][d]
    const float *part_lse;  // explicit mode [n_parts][rows];    plan mode [slots][slot_rows]
    float *out;             // [rows][d]
    float *out_lse;         // [rows] or null
    int32_t rows;
    int32_t n_q_heads;       // rows of one sequence (plan mode)
    // explicit mode (rowrec == null): every row merges parts 0..n_parts-1
    int32_t n_parts;
    // plan mode: row (s, h) merges the slots of its prefix item and of its suffix item
    const int32_t *rowrec[3];  // slot records: candidates 0 and 1 of this launch, live (see kRowRec)
    const int32_t *sel;        // which of them this launch's partial kernel used
    const int32_t *lens;       // this launch's clamped suffix lengths
    int32_t slot_rows;
    int32_t n_slots;           // records pointing outside [0, n_slots * slot_rows) are not followed
    int32_t *err;
    // schedule cache for the next launch (tab_next[0] null: none is built)
    int32_t *tab_next[2], *key_next[2], *rowrec_next[2];
    const PrefixItem *pre_items;
    int32_t n_pre;
    int32_t pre_slices;
    int32_t pre_nonempty;
    int32_t n_seqs;
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
hipError_t launch_merge(const MergeArgs &a, int head_dim, hipStream_t s);
hipError_t launch_append(const AppendArgs &a, int n_seqs, hipStream_t s);
hipError_t launch_gather(const GatherArgs &a, hipStream_t s);
hipError_t launch_scatter(const ScatterArgs &a, hipStream_t s);

}  // namespace fka
