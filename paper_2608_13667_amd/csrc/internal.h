// Internal interface between the C ABI layer (api.hip) and the kernels (kernels.hip).
#pragma once

#include <hip/hip_runtime.h>
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

// Per-launch schedule snapshot written by the partial kernel (block 0) for the merge.
// int32 words: [0] T, [1] non-empty items, [2] NV, [3] unused, then for sequence s:
// [4 + 3s] clamped suffix length, [5 + 3s] CS(s), [6 + 3s] NE(s), where CS(s) and NE(s)
// count the slices and the non-empty items of the suffix items of sequences before s.
constexpr int kSchedHeader = 4;

// Static per-row table of the merge (row = s * Hq + h, g = h / G), int32 words:
// [0] prefix item of the row (-1 if none), [1] the row's row within it, [2] its C, [3] its K,
// [4] its slices, [5] s, [6] g, [7] h % G (the row within the suffix item (s, g)).
constexpr int kRowInfo = 8;
__host__ __device__ inline int sched_words(int n_seqs) { return kSchedHeader + 3 * n_seqs; }

__host__ __device__ inline int32_t slices_of(int32_t tokens) { return (tokens + kSlice - 1) / kSlice; }

// Fixed-point ratio workers per slice, R = floor(A * 2^32 / T) (A < 2^31, T > 0).
__host__ __device__ inline uint64_t sched_ratio(int64_t A, int64_t T)
{
    return ((uint64_t)A << 32) / (uint64_t)T;
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

struct AttnArgs {
    const PrefixItem *pre_items;  // [n_pre]
    int32_t n_pre;
    int32_t pre_slices;   // sum of the prefix items' slices
    int32_t pre_nonempty; // non-empty prefix items
    const int32_t *seq_prefix_len;  // [S] prefix length of each sequence's unit (paged page offsets)
    int32_t *sched;       // per-launch snapshot for the merge
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
    // explicit mode (sched == null): every row merges parts 0..n_parts-1
    int32_t n_parts;
    // plan mode: row (s, h) merges the slots of its prefix item and of its suffix item
    const int32_t *sched;         // snapshot written by the partial kernel
    const int32_t *row_info;      // [rows][kRowInfo] static per-row table (see kRowInfo)
    int32_t n_pre;
    int32_t pre_slices;
    int32_t pre_nonempty;
    int32_t waves;          // NW: workers per virtual block
    int32_t slot_rows;
    int32_t *err;
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
    uint16_t *k_out, *v_out;  // [Hkv][out_len][d]
    int32_t seq;
    int32_t prefix_len;
    int32_t out_len;
    int32_t max_pages;
    int32_t n_pool_pages;
    int32_t n_kv_heads;
    int32_t head_dim;
    int32_t *err;
};

// error-flag bits (device)
constexpr int32_t kErrSuffixClamped = 1;
constexpr int32_t kErrAppendNoRoom = 2;
constexpr int32_t kErrBadPage = 4;

hipError_t launch_partials(const AttnArgs &a, int n_blocks, int head_dim, int row_tiles, hipStream_t s);
// Resident blocks per compute unit of the partial kernel for this shape (0 on error).
int partials_blocks_per_cu(int head_dim, int row_tiles, bool paged);
// Waves per block of the partial kernel for this shape.
int partials_waves_per_block(int head_dim, int row_tiles);
hipError_t launch_merge(const MergeArgs &a, int head_dim, hipStream_t s);
hipError_t launch_append(const AppendArgs &a, int n_seqs, hipStream_t s);
hipError_t launch_gather(const GatherArgs &a, hipStream_t s);

}  // namespace fka
