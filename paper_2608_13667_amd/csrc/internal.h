// Internal interface between the C ABI layer (api.hip) and the kernels (kernels.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fka {

// Where a work item's keys come from.
enum ItemKind : int32_t {
    kPrefix = 0,  // shared prefix of the item's sequence group
    kSuffix = 1,  // own suffix of sequence seq0 (nseq == 1); clipped by suffix_len at run time
};

// One block of the partial-attention kernel: query rows of sequences
// [seq0, seq0 + nseq) x the G query heads of kv_head, over keys
// [tok_begin, tok_end) of the item's source; result goes to partial slot `part`.
struct WorkItem {  // eight int32 fields, read field by field on the device
    int32_t kind;
    int32_t seq0;
    int32_t nseq;
    int32_t kv_head;
    int32_t tok_begin;
    int32_t tok_end;
    int32_t part;
    int32_t prefix_len;  // prefix length of the sequence group (paged suffix page offset)
};

struct AttnArgs {
    const WorkItem *items;
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
    float *part_o;     // [slots][S][Hq][d]
    float *part_lse;   // [slots][S][Hq]
    int32_t *err;
    // persistent scheduling
    int32_t n_items;
    int32_t *queue;          // next item to hand out; zero between launches
    int32_t *done;           // blocks finished; zero between launches
};

struct MergeArgs {
    const float *part_o;    // [slots][rows][d]
    const float *part_lse;  // [slots][rows]
    float *out;             // [rows][d]
    float *out_lse;         // [rows] or null
    int32_t rows;
    int32_t n_q_heads;       // rows of one sequence (plan-driven mode)
    // explicit mode: every row merges parts 0..n_parts-1
    int32_t n_parts;
    // plan-driven mode (seq_prefix_parts != null): row of sequence s merges its
    // group's prefix parts 0..seq_prefix_parts[s]-1 and suffix parts
    // max_prefix_parts + j for j < ceil(min(suffix_len[s], max_suffix_len) / suffix_split)
    const int32_t *seq_prefix_parts;
    int32_t max_prefix_parts;
    int32_t *suffix_len;  // written only by a fused step
    int32_t suffix_split;
    int32_t max_suffix_len;
    int32_t *err;
    // fused step: the token in k_new / v_new (not yet in the cache) joins each row as one
    // more part; the last block then appends it and advances suffix_len
    int32_t step_mode;
    const uint16_t *q;  // [S][Hq][d]
    float scale;        // softmax scale (natural-log units)
    int32_t group;      // G = Hq / Hkv
    int32_t *counter;               // zero between launches
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

constexpr int kTileTokens = 128;  // split sizes are whole multiples of this many tokens
constexpr int kPageSize = 16;
constexpr int kMaxRows = 64;      // query rows (sequences x G) per KV head that one item can hold

hipError_t launch_partials(const AttnArgs &a, int n_blocks, int head_dim, int row_tiles, hipStream_t s);
hipError_t launch_merge(const MergeArgs &a, int head_dim, hipStream_t s);
hipError_t launch_append(const AppendArgs &a, int n_seqs, hipStream_t s);
hipError_t launch_gather(const GatherArgs &a, hipStream_t s);

}  // namespace fka
