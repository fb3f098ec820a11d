/*
 * forkattn.h -- C ABI of libforkattn.so: fork-aware decode attention on gfx950.
 *
 * The operation (paper, Sec. 3.2 Overview and Sec. 3.3 Forking via Trajectory
 * Continuation).  When the main thread of a ReAct agent finishes its Thought,
 * auxiliary branches are forked; every branch receives the same snapshot (the
 * history H_t followed by the thought R_t) plus its own short continuation, and
 * the key/value cache of the shared snapshot is reused by all decoding streams.
 * The main thread and the branches then decode concurrently.  One decode step is
 * therefore N sequences (main thread + branches), each with one new query token,
 * all reading one shared prefix K/V and each reading its own suffix K/V.  The
 * result for sequence b and query head h is ordinary scaled dot-product softmax
 * attention of q[b][h] over [shared prefix ; suffix of b], using the K/V head
 * h / G (G = n_q_heads / n_kv_heads).  Sharing the prefix is purely an
 * optimisation: the library reads each prefix K/V tile from memory once and
 * scores it against all N * G query rows of its K/V head, so the results equal
 * the per-branch attention.  Branches never see each other's suffixes.
 *
 * Conventions for every call
 *   - Tensors are caller-owned device memory passed as raw pointers.  bf16 means
 *     IEEE bfloat16 bit patterns (uint16 in memory).  All layouts are dense,
 *     row-major (C order), innermost dimension last.
 *   - Pointers to K/V/q data must be 16-byte aligned (the kernels use 128-bit loads).
 *   - Calls enqueue work on `stream` (a hipStream_t; NULL = the default stream)
 *     and return without synchronising.  Results are valid once the stream has
 *     reached that point.
 *   - Calls never allocate, free or synchronise, except fka_plan_create_*
 *     (allocates the plan's device workspace and schedule tables, copies the
 *     tables to the device), fka_plan_destroy (frees them) and
 *     fka_plan_device_error (reads the device error word).
 *   - A plan owns a workspace for partial results, so it may be used by one
 *     stream at a time.  Plans are independent of each other.
 *   - Every launch builds its work schedule on the device from the suffix lengths
 *     it finds there, so the lengths may change freely between calls.
 *   - Arguments are validated on the host before anything is launched; on an
 *     error nothing is enqueued, the call returns a negative fka_status and
 *     fka_last_error() describes it.  Values that live on the device (suffix
 *     lengths, page ids) are not visible to the host: the kernels clamp them to
 *     the plan's bounds and record a violation in a device flag that
 *     fka_plan_device_error() reports.
 *   - Nothing crosses the ABI as an exception; the library never prints or exits.
 */
#ifndef FORKATTN_H
#define FORKATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    FKA_OK = 0,
    FKA_ERR_INVALID_ARG = -1, /* null/misaligned pointer, inconsistent sizes */
    FKA_ERR_UNSUPPORTED = -2, /* valid request outside what the kernels implement (head_dim, rows per KV head) */
    FKA_ERR_HIP = -3,         /* a HIP runtime call or kernel launch failed; the HIP message is in fka_last_error() */
    FKA_ERR_NOMEM = -4        /* device allocation failed in fka_plan_create_* */
} fka_status;

/* Version of this ABI (major * 10000 + minor * 100 + patch). */
int fka_version(void);

/* Message describing the last failed call on this thread ("" if none).  The
 * string is owned by the library and valid until the next fka_* call on the
 * same thread. */
const char *fka_last_error(void);

/* Attention head geometry shared by all sequences of a plan. */
typedef struct {
    int32_t n_q_heads;   /* Hq: query heads per sequence */
    int32_t n_kv_heads;  /* Hkv: key/value heads; Hq % Hkv == 0, G = Hq / Hkv */
    int32_t head_dim;    /* d: 64 or 128 */
    float softmax_scale; /* scores are scale * q.k; 0 selects 1 / sqrt(head_dim) */
} fka_heads;

/* Opaque plan: the static part of the work schedule (the prefix-sharing units), the
 * grid, and the workspace for partial (o, lse) results.  Built once per fork (the
 * prefix length is fixed at the fork instant), reused for every decode step. */
typedef struct fka_plan fka_plan;

/* ---------------------------------------------------------------- contiguous KV */

/* One fork: n_branches sequences (main thread + auxiliary branches) sharing a
 * contiguous prefix of prefix_len tokens (Sec. 3.3). */
typedef struct {
    int32_t n_branches;     /* N >= 1 sequences sharing the prefix */
    int32_t prefix_len;     /* Lp >= 0, fixed at the fork */
    int32_t suffix_cap;     /* rows allocated per (branch, kv head) in the suffix buffers, >= 1 */
    int32_t max_suffix_len; /* upper bound on suffix_len[b] over the plan's lifetime, <= suffix_cap */
    int32_t share_prefix;   /* 1: fork-aware (prefix tiles read once for all N branches);
                               0: naive baseline, every branch re-reads the prefix on its own */
    int32_t rounds;         /* 0 = automatic; k in [1, 64] = spread the keys over at least k
                               rounds of the resident waves (more, smaller partial results) */
    int32_t blocks;         /* 0 = automatic (enough blocks for the keys at max_suffix_len, at most
                               those resident at once); k >= 1 = k blocks per round (capped at
                               the resident ones) */
} fka_contig_desc;

/* Build a plan for the contiguous layout.  Allocates device memory (schedule
 * tables, workspace, error flag) on the current device.  *out receives the plan,
 * owned by the caller until fka_plan_destroy.  Errors: FKA_ERR_INVALID_ARG (null
 * pointer, non-positive sizes, Hq % Hkv != 0, max_suffix_len > suffix_cap, rounds
 * outside [0, 64], blocks < 0), FKA_ERR_UNSUPPORTED (head_dim not 64/128, more than 64 rows N*G
 * per KV head, more than 512 sequences), FKA_ERR_NOMEM, FKA_ERR_HIP. */
fka_status fka_plan_create_contig(const fka_heads *heads, const fka_contig_desc *desc, fka_plan **out);

/*
 * One decode step: every branch's query attends to the shared prefix and to its
 * own suffix (Sec. 3.2, Sec. 3.3).
 *   q          bf16 [N][Hq][d]                  one new query token per branch
 *   prefix_k   bf16 [Hkv][Lp][d]                shared prefix keys (prefix_v likewise)
 *   suffix_k   bf16 [N][Hkv][suffix_cap][d]     per-branch suffix keys (suffix_v likewise)
 *   suffix_len int32 [N] (device)               valid suffix rows per branch, 0..max_suffix_len
 *   out        fp32 [N][Hq][d]                  attention output
 *   out_lse    fp32 [N][Hq] or NULL             natural-log log-sum-exp of the scaled scores
 * A sequence with no keys at all (Lp = 0 and suffix_len = 0) gets out = 0 and
 * out_lse = -inf.  Suffix rows at or past suffix_len[b] are never read.
 */
fka_status fka_fork_decode(const fka_plan *plan, const void *q, const void *prefix_k, const void *prefix_v,
                           const void *suffix_k, const void *suffix_v, const int32_t *suffix_len, float *out,
                           float *out_lse, void *stream);

/*
 * fka_fork_decode without a plan and without allocating: for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses that forbid
 * it).  heads and desc are those of fka_plan_create_contig, with share_prefix = 1; the
 * schedule is the one such a plan gets (the same blocks and rounds for the same desc, so
 * the same results bit for bit).  The partial results, the clamped lengths and a spare error
 * word live in a 16 MiB array of the library's own, one per device, which a device holds from
 * the first call on it until the process ends.  Nothing in it needs to start at zero, but
 * every call on a device uses the same array: calls that overlap on one device (two streams,
 * two threads) race and return garbage; order them.  The first call on each device looks up
 * the array's address; later ones touch no allocator at all.
 *   q ... out_lse   as in fka_fork_decode
 *   err             int32 (device) or NULL: the call ORs into *err the flag bits that
 *                   fka_plan_device_error describes (1: a suffix length was clamped); the
 *                   caller clears it
 * Errors: those of fka_plan_create_contig and fka_fork_decode; FKA_ERR_INVALID_ARG for
 * share_prefix = 0; FKA_ERR_UNSUPPORTED when the decode needs more than the 16 MiB (the
 * message says how much: (blocks x rounds + Hkv) x N x G x (d + 1) x 4 bytes of partials plus
 * 4 N + 256 bytes) or the device id is 64 or more.
 */
fka_status fka_fork_decode_noalloc(const fka_heads *heads, const fka_contig_desc *desc, const void *q,
                                   const void *prefix_k, const void *prefix_v, const void *suffix_k,
                                   const void *suffix_v, const int32_t *suffix_len, float *out, float *out_lse,
                                   int32_t *err, void *stream);

/*
 * Append one token per branch (each branch decodes its own continuation,
 * Sec. 3.2): for every branch b, K/V row suffix_len[b] of every KV head is set to
 * k_new[b] / v_new[b] and suffix_len[b] is incremented.  A branch already at
 * max_suffix_len is left unchanged and flagged (fka_plan_device_error).
 *   k_new, v_new bf16 [N][Hkv][d];  suffix_k/suffix_v/suffix_len as in fka_fork_decode.
 */
fka_status fka_append_kv(const fka_plan *plan, const void *k_new, const void *v_new, void *suffix_k,
                         void *suffix_v, int32_t *suffix_len, void *stream);

/* Append (as fka_append_kv) and then decode (as fka_fork_decode), fused into two
 * kernel launches: the merge stage scores each branch's new K/V row straight from
 * k_new / v_new as one more part of the log-sum-exp merge, and one block per branch
 * stores it at suffix_len[b] and increments suffix_len[b].  The caches and lengths end up as
 * after fka_append_kv; the outputs equal fka_append_kv + fka_fork_decode up to the
 * order of the fp32 sums. */
fka_status fka_fork_step(const fka_plan *plan, const void *q, const void *k_new, const void *v_new,
                         const void *prefix_k, const void *prefix_v, void *suffix_k, void *suffix_v,
                         int32_t *suffix_len, float *out, float *out_lse, void *stream);

/* ---------------------------------------------------------------------- paged KV */

/* Several independent forks ("groups", e.g. one per agent task) whose K/V live in
 * one pool of fixed-size pages.  Sequence i of group t shares the t-th prefix
 * pages with the other sequences of its group: within a group this is the fork of
 * Sec. 3.3 (every branch continues from the same snapshot, whose prefix K/V all of
 * them reuse), and the groups are the agent tasks served side by side.  The page
 * layout itself is a serving choice the paper leaves open. */
typedef struct {
    int32_t n_seqs;            /* S sequences over all groups */
    int32_t n_groups;          /* T groups */
    int32_t page_size;         /* tokens per page: 16 */
    int32_t max_pages_per_seq; /* columns of page_table */
    int32_t n_pool_pages;      /* pages in k_pool / v_pool; page ids outside [0, n_pool_pages) are never read */
    int32_t max_suffix_len;    /* upper bound on suffix_len[i] over the plan's lifetime */
    int32_t share_prefix;      /* 1 fork-aware, 0 naive baseline (as in fka_contig_desc) */
    int32_t rounds;            /* as in fka_contig_desc */
    int32_t blocks;            /* as in fka_contig_desc */
} fka_paged_desc;

/*
 * Build a plan for the paged layout.
 *   host_group_start      host int32 [n_groups + 1]: sequences of group t are
 *                         group_start[t] .. group_start[t+1]-1 (0 = start[0] <= ... = n_seqs)
 *   host_group_prefix_len host int32 [n_groups]: shared prefix length of each group
 * Page-table convention: logical position p < Lp of a sequence lives in page
 * page_table[i][p / page_size] at slot p % page_size; suffix position u starts on a
 * fresh page, at page index ceil(Lp / page_size) + u / page_size, slot u % page_size.
 * The sequences of one group hold the same prefix page ids.
 * Errors as fka_plan_create_contig; also FKA_ERR_INVALID_ARG when a group is empty,
 * page_size is not 16, or a group's prefix plus max_suffix_len needs more than
 * max_pages_per_seq pages.
 */
fka_status fka_plan_create_paged(const fka_heads *heads, const fka_paged_desc *desc, const int32_t *host_group_start,
                                 const int32_t *host_group_prefix_len, fka_plan **out);

/*
 * One decode step over the paged pool (Sec. 3.2 Overview: the branches of every fork
 * decode concurrently; Sec. 3.3: the prefix pages of a group are read once for all its
 * sequences).
 *   q          bf16 [S][Hq][d]
 *   k_pool     bf16 [n_pages][Hkv][page_size][d]   (v_pool likewise); a (page, head) block is contiguous
 *   page_table int32 [S][max_pages_per_seq] (device)
 *   suffix_len int32 [S] (device)
 *   out fp32 [S][Hq][d]; out_lse fp32 [S][Hq] or NULL
 * A page id outside [0, n_pool_pages) is not read: its rows count as zeros and
 * flag 4 is raised in the plan's device error word.
 */
fka_status fka_fork_decode_paged(const fka_plan *plan, const void *q, const void *k_pool, const void *v_pool,
                                 const int32_t *page_table, const int32_t *suffix_len, float *out, float *out_lse,
                                 void *stream);

/* Append one token per sequence into its pre-assigned suffix page (the caller
 * assigns suffix pages in page_table ahead of time), then increment suffix_len.
 *   k_new, v_new bf16 [S][Hkv][d]. */
fka_status fka_append_kv_paged(const fka_plan *plan, const void *k_new, const void *v_new, void *k_pool,
                               void *v_pool, const int32_t *page_table, int32_t *suffix_len, void *stream);

/* Fused append + decode over the paged pool (as fka_fork_step). */
fka_status fka_fork_step_paged(const fka_plan *plan, const void *q, const void *k_new, const void *v_new,
                               void *k_pool, void *v_pool, const int32_t *page_table, int32_t *suffix_len,
                               float *out, float *out_lse, void *stream);

/* Copy logical positions [0, out_len) of sequence `seq` out of the pool into
 * contiguous k_out / v_out bf16 [Hkv][out_len][d] (bit copies).  out_len counts
 * prefix plus suffix positions and must fit in max_pages_per_seq pages. */
fka_status fka_gather_paged(const fka_plan *plan, int32_t seq, const void *k_pool, const void *v_pool,
                            const int32_t *page_table, int32_t out_len, void *k_out, void *v_out, void *stream);

/* As fka_gather_paged for logical positions [begin, out_len) only: k_out / v_out bf16
 * [Hkv][out_len - begin][d].  0 <= begin <= out_len. */
fka_status fka_gather_paged_range(const fka_plan *plan, int32_t seq, int32_t begin, int32_t out_len,
                                  const void *k_pool, const void *v_pool, const int32_t *page_table, void *k_out,
                                  void *v_out, void *stream);

/* ------------------------------------------------ page pool: the K/V lifecycle of a fork */

/*
 * Host-side bookkeeping of the page ids [0, n_pages) of a paged K/V pool, one reference count per
 * page, following the lifecycle of a fork (Sec. 3.2 Overview; Sec. 3.3 Forking via Trajectory
 * Continuation; Sec. 3.5 Thought Harvesting):
 *   fork       every sequence of the group reads the snapshot's pages: one reference per page
 *              table row (fka_pool_fork);
 *   decode     a sequence takes a fresh page when its suffix reaches a page boundary; suffix
 *              position j of a sequence whose group prefix is Lp tokens is at page-table index
 *              ceil(Lp / 16) + j / 16, slot j % 16 (fka_pool_reserve, ahead of the appends);
 *   merge      the branches are terminated and their pages released (fka_pool_drop); what is
 *              harvested returns as text, so no branch K/V outlives the turn;
 *   next turn  the main sequence's context becomes the next snapshot, laid out densely
 *              (position p at index p / 16, slot p % 16): fka_pool_promote assigns the pages and
 *              fka_scatter_pages moves the K/V on the device.
 * Page tables here are host int32 arrays [rows][max_pages], -1 = no page; the caller copies the
 * rows it changed to the device table the kernels read.  A pool is not thread-safe.  Errors:
 * FKA_ERR_INVALID_ARG (a bad argument, or a page id that is not live), FKA_ERR_NOMEM (too few
 * free pages).  A call that fails changes nothing.
 */
typedef struct fka_pool fka_pool;

fka_status fka_pool_create(int32_t n_pages, fka_pool **out);
void fka_pool_destroy(fka_pool *pool);  /* NULL is ignored */

/* Free pages; -1 for a NULL pool. */
int32_t fka_pool_free_pages(const fka_pool *pool);

/* Reference count of `page` (0 = free); -1 for a NULL pool or an id outside [0, n_pages). */
int32_t fka_pool_refcount(const fka_pool *pool, int32_t page);

/* Take n free pages (count 1 each), lowest ids first, into ids[n]. */
fka_status fka_pool_alloc(fka_pool *pool, int32_t n, int32_t *ids);

/* One more / one less reference to each of ids[n]; every id must be live (an id may repeat as
 * often as it has references to drop).  A page whose count reaches 0 is free. */
fka_status fka_pool_retain(fka_pool *pool, int32_t n, const int32_t *ids);
fka_status fka_pool_release(fka_pool *pool, int32_t n, const int32_t *ids);

/* Fork: rows [first, first + n) of page_table, which must hold no pages, receive the snapshot's
 * page ids prefix_pages[n_prefix_pages] at indices [0, n_prefix_pages), one reference per row. */
fka_status fka_pool_fork(fka_pool *pool, const int32_t *prefix_pages, int32_t n_prefix_pages,
                         int32_t *page_table, int32_t max_pages, int32_t first, int32_t n);

/* Row `seq` (group prefix prefix_len tokens, whose ceil(prefix_len / 16) pages it holds) gets
 * pages for suffix positions [0, suffix_len): the missing ones are taken (count 1) and written at
 * indices ceil(prefix_len / 16) + j / 16.  *n_new (nullable) receives how many were taken. */
fka_status fka_pool_reserve(fka_pool *pool, int32_t *page_table, int32_t max_pages, int32_t seq,
                            int32_t prefix_len, int32_t suffix_len, int32_t *n_new);

/* Cancel or harvest row `seq`: one reference to each of its pages is released; the row becomes -1. */
fka_status fka_pool_drop(fka_pool *pool, int32_t *page_table, int32_t max_pages, int32_t seq);

/* Next snapshot from row `seq`, a context of prefix_len + suffix_len tokens in the fork layout.
 * dense[ceil((prefix_len + suffix_len) / 16)] receives page ids for the same context laid out
 * densely; the row's references move there and the row becomes -1.  Pages are reused where the
 * row holds the only reference: the full prefix pages keep their ids and positions; the last,
 * partly filled prefix page (unless shared) and the suffix pages are refilled in order; pages
 * left over are released and missing ones taken.  *from receives 16 * floor(prefix_len / 16):
 * positions [from, prefix_len + suffix_len) must be rewritten by fka_scatter_pages from a copy
 * gathered (fka_gather_paged_range) with the row's old device table before the scatter runs. */
fka_status fka_pool_promote(fka_pool *pool, int32_t *page_table, int32_t max_pages, int32_t seq,
                            int32_t prefix_len, int32_t suffix_len, int32_t *dense, int32_t *from);

/* Device copy of positions [from, len), held in k_src / v_src bf16 [n_kv_heads][len - from][head_dim]
 * (contiguous), into the pool bf16 [n_pool_pages][n_kv_heads][16][head_dim] at the dense layout
 * of page_row (device int32 [ceil(len / 16)]): position p goes to page page_row[p / 16], slot
 * p % 16.  Bit copies.  A page id outside [0, n_pool_pages) is skipped and bit 4 is or-ed into
 * *err (device int32; nullable).  Enqueued on `stream`. */
fka_status fka_scatter_pages(const void *k_src, const void *v_src, int32_t len, int32_t from,
                             const int32_t *page_row, int32_t n_kv_heads, int32_t head_dim, int32_t n_pool_pages,
                             void *k_pool, void *v_pool, int32_t *err, void *stream);

/* -------------------------------------------------------------- instruction prefill */

/* Branch-instruction prefill at the fork (Sec. 3.3: each branch continues from the snapshot
 * of the shared context followed by a short instruction of its own; Sec. 4.4: a branch's load
 * is dominated by prefill over the cached prefix).  Every branch b takes n_tokens instruction
 * tokens at once: token t's queries attend to the whole shared prefix and, causally, to b's
 * suffix up to and including its own position (suffix positions [0, suffix_len[b] + t]).
 * With head_dim 128 and at least 256 query rows (N x n_tokens x G) per KV head, a tiled kernel
 * runs: each KV head's rows are cut into units of 32 consecutive rows, a block of eight waves
 * takes eight units (one each) over one range of whole 64-key prefix tiles, which it loads once
 * into LDS for all eight, and the blocks of one KV head run on one XCD (the KV head varies
 * fastest in the grid) so that its ranges come from HBM once; the block of the last range also
 * reads the prefix's last prefix_len mod 64 keys and the suffix keys.  Otherwise the plan splits the tokens into units of consecutive tokens (at most
 * 32 query rows per KV head each for head_dim 128 with G <= 32, else 64), all streaming the same
 * prefix on the partial kernel, the blocks that read one prefix range for different units
 * together on one XCD (block vb holds work item vb mod n_items).  Then the merge stage combines
 * each row's partials. */
typedef struct {
    int32_t n_branches;      /* N, >= 1 */
    int32_t n_tokens;        /* n instruction tokens per branch, >= 1; N x n <= 512 */
    int32_t prefix_len;      /* Lp, >= 0 */
    int32_t suffix_cap;      /* rows of each branch's suffix buffer */
    int32_t max_suffix_len;  /* bound on suffix_len[b] + n_tokens, in [n_tokens, suffix_cap] */
    int32_t blocks;          /* 0 = automatic (fill the device); else about this many blocks */
} fka_prefill_desc;

/* Build an instruction-prefill plan (device workspace as fka_plan_create_contig).  Only
 * fka_prefill, fka_plan_get_info, fka_plan_device_error and fka_plan_destroy take it.
 * Errors: FKA_ERR_INVALID_ARG (null pointer, sizes out of range), FKA_ERR_UNSUPPORTED
 * (head_dim not 64/128, more than 64 query heads per KV head, more than 512 tokens),
 * FKA_ERR_NOMEM, FKA_ERR_HIP. */
fka_status fka_plan_create_prefill(const fka_heads *heads, const fka_prefill_desc *desc, fka_plan **out);

/*
 * Instruction prefill (two kernel launches: the partial kernel, then the merge).
 *   q          bf16 [N][n][Hq][d]                 the instruction tokens' queries
 *   prefix_k   bf16 [Hkv][Lp][d]                  shared prefix keys (prefix_v likewise)
 *   suffix_k   bf16 [N][Hkv][suffix_cap][d]       each branch's suffix followed by the keys of its
 *                                                 n instruction tokens at positions
 *                                                 [suffix_len[b], suffix_len[b] + n) (suffix_v likewise)
 *   suffix_len int32 [N] (device)                 each branch's suffix before the instruction; not
 *                                                 changed (the caller advances it by n afterwards);
 *                                                 a value outside [0, max_suffix_len - n] is
 *                                                 clamped into it and flagged (1)
 *   out        fp32 [N][n][Hq][d]                 attention output of every instruction token
 *   out_lse    fp32 [N][n][Hq] or NULL            natural-log log-sum-exp of its scaled scores
 * The plan's workspace is used: one stream at a time per plan.
 */
fka_status fka_prefill(const fka_plan *plan, const void *q, const void *prefix_k, const void *prefix_v,
                       const void *suffix_k, const void *suffix_v, const int32_t *suffix_len, float *out,
                       float *out_lse, void *stream);

/* The same prefill over the paged pool (the branches of one fork as in fka_fork_decode_paged):
 * branch b's row of page_table holds the shared prefix pages at indices [0, ceil(Lp / 16)) (the
 * same ids in every row) and its suffix position u at index ceil(Lp / 16) + u / 16, slot u % 16;
 * its n instruction tokens' keys and values are already in its pages at positions
 * [suffix_len[b], suffix_len[b] + n) (fka_pool_reserve, then fka_scatter_pages or appends). */
typedef struct {
    int32_t n_branches;         /* N, >= 1 */
    int32_t n_tokens;           /* n instruction tokens per branch, >= 1; N x n <= 512 */
    int32_t prefix_len;         /* Lp, >= 0 */
    int32_t page_size;          /* tokens per page: 16 */
    int32_t max_pages_per_seq;  /* columns of page_table; must hold ceil(Lp/16) + ceil(max_suffix_len/16) */
    int32_t n_pool_pages;       /* pages in k_pool / v_pool; ids outside [0, n_pool_pages) are never read */
    int32_t max_suffix_len;     /* bound on suffix_len[b] + n_tokens, >= n_tokens */
    int32_t blocks;             /* 0 = automatic (fill the device); else about this many blocks */
} fka_prefill_paged_desc;

/* Build a paged instruction-prefill plan.  Only fka_prefill_paged, fka_plan_get_info,
 * fka_plan_device_error and fka_plan_destroy take it.  Errors as fka_plan_create_prefill; also
 * FKA_ERR_INVALID_ARG when page_size is not 16 or the pages do not fit max_pages_per_seq. */
fka_status fka_plan_create_prefill_paged(const fka_heads *heads, const fka_prefill_paged_desc *desc,
                                         fka_plan **out);

/*
 * Instruction prefill over the paged pool (two kernel launches, as fka_prefill).
 *   q          bf16 [N][n][Hq][d]
 *   k_pool     bf16 [n_pages][Hkv][16][d]   (v_pool likewise)
 *   page_table int32 [N][max_pages_per_seq] (device), one row per branch
 *   suffix_len int32 [N] (device): each branch's suffix before the instruction; not changed; a
 *              value outside [0, max_suffix_len - n] is clamped into it and flagged (1)
 *   out        fp32 [N][n][Hq][d];  out_lse fp32 [N][n][Hq] or NULL
 * A page id outside [0, n_pool_pages) is not read (its rows count as zeros) and flag 4 is raised.
 */
fka_status fka_prefill_paged(const fka_plan *plan, const void *q, const void *k_pool, const void *v_pool,
                             const int32_t *page_table, const int32_t *suffix_len, float *out, float *out_lse,
                             void *stream);

/* -------------------------------------------------------------- stage entry points */

/* The first stage (Sec. 3.3: the prefix is read once for all branches) runs as one kernel
 * over work items: one per (prefix unit, KV head) -- a unit is a sequence group sharing its
 * prefix, or one sequence in the naive baseline.  An item's keys are the unit's prefix
 * (scored against all the unit's query rows) followed by each of its sequences' suffixes
 * (scored against that sequence's rows only), so the prefix and the suffix partial
 * attentions are one launch and one hook, fka_partials.  Every decode spreads the slices
 * (32 keys) of the items over n_blocks * rounds * waves_per_block waves: statically when
 * the plan has one unit (each item the same share), else in proportion to each item's
 * slices at the suffix lengths it finds on the device.  The waves of one block that work on
 * the same item share their slices and write one partial result per row to a slot;
 * fka_lse_merge is the second stage.  workspace_bytes is the plan's device memory. */
typedef struct {
    int32_t n_items;           /* units * n_kv_heads */
    int32_t n_units;           /* prefix-sharing units */
    int32_t waves_per_block;   /* waves of one block of the partial kernel */
    int32_t n_blocks;          /* blocks of the partial kernel per round */
    int32_t rounds;            /* the kernel runs n_blocks * rounds blocks */
    int32_t n_slots;           /* partial-result slots in the workspace (tiled prefill: one per prefix range) */
    int32_t slot_rows;         /* rows per slot: the largest item's query rows (tiled prefill: all
                                  N x n_tokens x Hq output rows) */
    int32_t static_split;      /* 1: one unit, items split statically */
    int32_t units_per_block;   /* instruction prefill: units a block takes: 8 on the tiled kernel, else
                                  1 or 2 (decode plans: 1) */
    size_t workspace_bytes;    /* device bytes held by the plan */
} fka_plan_info;

fka_status fka_plan_get_info(const fka_plan *plan, fka_plan_info *info);

/* One partial result written by the first stage: rows of sequences [seq0, seq0 + nseq)
 * x the G query heads of kv_head (row r = (s - seq0) * G + h % G).  Row r of sequence
 * s attends over prefix positions [prefix_begin, prefix_end) and over the slices
 * [suffix_begin, suffix_end) of the unit's suffix list that belong to s: the list holds,
 * for each sequence of the unit in order, its ceil(suffix_len / 32) slices of 32 suffix
 * positions (the last one partial).  prefix_len is the unit's prefix length. */
typedef struct {
    int32_t slot;
    int32_t seq0;
    int32_t nseq;
    int32_t kv_head;
    int32_t rows;
    int32_t prefix_begin;
    int32_t prefix_end;
    int32_t suffix_begin;
    int32_t suffix_end;
    int32_t prefix_len;
} fka_slot;

/* The slots a decode writes when the device holds the suffix lengths
 * host_suffix_len (host int32 [n_seqs]), computed on the host with the same
 * arithmetic as the kernels.  Fills up to `capacity` entries of `slots` and sets
 * *n_slots to the number of slots (which may exceed capacity). */
fka_status fka_plan_slots(const fka_plan *plan, const int32_t *host_suffix_len, fka_slot *slots, int32_t capacity,
                          int32_t *n_slots);

/*
 * Partial results of the first stage (test hook; the decode calls write the same
 * values to the plan's workspace).  For every slot listed by fka_plan_slots, rows
 * [0, rows) of slot `slot` hold the attention of those rows over the slot's keys:
 * o normalised, lse the natural-log log-sum-exp of the scaled scores, (0, -inf)
 * for a row without keys there.  Other slots and rows are left unwritten.
 *   part_o   fp32 [n_slots][slot_rows][d]
 *   part_lse fp32 [n_slots][slot_rows]
 */
fka_status fka_partials(const fka_plan *plan, const void *q, const void *prefix_k, const void *prefix_v,
                        const void *suffix_k, const void *suffix_v, const int32_t *suffix_len, float *part_o,
                        float *part_lse, void *stream);

/* As fka_partials for a paged plan (arguments as in fka_fork_decode_paged). */
fka_status fka_partials_paged(const fka_plan *plan, const void *q, const void *k_pool, const void *v_pool,
                              const int32_t *page_table, const int32_t *suffix_len, float *part_o,
                              float *part_lse, void *stream);

/*
 * Log-sum-exp merge of partial softmax results (combine attention over disjoint
 * key sets into attention over their union):
 *   M = max_p lse_p;  w_p = exp(lse_p - M);  o = sum_p w_p o_p / sum_p w_p;  lse = M + ln sum_p w_p
 * Parts with lse = -inf have weight 0; all parts empty gives o = 0, lse = -inf.
 *   part_o fp32 [n_parts][rows][d], part_lse fp32 [n_parts][rows]; out fp32 [rows][d];
 *   out_lse fp32 [rows] or NULL.  d must be 64 or 128.
 */
fka_status fka_lse_merge(int32_t rows, int32_t n_parts, int32_t head_dim, const float *part_o,
                         const float *part_lse, float *out, float *out_lse, void *stream);

/* ------------------------------------------------------------------ measurement */

/* Read-only streaming probe (the achievable read bandwidth of the device, a yardstick for the
 * partial kernel's K/V stream): `blocks` blocks of `threads` threads each read a contiguous
 * share of the device buffer buf[bytes] with non-temporal 16-byte loads, `unroll` loads in
 * flight per thread, and fold the words into a value written to sink (device uint32 [64]) only
 * in a case that practically never occurs.  bytes a positive multiple of 16, buf 16-byte
 * aligned, threads a multiple of 64 in [64, 1024], unroll 4, 8 or 16. */
fka_status fka_read_probe(const void *buf, size_t bytes, int32_t blocks, int32_t threads, int32_t unroll,
                          uint32_t *sink, void *stream);

/* Read and clear the plan's device error flag (synchronises with the device):
 * *flags receives a bit mask: 1 = a suffix length above max_suffix_len was
 * clamped, 2 = an append found no room (length at max_suffix_len or no page),
 * 4 = a page id outside the page table bounds was met, 8 = a merge record in
 * the plan's workspace pointed outside it (only if that memory was written from
 * outside the library; the record was not followed). */
fka_status fka_plan_device_error(const fka_plan *plan, int32_t *flags);

/* Release a plan and its device memory.  NULL is ignored. */
void fka_plan_destroy(fka_plan *plan);

#ifdef __cplusplus
}
#endif

#endif /* FORKATTN_H */
