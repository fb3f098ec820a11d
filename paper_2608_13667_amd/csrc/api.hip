// C ABI of libforkattn.so: argument validation, plans (schedule tables and
// workspaces) and kernel launches.  Declared in include/forkattn.h.
#include <algorithm>
#include <array>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <set>
#include <vector>

#include "forkattn.h"
#include "internal.h"

struct fka_plan {
    bool paged = false;
    int32_t Hq = 0, Hkv = 0, d = 0, G = 0;
    float scale = 0.f;
    int32_t n_seqs = 0;
    int32_t share_prefix = 1;
    int32_t prefill_n = 0;     // instruction prefill plan: tokens per branch (sequences are b * n + t)
    int32_t n_branches = 0;    // instruction prefill plan: branches
    int32_t prefill_groups = 1; // instruction prefill plan: units per block
    // instruction prefill on the tiled kernel (head_dim 128): 32-row units per KV head, blocks of
    // eight units, prefix ranges, prefix tiles of 64 keys, tiles of balance left to the suffix keys
    bool prefill_tiles = false;
    int32_t tile_units = 0, tile_unit_groups = 0, tile_ranges = 0, tile_prefix = 0, tile_reserve = 0;
    int32_t max_suffix_len = 0;
    // contiguous
    int32_t prefix_len = 0, suffix_cap = 0;
    // paged
    int32_t n_groups = 0, page_size = 0, max_pages = 0, n_pool_pages = 0;
    std::vector<int32_t> group_start, group_prefix_len;
    // schedule (see the work schedule in internal.h)
    std::vector<fka::UnitRec> units;       // prefix-sharing units in sequence order
    std::vector<int32_t> seq_prefix_len;   // prefix length of s's unit
    int32_t ps_total = 0;      // prefix slices of all units
    bool static_split = false; // one unit: items split statically
    int32_t n_items = 0;       // units * Hkv
    int32_t slot_rows = 0;     // rows of the largest item
    int32_t row_tiles = 1;
    int32_t waves = 0;         // waves per block of the partial kernel
    int32_t n_blocks = 0;      // blocks launched per round (at most those resident at once)
    int32_t rounds = 1;        // launches n_blocks * rounds blocks
    int32_t n_slots = 0;       // partial-result slots in the workspace
    size_t workspace_bytes = 0;
    int device = 0;
    // device memory (one allocation, carved)
    void *mem = nullptr;
    fka::UnitRec *d_units = nullptr;
    int32_t *d_seq_prefix_len = nullptr;
    int32_t *err = nullptr;
    int32_t *d_rowrec = nullptr;
    int32_t *d_lens = nullptr;
    float *part_o = nullptr;
    float *part_lse = nullptr;
};

// Page pool: reference count per page id; free ids kept ordered so allocation takes the lowest.
struct fka_pool {
    std::vector<int32_t> ref;
    std::set<int32_t> free_ids;
    std::vector<int32_t> pending;  // references a call is about to drop, per page (zero between calls)
    std::vector<int32_t> touched;  // pages with a pending count
};

// Scratch of the no-allocation decode, one copy per device (see scratch_of below).
constexpr size_t kScratchBytes = size_t(16) << 20;
static __device__ __align__(256) char scratch[kScratchBytes];

namespace {

thread_local char g_err[512] = "";

fka_status fail(fka_status st, const char *fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return st;
}

fka_status ok()
{
    g_err[0] = '\0';
    return FKA_OK;
}

fka_status hip_fail(hipError_t e, const char *what)
{
    return fail(FKA_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool aligned4(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }

#define REQUIRE(cond, ...)                                  \
    do {                                                    \
        if (!(cond)) return fail(FKA_ERR_INVALID_ARG, __VA_ARGS__); \
    } while (0)

#define REQUIRE_PTR16(p)                                                          \
    do {                                                                          \
        if (!(p)) return fail(FKA_ERR_INVALID_ARG, "%s is null", #p);             \
        if (!aligned16(p)) return fail(FKA_ERR_INVALID_ARG, "%s is not 16-byte aligned", #p); \
    } while (0)

// int32 / fp32 arrays: non-null and 4-byte aligned (REQUIRE_OPT4: or null)
#define REQUIRE_PTR4(p)                                                           \
    do {                                                                          \
        if (!(p)) return fail(FKA_ERR_INVALID_ARG, "%s is null", #p);             \
        if (!aligned4(p)) return fail(FKA_ERR_INVALID_ARG, "%s is not 4-byte aligned", #p); \
    } while (0)
#define REQUIRE_OPT4(p)                                                           \
    do {                                                                          \
        if ((p) && !aligned4(p)) return fail(FKA_ERR_INVALID_ARG, "%s is not 4-byte aligned", #p); \
    } while (0)

fka_status check_heads(const fka_heads *h)
{
    REQUIRE(h != nullptr, "heads is null");
    REQUIRE(h->n_q_heads > 0 && h->n_kv_heads > 0, "head counts must be positive");
    REQUIRE(h->n_q_heads % h->n_kv_heads == 0, "n_q_heads (%d) is not a multiple of n_kv_heads (%d)",
            h->n_q_heads, h->n_kv_heads);
    REQUIRE(std::isfinite(h->softmax_scale) && h->softmax_scale >= 0.f, "softmax_scale must be finite and >= 0");
    if (h->head_dim != 64 && h->head_dim != 128)
        return fail(FKA_ERR_UNSUPPORTED, "head_dim %d not supported (64 or 128)", h->head_dim);
    return FKA_OK;
}

int32_t ceil_div(int64_t a, int64_t b) { return (int32_t)((a + b - 1) / b); }

void init_heads(fka_plan *p, const fka_heads *h)
{
    p->Hq = h->n_q_heads;
    p->Hkv = h->n_kv_heads;
    p->d = h->head_dim;
    p->G = p->Hq / p->Hkv;
    p->scale = h->softmax_scale > 0.f ? h->softmax_scale : 1.0f / std::sqrt((float)h->head_dim);
}

fka_status check_grid(int32_t rounds, int32_t blocks)
{
    REQUIRE(rounds >= 0 && rounds <= 64, "rounds (%d) must be in [0, 64]", rounds);
    REQUIRE(blocks >= 0, "blocks (%d) must be >= 0", blocks);
    return FKA_OK;
}

// Slices of work a wave takes at the least before the automatic grid uses another block:
// a small fork then runs on a few blocks (fewer partials for the merge) instead of the whole
// device.
constexpr int32_t kMinSlicesPerWave = 2;

// The grid for a schedule with n_units units of at most max_nseq sequences and est slices per
// KV head with every suffix at max_suffix_len: slot geometry, blocks, rounds and slots.  Touches
// no memory beyond the plan's fields (the no-allocation decode calls it too).
fka_status set_grid(fka_plan *p, int64_t est, int32_t max_nseq, int32_t n_units, int32_t rounds_req, int32_t blocks_req)
{
    // the schedule's total slices (every item at its longest, over all KV heads) stay in int32
    if (est * p->Hkv > (int64_t)1 << 30)
        return fail(FKA_ERR_UNSUPPORTED, "prefix and suffixes of %lld slices are too long", (long long)(est * p->Hkv));
    p->static_split = n_units == 1;
    p->n_items = n_units * p->Hkv;
    p->slot_rows = max_nseq * p->G;
    p->row_tiles = ceil_div(p->slot_rows, 16);

    hipError_t e = hipGetDevice(&p->device);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    int cus = 0;
    if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, p->device)) != hipSuccess)
        return hip_fail(e, "hipDeviceGetAttribute");
    const int per_cu = fka::partials_blocks_per_cu(p->d, p->row_tiles, p->paged);
    p->waves = fka::partials_waves_per_block(p->d, p->row_tiles, p->paged);
    if (per_cu <= 0 || p->waves <= 0) return fail(FKA_ERR_HIP, "occupancy query of the partial kernel failed");
    const int32_t resident = cus * per_cu;
    if (blocks_req > 0) {
        p->n_blocks = std::min(blocks_req, resident);
    } else {
        // enough blocks that every wave has kMinSlicesPerWave slices at the longest suffixes,
        // a multiple of Hkv (so that items start on block boundaries), at most the resident ones
        int64_t b = (est * p->Hkv + (int64_t)p->waves * kMinSlicesPerWave - 1) / ((int64_t)p->waves * kMinSlicesPerWave);
        b = (b + p->Hkv - 1) / p->Hkv * p->Hkv;
        p->n_blocks = (int32_t)std::max<int64_t>(1, std::min<int64_t>(b, resident));
    }
    // at least two workers per item, so that A = workers - non-empty items stays >= half
    const int32_t per_round = p->n_blocks * p->waves;
    const int32_t need = ceil_div(2 * (int64_t)p->n_items, per_round);
    p->rounds = std::max<int32_t>(std::max<int32_t>(1, need), rounds_req);
    p->n_slots = p->n_blocks * p->rounds + p->n_items;
    return FKA_OK;
}

// token counts stay far enough below 2^31 that ceil(tokens / kSlice) cannot overflow
constexpr int32_t kMaxTokens = 1 << 30;

// Prefix units in order: unit u covers sequences [seq0, seq0 + nseq) that share a prefix of
// n_tok tokens.  Builds the unit table, the per-sequence prefix lengths, the slot geometry,
// the grid and the round count.
fka_status build_schedule(fka_plan *p, const std::vector<std::array<int32_t, 3>> &units, int32_t rounds_req,
                          int32_t blocks_req)
{
    p->units.clear();
    p->seq_prefix_len.assign(p->n_seqs, 0);
    if (p->max_suffix_len > kMaxTokens)
        return fail(FKA_ERR_UNSUPPORTED, "max_suffix_len %d is too long (limit %d)", p->max_suffix_len, kMaxTokens);
    for (const auto &u : units)
        if (u[2] > kMaxTokens) return fail(FKA_ERR_UNSUPPORTED, "prefix of %d tokens is too long (limit %d)", u[2], kMaxTokens);
    int64_t c = 0;
    int32_t max_nseq = 1;
    int64_t est = 0;  // slices per KV head with every suffix at max_suffix_len
    for (size_t u = 0; u < units.size(); ++u) {
        const int32_t seq0 = units[u][0], nseq = units[u][1], n_tok = units[u][2];
        max_nseq = std::max(max_nseq, nseq);
        for (int32_t i = seq0; i < seq0 + nseq; ++i) p->seq_prefix_len[i] = n_tok;
        fka::UnitRec r{};
        r.seq0 = seq0;
        r.nseq = nseq;
        r.plen = n_tok;
        r.ps_before = (int32_t)c;
        p->units.push_back(r);
        c += fka::slices_of(n_tok);
        est += fka::slices_of(n_tok) + (int64_t)nseq * fka::slices_of(p->max_suffix_len);
    }
    p->ps_total = (int32_t)c;
    return set_grid(p, est, max_nseq, (int32_t)units.size(), rounds_req, blocks_req);
}

// Allocate device memory for the unit table, the error flag, the merge records, the lengths
// and the partial-result workspace, and upload the tables.
fka_status finish_plan(fka_plan *p)
{
    hipError_t e;
    auto up = [](size_t x) { return (x + 255) & ~size_t(255); };
    const size_t rows = (size_t)p->n_seqs * p->Hq;
    const size_t b_units = up(std::max<size_t>(1, p->units.size()) * sizeof(fka::UnitRec));
    const size_t b_seq = up((size_t)p->n_seqs * sizeof(int32_t));
    const size_t b_err = 256;
    const size_t b_rec = up(rows * fka::kRowRec * sizeof(int32_t));
    const size_t b_po = up((size_t)p->n_slots * p->slot_rows * p->d * sizeof(float));
    // the merge addresses the partials with 32-bit byte offsets
    if (b_po >= ((size_t)1 << 31))
        return fail(FKA_ERR_UNSUPPORTED, "partial results of %zu bytes exceed the 2 GiB the merge addresses", b_po);
    const size_t b_pl = up((size_t)p->n_slots * p->slot_rows * sizeof(float));
    const size_t b_zero = b_err + b_rec + b_seq;  // err, records, lengths: zeroed
    const size_t total = b_units + b_seq + b_zero + b_po + b_pl;
    e = hipMalloc(&p->mem, total);
    if (e != hipSuccess) {
        p->mem = nullptr;
        (void)hipGetLastError();
        return fail(FKA_ERR_NOMEM, "hipMalloc(%zu) failed: %s", total, hipGetErrorString(e));
    }
    char *m = static_cast<char *>(p->mem);
    p->d_units = reinterpret_cast<fka::UnitRec *>(m);
    m += b_units;
    p->d_seq_prefix_len = reinterpret_cast<int32_t *>(m);
    m += b_seq;
    char *zero = m;
    p->err = reinterpret_cast<int32_t *>(m);
    m += b_err;
    p->d_rowrec = reinterpret_cast<int32_t *>(m);
    m += b_rec;
    p->d_lens = reinterpret_cast<int32_t *>(m);
    m += b_seq;
    p->part_o = reinterpret_cast<float *>(m);
    m += b_po;
    p->part_lse = reinterpret_cast<float *>(m);
    p->workspace_bytes = total;
    auto put = [&](void *dst, const void *src, size_t bytes, const char *what) -> fka_status {
        if (bytes == 0) return FKA_OK;
        const hipError_t r = hipMemcpy(dst, src, bytes, hipMemcpyHostToDevice);
        return r == hipSuccess ? FKA_OK : hip_fail(r, what);
    };
    fka_status st;
    if ((st = put(p->d_units, p->units.data(), p->units.size() * sizeof(fka::UnitRec), "hipMemcpy(units)")) != FKA_OK ||
        (st = put(p->d_seq_prefix_len, p->seq_prefix_len.data(), p->seq_prefix_len.size() * sizeof(int32_t),
                  "hipMemcpy(sequence tables)")) != FKA_OK)
        return st;
    if ((e = hipMemset(zero, 0, b_zero)) != hipSuccess) return hip_fail(e, "hipMemset(flags and records)");
    return FKA_OK;
}

fka_status check_contig(const fka_heads *heads, const fka_contig_desc *desc)
{
    fka_status st = check_heads(heads);
    if (st != FKA_OK) return st;
    REQUIRE(desc != nullptr, "desc is null");
    REQUIRE(desc->n_branches >= 1, "n_branches (%d) must be >= 1", desc->n_branches);
    REQUIRE(desc->prefix_len >= 0, "prefix_len (%d) must be >= 0", desc->prefix_len);
    REQUIRE(desc->suffix_cap >= 1, "suffix_cap (%d) must be >= 1", desc->suffix_cap);
    REQUIRE(desc->max_suffix_len >= 0 && desc->max_suffix_len <= desc->suffix_cap,
            "max_suffix_len (%d) must be in [0, suffix_cap=%d]", desc->max_suffix_len, desc->suffix_cap);
    REQUIRE(desc->share_prefix == 0 || desc->share_prefix == 1, "share_prefix must be 0 or 1");
    if ((st = check_grid(desc->rounds, desc->blocks)) != FKA_OK) return st;
    if (desc->n_branches > fka::kMaxSeqs)
        return fail(FKA_ERR_UNSUPPORTED, "%d sequences exceed the limit of %d", desc->n_branches, fka::kMaxSeqs);
    const int G = heads->n_q_heads / heads->n_kv_heads;
    const int rows = (desc->share_prefix ? desc->n_branches : 1) * G;
    if (G > fka::kMaxRows || rows > fka::kMaxRows)
        return fail(FKA_ERR_UNSUPPORTED, "%d query rows per KV head exceed the limit of %d", rows, fka::kMaxRows);
    return FKA_OK;
}

fka::AttnArgs attn_args(const fka_plan *p)
{
    fka::AttnArgs a{};
    a.units = p->d_units;
    a.n_units = (int32_t)p->units.size();
    a.static_split = p->static_split ? 1 : 0;
    a.ps_total = p->ps_total;
    a.seq_prefix_len = p->d_seq_prefix_len;
    a.rowrec = p->d_rowrec;
    a.lens = p->d_lens;
    a.max_suffix_len = p->max_suffix_len;
    a.n_seqs = p->n_seqs;
    a.n_q_heads = p->Hq;
    a.n_kv_heads = p->Hkv;
    a.group = p->G;
    a.scale_log2 = p->scale * 1.4426950408889634f;
    a.part_o = p->part_o;
    a.part_lse = p->part_lse;
    a.slot_rows = p->slot_rows;
    a.n_slots = p->n_slots;
    a.err = p->err;
    // contiguous: the prefix buffer's length; a static split also takes its one unit's prefix
    // length from here (paged with one group)
    a.prefix_len = p->paged ? p->units[0].plen : p->prefix_len;
    a.suffix_cap = p->suffix_cap;
    a.max_pages = p->max_pages;
    a.n_pool_pages = p->n_pool_pages;
    a.paged = p->paged ? 1 : 0;
    a.prefill_groups = p->prefill_groups;
    return a;
}

fka::MergeArgs merge_args(const fka_plan *p, const int32_t *suffix_len, float *out, float *out_lse)
{
    fka::MergeArgs m{};
    m.part_o = p->part_o;
    m.part_lse = p->part_lse;
    m.out = out;
    m.out_lse = out_lse;
    m.rows = p->n_seqs * p->Hq;
    m.n_q_heads = p->Hq;
    m.n_parts = 0;
    m.plan = 1;
    m.static_split = p->static_split ? 1 : 0;
    m.rowrec = p->d_rowrec;
    m.lens = p->d_lens;
    m.slot_rows = p->slot_rows;
    m.n_slots = p->n_slots;
    m.waves = p->waves;
    m.n_workers = p->n_blocks * p->rounds * p->waves;
    m.suffix_len = const_cast<int32_t *>(suffix_len);  // only a fused step writes it
    m.max_suffix_len = p->max_suffix_len;
    m.err = p->err;
    m.seq_prefix_len = p->d_seq_prefix_len;
    m.suffix_cap = p->suffix_cap;
    m.max_pages = p->max_pages;
    m.n_pool_pages = p->n_pool_pages;
    m.n_kv_heads = p->Hkv;
    m.paged = p->paged ? 1 : 0;
    m.scale = p->scale;
    m.group = p->G;
    return m;
}

fka_status run_decode(const fka_plan *p, const fka::AttnArgs &a, const int32_t *suffix_len, float *out,
                      float *out_lse, hipStream_t s, const fka::MergeArgs *step = nullptr)
{
    hipError_t e = fka::launch_partials(a, p->n_blocks * p->rounds, p->d, p->row_tiles, s);
    if (e != hipSuccess) return hip_fail(e, "partials kernel launch");
    e = fka::launch_merge(step ? *step : merge_args(p, suffix_len, out, out_lse), p->d, s);
    if (e != hipSuccess) return hip_fail(e, "merge kernel launch");
    return ok();
}

// The instruction prefill's two launches: the tiled kernel (head_dim 128) with the merge in its
// explicit mode (every row merges its ranges' partials), or the partial kernel's prefill
// instantiation with the plan-mode merge.
fka_status run_prefill(const fka_plan *p, const fka::AttnArgs &a, float *out, float *out_lse, hipStream_t s)
{
    hipError_t e;
    if (p->prefill_tiles) {
        fka::PrefillArgs t{};
        t.q = a.q;
        t.prefix_k = a.prefix_k;
        t.prefix_v = a.prefix_v;
        t.suffix_k = a.suffix_k;
        t.suffix_v = a.suffix_v;
        t.k_pool = a.k_pool;
        t.v_pool = a.v_pool;
        t.page_table = a.page_table;
        t.suffix_len = a.suffix_len;
        t.part_o = p->part_o;
        t.part_lse = p->part_lse;
        t.err = p->err;
        t.n_branches = p->n_branches;
        t.n_tokens = p->prefill_n;
        t.prefix_len = p->prefix_len;
        t.suffix_cap = p->suffix_cap;
        t.max_suffix_len = p->max_suffix_len;
        t.max_pages = p->max_pages;
        t.n_pool_pages = p->n_pool_pages;
        t.paged = p->paged ? 1 : 0;
        t.n_q_heads = p->Hq;
        t.n_kv_heads = p->Hkv;
        t.group = p->G;
        t.n_units = p->tile_units;
        t.unit_groups = p->tile_unit_groups;
        t.ranges = p->tile_ranges;
        t.prefix_tiles = p->tile_prefix;
        t.tail_reserve = p->tile_reserve;
        t.scale_log2 = p->scale * 1.4426950408889634f;
        e = fka::launch_prefill_tiles(t, p->n_blocks, s);
        if (e != hipSuccess) return hip_fail(e, "prefill kernel launch");
        fka::MergeArgs m{};
        m.part_o = p->part_o;
        m.part_lse = p->part_lse;
        m.out = out;
        m.out_lse = out_lse;
        m.rows = p->n_seqs * p->Hq;
        m.n_q_heads = p->Hq;
        m.n_parts = p->tile_ranges;
        m.plan = 0;
        m.err = p->err;
        e = fka::launch_merge(m, p->d, s);
        if (e != hipSuccess) return hip_fail(e, "merge kernel launch");
        return ok();
    }
    e = fka::launch_prefill(a, p->n_blocks, p->d, p->row_tiles, s);
    if (e != hipSuccess) return hip_fail(e, "prefill kernel launch");
    e = fka::launch_merge(merge_args(p, a.suffix_len, out, out_lse), p->d, s);
    if (e != hipSuccess) return hip_fail(e, "merge kernel launch");
    return ok();
}

// ---------------------------------------------------------------------------------------
// Scratch of the no-allocation decode (fka_fork_decode_noalloc): the device memory one decode
// needs beyond its inputs and outputs -- the partial results, the clamped lengths and an error
// word -- in a file-scope array, so that the call allocates nothing.  Each device holds its own
// copy from the library's load until the process ends.  Host code reaches it only through the
// device address hipGetSymbolAddress returns (the array's name is a host-side stand-in).
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
char *g_scratch_ptr[kMaxDevices];  // device address of each device's scratch, once looked up

// This device's scratch address, looked up on the first call on the device (which is current).
fka_status scratch_of(int device, char **out)
{
    if (device < 0 || device >= kMaxDevices)
        return fail(FKA_ERR_UNSUPPORTED, "device %d: the no-allocation decode serves devices 0..%d", device, kMaxDevices - 1);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[device]) {
        void *ptr = nullptr;
        const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
        if (!ptr) return fail(FKA_ERR_HIP, "hipGetSymbolAddress(scratch) returned null");
        g_scratch_ptr[device] = static_cast<char *>(ptr);
    }
    *out = g_scratch_ptr[device];
    return FKA_OK;
}

// The layout of a prefill plan's suffix keys: contiguous buffers of cap rows, or the page pool.
struct PrefillLayout {
    bool paged;
    int32_t cap;        // contiguous: rows of each branch's suffix buffer
    int32_t max_pages;  // paged: columns of the page table
    int32_t n_pool_pages;
};

fka_status create_prefill(const fka_heads *heads, int32_t N, int32_t n, int32_t Lp, int32_t max_suffix_len,
                          int32_t blocks, const PrefillLayout &lay, fka_plan **out)
{
    const int64_t S = (int64_t)N * n;  // virtual sequences
    if (S > fka::kMaxSeqs)
        return fail(FKA_ERR_UNSUPPORTED, "%lld instruction tokens (n_branches x n_tokens) exceed the limit of %d",
                    (long long)S, fka::kMaxSeqs);
    const int G = heads->n_q_heads / heads->n_kv_heads;
    if (G > fka::kMaxRows)
        return fail(FKA_ERR_UNSUPPORTED, "%d query heads per KV head exceed the limit of %d", G, fka::kMaxRows);
    if (Lp > kMaxTokens || max_suffix_len > kMaxTokens)
        return fail(FKA_ERR_UNSUPPORTED, "prefix or suffix longer than %d tokens", kMaxTokens);

    fka_plan *p = new (std::nothrow) fka_plan();
    if (!p) return fail(FKA_ERR_NOMEM, "host allocation failed");
    auto bail = [&](fka_status e) {
        fka_plan_destroy(p);
        return e;
    };
    init_heads(p, heads);
    p->prefill_n = n;
    p->n_branches = N;
    p->n_seqs = (int32_t)S;
    p->share_prefix = 1;
    p->prefix_len = Lp;
    p->max_suffix_len = max_suffix_len;
    p->paged = lay.paged;
    if (lay.paged) {
        p->n_groups = 1;
        p->page_size = fka::kPageSize;
        p->max_pages = lay.max_pages;
        p->n_pool_pages = lay.n_pool_pages;
    } else {
        p->suffix_cap = lay.cap;
    }
    hipError_t e = hipGetDevice(&p->device);
    if (e != hipSuccess) return bail(hip_fail(e, "hipGetDevice"));
    int cus = 0;
    if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, p->device)) != hipSuccess)
        return bail(hip_fail(e, "hipDeviceGetAttribute"));
    // The tiled kernel when each KV head has at least one block's worth of units (eight of 32
    // rows); fewer rows than that leave most of a block's waves idle there, and the partial kernel's
    // prefill instantiation, which spreads each unit's keys over four waves, is faster.
    const int tile_rows = fka::prefill_tiles_unit_rows(), tile_waves = fka::prefill_tiles_waves();
    if (p->d == 128 && S * G >= (int64_t)tile_waves * tile_rows) {
        // The tiled kernel: units of 32 consecutive rows of a KV head, eight per block (one per
        // wave) over one range of whole 64-key prefix tiles; R ranges fill the device, and the
        // last range's share is shortened by the keys it also reads per wave: the prefix's last
        // Lp mod 64 and the suffix keys, taken as the instruction itself (the branches' suffixes
        // are empty at the fork); a 32-key tile, read without prefetch, is counted as one 64-key
        // prefix tile.
        const int per_cu = fka::prefill_tiles_blocks_per_cu(lay.paged);
        if (per_cu <= 0) return bail(fail(FKA_ERR_HIP, "occupancy query of the prefill kernel failed"));
        const int64_t rows_head = S * G;
        const int32_t U = (int32_t)ceil_div(rows_head, tile_rows);
        const int32_t UG = ceil_div(U, tile_waves);
        const int32_t PT = Lp / 64;  // whole tiles; the last range reads the rest per wave
        const int64_t base = (int64_t)p->Hkv * UG;
        const int64_t want = blocks > 0 ? blocks : (int64_t)cus * per_cu;
        int64_t R = std::max<int64_t>(1, want / base);
        R = std::min<int64_t>(R, std::max(1, PT));
        // the partials of one range: S Hq rows of d floats; the ranges together stay below 256 MiB
        const int64_t range_bytes = S * p->Hq * (int64_t)p->d * 4;
        R = std::max<int64_t>(1, std::min<int64_t>(R, ((int64_t)256 << 20) / range_bytes));
        p->prefill_tiles = true;
        p->tile_units = U;
        p->tile_unit_groups = UG;
        p->tile_ranges = (int32_t)R;
        p->tile_prefix = PT;
        p->tile_reserve = (int32_t)std::min<int64_t>(ceil_div(n, 32) + (Lp % 64 != 0), PT / (2 * R));
        for (int32_t u = 0; u < U; ++u) {
            fka::UnitRec r{};
            r.seq0 = (int32_t)(((int64_t)u * tile_rows) / G);
            r.nseq = (int32_t)((std::min<int64_t>(rows_head, (int64_t)u * tile_rows + tile_rows) - 1) / G) - r.seq0 + 1;
            r.plen = Lp;
            p->units.push_back(r);
        }
        p->seq_prefix_len.assign(p->n_seqs, Lp);
        p->static_split = false;
        p->n_items = U * p->Hkv;
        p->slot_rows = (int32_t)(S * p->Hq);
        p->row_tiles = tile_rows / 16;
        p->waves = tile_waves;
        p->prefill_groups = tile_waves;
        p->n_blocks = (int32_t)(base * R);
        p->rounds = 1;
        p->n_slots = (int32_t)R;
        fka_status st = finish_plan(p);
        if (st != FKA_OK) return bail(st);
        *out = p;
        return ok();
    }
    // Units of consecutive instruction tokens, at most prefill_max_rows query rows each (32 for
    // d = 128: two waves per SIMD), all over the one prefix: as few as that allows.  Each unit's
    // waves load every prefix tile once more (from L2) and score it against the unit's 16-row
    // tiles, so taller units keep the matrix cores busy per byte loaded.  Each set of P units of
    // one KV head then takes B = resident / sets blocks (at least one); with the sets a multiple
    // of the 8 XCDs the blocks of a KV head all run on one XCD and share its prefix tiles in L2.
    const int32_t best_U = ceil_div(S, fka::prefill_max_rows(p->d, G) / G);
    const int32_t best_tiles = ceil_div(ceil_div(S, best_U) * G, 16);
    const int per_cu = fka::prefill_blocks_per_cu(p->d, best_tiles, lay.paged);
    if (per_cu <= 0) return bail(fail(FKA_ERR_HIP, "occupancy query of the prefill kernel failed"));
    const int64_t items = (int64_t)best_U * p->Hkv;
    const int64_t resident = (int64_t)cus * per_cu;
    // Units per block: when the items alone would need more blocks than are resident at once (a
    // second round would fetch the prefix from HBM again), an eight-wave block takes two units of
    // one KV head, four waves each, over the same prefix range.
    const int waves = fka::prefill_waves_per_block(p->d, best_tiles, lay.paged);
    const int32_t P = (waves == 8 && p->d == 128 && items > resident && best_U > 1) ? 2 : 1;
    const int64_t sets = (int64_t)ceil_div(best_U, P) * p->Hkv;
    const int32_t best_B = (int32_t)(blocks > 0 ? std::max<int64_t>(1, blocks / sets)
                                               : std::max<int64_t>(1, resident / sets));
    const int32_t U = best_U;
    int32_t max_nseq = 0;
    for (int32_t u = 0; u < U; ++u) {
        fka::UnitRec r{};
        r.seq0 = (int32_t)(u * S / U);
        r.nseq = (int32_t)((u + 1) * S / U) - r.seq0;
        r.plen = Lp;
        r.ps_before = u * fka::slices_of(Lp);
        max_nseq = std::max(max_nseq, r.nseq);
        p->units.push_back(r);
    }
    p->seq_prefix_len.assign(p->n_seqs, Lp);
    p->ps_total = U * fka::slices_of(Lp);
    p->static_split = false;
    p->n_items = U * p->Hkv;
    p->slot_rows = max_nseq * G;
    p->row_tiles = best_tiles;
    p->waves = waves;
    p->prefill_groups = P;
    p->n_blocks = (int32_t)(best_B * sets);
    p->rounds = 1;
    p->n_slots = best_B * p->n_items;
    fka_status st = finish_plan(p);
    if (st != FKA_OK) return bail(st);
    *out = p;
    return ok();
}

}  // namespace

extern "C" {

int fka_version(void) { return 20000; }

const char *fka_last_error(void) { return g_err; }

fka_status fka_plan_create_contig(const fka_heads *heads, const fka_contig_desc *desc, fka_plan **out)
{
    REQUIRE(out != nullptr, "out is null");
    *out = nullptr;
    fka_status st = check_contig(heads, desc);
    if (st != FKA_OK) return st;

    fka_plan *p = new (std::nothrow) fka_plan();
    if (!p) return fail(FKA_ERR_NOMEM, "host allocation failed");
    init_heads(p, heads);
    p->n_seqs = desc->n_branches;
    p->share_prefix = desc->share_prefix;
    p->prefix_len = desc->prefix_len;
    p->suffix_cap = desc->suffix_cap;
    p->max_suffix_len = desc->max_suffix_len;
    std::vector<std::array<int32_t, 3>> units;
    if (desc->share_prefix)
        units.push_back({0, desc->n_branches, desc->prefix_len});
    else
        for (int b = 0; b < desc->n_branches; ++b) units.push_back({b, 1, desc->prefix_len});
    if ((st = build_schedule(p, units, desc->rounds, desc->blocks)) != FKA_OK || (st = finish_plan(p)) != FKA_OK) {
        fka_plan_destroy(p);
        return st;
    }
    *out = p;
    return ok();
}

fka_status fka_plan_create_prefill(const fka_heads *heads, const fka_prefill_desc *desc, fka_plan **out)
{
    REQUIRE(out != nullptr, "out is null");
    *out = nullptr;
    fka_status st = check_heads(heads);
    if (st != FKA_OK) return st;
    REQUIRE(desc != nullptr, "desc is null");
    REQUIRE(desc->n_branches >= 1, "n_branches (%d) must be >= 1", desc->n_branches);
    REQUIRE(desc->n_tokens >= 1, "n_tokens (%d) must be >= 1", desc->n_tokens);
    REQUIRE(desc->prefix_len >= 0, "prefix_len (%d) must be >= 0", desc->prefix_len);
    REQUIRE(desc->suffix_cap >= 1, "suffix_cap (%d) must be >= 1", desc->suffix_cap);
    REQUIRE(desc->max_suffix_len >= desc->n_tokens && desc->max_suffix_len <= desc->suffix_cap,
            "max_suffix_len (%d) must be in [n_tokens=%d, suffix_cap=%d]", desc->max_suffix_len, desc->n_tokens,
            desc->suffix_cap);
    REQUIRE(desc->blocks >= 0, "blocks (%d) must be >= 0", desc->blocks);
    return create_prefill(heads, desc->n_branches, desc->n_tokens, desc->prefix_len, desc->max_suffix_len,
                          desc->blocks, PrefillLayout{false, desc->suffix_cap, 0, 0}, out);
}

fka_status fka_plan_create_prefill_paged(const fka_heads *heads, const fka_prefill_paged_desc *desc, fka_plan **out)
{
    REQUIRE(out != nullptr, "out is null");
    *out = nullptr;
    fka_status st = check_heads(heads);
    if (st != FKA_OK) return st;
    REQUIRE(desc != nullptr, "desc is null");
    REQUIRE(desc->n_branches >= 1, "n_branches (%d) must be >= 1", desc->n_branches);
    REQUIRE(desc->n_tokens >= 1, "n_tokens (%d) must be >= 1", desc->n_tokens);
    REQUIRE(desc->prefix_len >= 0, "prefix_len (%d) must be >= 0", desc->prefix_len);
    REQUIRE(desc->page_size == fka::kPageSize, "page_size (%d) must be %d", desc->page_size, fka::kPageSize);
    REQUIRE(desc->n_pool_pages >= 1, "n_pool_pages must be >= 1");
    REQUIRE(desc->max_suffix_len >= desc->n_tokens, "max_suffix_len (%d) must be >= n_tokens (%d)",
            desc->max_suffix_len, desc->n_tokens);
    REQUIRE(desc->blocks >= 0, "blocks (%d) must be >= 0", desc->blocks);
    const int64_t pages = ceil_div(desc->prefix_len, fka::kPageSize) + ceil_div(desc->max_suffix_len, fka::kPageSize);
    REQUIRE(pages <= desc->max_pages_per_seq, "the prefix and max_suffix_len need %lld pages, max_pages_per_seq is %d",
            (long long)pages, desc->max_pages_per_seq);
    return create_prefill(heads, desc->n_branches, desc->n_tokens, desc->prefix_len, desc->max_suffix_len,
                          desc->blocks, PrefillLayout{true, 0, desc->max_pages_per_seq, desc->n_pool_pages}, out);
}

fka_status fka_plan_create_paged(const fka_heads *heads, const fka_paged_desc *desc, const int32_t *host_group_start,
                                 const int32_t *host_group_prefix_len, fka_plan **out)
{
    REQUIRE(out != nullptr, "out is null");
    *out = nullptr;
    fka_status st = check_heads(heads);
    if (st != FKA_OK) return st;
    REQUIRE(desc != nullptr, "desc is null");
    REQUIRE(host_group_start != nullptr && host_group_prefix_len != nullptr, "group arrays are null");
    REQUIRE(desc->n_seqs >= 1 && desc->n_groups >= 1, "n_seqs and n_groups must be >= 1");
    REQUIRE(desc->page_size == fka::kPageSize, "page_size (%d) must be %d", desc->page_size, fka::kPageSize);
    REQUIRE(desc->max_pages_per_seq >= 1, "max_pages_per_seq must be >= 1");
    REQUIRE(desc->n_pool_pages >= 1, "n_pool_pages must be >= 1");
    REQUIRE(desc->max_suffix_len >= 0, "max_suffix_len must be >= 0");
    REQUIRE(desc->share_prefix == 0 || desc->share_prefix == 1, "share_prefix must be 0 or 1");
    if ((st = check_grid(desc->rounds, desc->blocks)) != FKA_OK) return st;
    REQUIRE(host_group_start[0] == 0 && host_group_start[desc->n_groups] == desc->n_seqs,
            "group_start must begin at 0 and end at n_seqs");
    const int G = heads->n_q_heads / heads->n_kv_heads;
    int max_group = 0;
    for (int t = 0; t < desc->n_groups; ++t) {
        const int n = host_group_start[t + 1] - host_group_start[t];
        REQUIRE(n >= 1, "group %d is empty", t);
        const int lp = host_group_prefix_len[t];
        REQUIRE(lp >= 0, "group %d has a negative prefix length", t);
        const int64_t pages = ceil_div(lp, fka::kPageSize) + ceil_div(desc->max_suffix_len, fka::kPageSize);
        REQUIRE(pages <= desc->max_pages_per_seq, "group %d needs %lld pages, max_pages_per_seq is %d", t,
                (long long)pages, desc->max_pages_per_seq);
        max_group = std::max(max_group, n);
    }
    if (desc->n_seqs > fka::kMaxSeqs)
        return fail(FKA_ERR_UNSUPPORTED, "%d sequences exceed the limit of %d", desc->n_seqs, fka::kMaxSeqs);
    const int rows = (desc->share_prefix ? max_group : 1) * G;
    if (G > fka::kMaxRows || rows > fka::kMaxRows)
        return fail(FKA_ERR_UNSUPPORTED, "%d query rows per KV head exceed the limit of %d", rows, fka::kMaxRows);

    fka_plan *p = new (std::nothrow) fka_plan();
    if (!p) return fail(FKA_ERR_NOMEM, "host allocation failed");
    init_heads(p, heads);
    p->paged = true;
    p->n_seqs = desc->n_seqs;
    p->n_groups = desc->n_groups;
    p->share_prefix = desc->share_prefix;
    p->page_size = desc->page_size;
    p->max_pages = desc->max_pages_per_seq;
    p->n_pool_pages = desc->n_pool_pages;
    p->max_suffix_len = desc->max_suffix_len;
    p->group_start.assign(host_group_start, host_group_start + desc->n_groups + 1);
    p->group_prefix_len.assign(host_group_prefix_len, host_group_prefix_len + desc->n_groups);
    std::vector<std::array<int32_t, 3>> units;
    for (int t = 0; t < desc->n_groups; ++t) {
        const int s0 = p->group_start[t], s1 = p->group_start[t + 1], lp = p->group_prefix_len[t];
        if (desc->share_prefix)
            units.push_back({s0, s1 - s0, lp});
        else
            for (int i = s0; i < s1; ++i) units.push_back({i, 1, lp});
    }
    if ((st = build_schedule(p, units, desc->rounds, desc->blocks)) != FKA_OK || (st = finish_plan(p)) != FKA_OK) {
        fka_plan_destroy(p);
        return st;
    }
    *out = p;
    return ok();
}

fka_status fka_plan_get_info(const fka_plan *p, fka_plan_info *info)
{
    REQUIRE(p != nullptr && info != nullptr, "null argument");
    info->n_items = p->n_items;
    info->n_units = (int32_t)p->units.size();
    info->waves_per_block = p->waves;
    info->n_blocks = p->n_blocks;
    info->rounds = p->rounds;
    info->n_slots = p->n_slots;
    info->slot_rows = p->slot_rows;
    info->static_split = p->static_split ? 1 : 0;
    info->units_per_block = p->prefill_groups;
    info->workspace_bytes = p->workspace_bytes;
    return ok();
}

fka_status fka_plan_slots(const fka_plan *p, const int32_t *host_suffix_len, fka_slot *slots, int32_t capacity,
                          int32_t *n_slots)
{
    REQUIRE(p != nullptr && host_suffix_len != nullptr && n_slots != nullptr, "null argument");
    REQUIRE(!p->prefill_n, "plan is an instruction-prefill plan: its slots follow the cyclic placement");
    REQUIRE(capacity >= 0 && (capacity == 0 || slots != nullptr), "slots is null");
    const int N = p->n_seqs, Hkv = p->Hkv, NW = p->waves;
    const int32_t NV = p->n_blocks * p->rounds * NW;
    // per sequence: clamped length; exclusive scan of slice counts (as the kernel's tables)
    std::vector<int32_t> cs(N + 1, 0);
    for (int s = 0; s < N; ++s) {
        const int32_t len = std::min(std::max(host_suffix_len[s], 0), p->max_suffix_len);
        cs[s + 1] = cs[s] + fka::slices_of(len);
    }
    const int n_units = (int)p->units.size();
    std::vector<int32_t> ne(n_units + 1, 0);
    for (int u = 0; u < n_units; ++u) {
        const fka::UnitRec &r = p->units[u];
        ne[u + 1] = ne[u] + ((fka::slices_of(r.plen) + cs[r.seq0 + r.nseq] - cs[r.seq0]) > 0 ? 1 : 0);
    }
    const int64_t T = (int64_t)Hkv * (p->ps_total + cs[N]), NNE = (int64_t)Hkv * ne[n_units];
    const uint64_t R = T > 0 ? fka::sched_ratio(NV - NNE, T) : 0;
    int32_t count = 0;
    for (int i = 0; i < p->n_items; ++i) {
        const int u = i / Hkv, g = i % Hkv;
        const fka::UnitRec &r = p->units[u];
        const int32_t P = fka::slices_of(r.plen), S = cs[r.seq0 + r.nseq] - cs[r.seq0];
        int32_t ws0, ws1;
        if (p->static_split) {
            ws0 = fka::static_start(g, NV, Hkv);
            ws1 = fka::static_start(g + 1, NV, Hkv);
        } else {
            if (P + S == 0 || T == 0) continue;
            const int64_t C = (int64_t)Hkv * (r.ps_before + cs[r.seq0]) + (int64_t)g * (P + S);
            const int64_t K = (int64_t)Hkv * ne[u] + g;
            ws0 = fka::worker_start(C, K, R);
            ws1 = fka::worker_start(C + P + S, K + 1, R);
        }
        if (ws1 <= ws0) continue;
        const int32_t W = ws1 - ws0;
        for (int32_t vb = ws0 / NW; vb <= (ws1 - 1) / NW; ++vb) {
            const int32_t lo = std::max(ws0, vb * NW) - ws0, hi = std::min(ws1, (vb + 1) * NW) - ws0;
            if (count < capacity) {
                fka_slot sl{};
                sl.slot = vb + i;
                sl.seq0 = r.seq0;
                sl.nseq = r.nseq;
                sl.kv_head = g;
                sl.rows = r.nseq * p->G;
                sl.prefix_begin = std::min(fka::pre_split(lo, W, P) * fka::kSlice, r.plen);
                sl.prefix_end = std::min(fka::pre_split(hi, W, P) * fka::kSlice, r.plen);
                sl.suffix_begin = fka::suf_split(lo, W, P, S);
                sl.suffix_end = fka::suf_split(hi, W, P, S);
                sl.prefix_len = r.plen;
                slots[count] = sl;
            }
            ++count;
        }
    }
    *n_slots = count;
    return ok();
}

fka_status fka_fork_decode(const fka_plan *p, const void *q, const void *prefix_k, const void *prefix_v,
                           const void *suffix_k, const void *suffix_v, const int32_t *suffix_len, float *out,
                           float *out_lse, void *stream)
{
    REQUIRE(p != nullptr, "plan is null");
    REQUIRE(!p->prefill_n, "plan is an instruction-prefill plan: use fka_prefill");
    REQUIRE(!p->paged, "plan is paged: use fka_fork_decode_paged");
    REQUIRE_PTR16(q);
    if (p->prefix_len > 0) {
        REQUIRE_PTR16(prefix_k);
        REQUIRE_PTR16(prefix_v);
    }
    REQUIRE_PTR16(suffix_k);
    REQUIRE_PTR16(suffix_v);
    REQUIRE_PTR4(suffix_len);
    REQUIRE_PTR16(out);
    REQUIRE_OPT4(out_lse);
    fka::AttnArgs a = attn_args(p);
    a.q = static_cast<const uint16_t *>(q);
    a.prefix_k = static_cast<const uint16_t *>(prefix_k);
    a.prefix_v = static_cast<const uint16_t *>(prefix_v);
    a.suffix_k = static_cast<const uint16_t *>(suffix_k);
    a.suffix_v = static_cast<const uint16_t *>(suffix_v);
    a.suffix_len = suffix_len;
    return run_decode(p, a, suffix_len, out, out_lse, static_cast<hipStream_t>(stream));
}

fka_status fka_fork_decode_noalloc(const fka_heads *heads, const fka_contig_desc *desc, const void *q,
                                   const void *prefix_k, const void *prefix_v, const void *suffix_k,
                                   const void *suffix_v, const int32_t *suffix_len, float *out, float *out_lse,
                                   int32_t *err, void *stream)
{
    fka_status st = check_contig(heads, desc);
    if (st != FKA_OK) return st;
    REQUIRE(desc->share_prefix == 1, "the no-allocation decode takes a shared prefix (share_prefix = 1)");
    if (desc->prefix_len > kMaxTokens || desc->max_suffix_len > kMaxTokens)
        return fail(FKA_ERR_UNSUPPORTED, "prefix or suffix longer than %d tokens", kMaxTokens);
    REQUIRE_PTR16(q);
    if (desc->prefix_len > 0) {
        REQUIRE_PTR16(prefix_k);
        REQUIRE_PTR16(prefix_v);
    }
    REQUIRE_PTR16(suffix_k);
    REQUIRE_PTR16(suffix_v);
    REQUIRE_PTR4(suffix_len);
    REQUIRE_PTR16(out);
    REQUIRE_OPT4(out_lse);
    REQUIRE_OPT4(err);
    // The plan of fka_plan_create_contig, built on the stack: the scalar fields only (its tables
    // stay empty and unallocated; the one-unit schedule reads none of them).
    fka_plan p;
    init_heads(&p, heads);
    p.n_seqs = desc->n_branches;
    p.share_prefix = 1;
    p.prefix_len = desc->prefix_len;
    p.suffix_cap = desc->suffix_cap;
    p.max_suffix_len = desc->max_suffix_len;
    p.ps_total = fka::slices_of(desc->prefix_len);
    const int64_t est = fka::slices_of(desc->prefix_len) + (int64_t)desc->n_branches * fka::slices_of(desc->max_suffix_len);
    if ((st = set_grid(&p, est, desc->n_branches, 1, desc->rounds, desc->blocks)) != FKA_OK) return st;
    // scratch: lengths, error word, partial lse, partial o; every word a call reads, the same
    // call writes first, so nothing needs clearing
    auto up = [](size_t x) { return (x + 255) & ~size_t(255); };
    const size_t parts = (size_t)p.n_slots * p.slot_rows;
    const size_t b_lens = up((size_t)p.n_seqs * sizeof(int32_t)), b_err = 256;
    const size_t b_pl = up(parts * sizeof(float)), b_po = up(parts * p.d * sizeof(float));
    const size_t need = b_lens + b_err + b_pl + b_po;
    if (need > kScratchBytes)
        return fail(FKA_ERR_UNSUPPORTED, "this decode needs %zu bytes of scratch; the no-allocation decode has %zu (use a plan)",
                    need, kScratchBytes);
    char *base = nullptr;
    if ((st = scratch_of(p.device, &base)) != FKA_OK) return st;
    p.d_lens = reinterpret_cast<int32_t *>(base);
    p.d_rowrec = p.d_lens;  // not read by a one-unit schedule
    p.err = err ? err : reinterpret_cast<int32_t *>(base + b_lens);
    p.part_lse = reinterpret_cast<float *>(base + b_lens + b_err);
    p.part_o = reinterpret_cast<float *>(base + b_lens + b_err + b_pl);
    fka::AttnArgs a = attn_args(&p);
    a.q = static_cast<const uint16_t *>(q);
    a.prefix_k = static_cast<const uint16_t *>(prefix_k);
    a.prefix_v = static_cast<const uint16_t *>(prefix_v);
    a.suffix_k = static_cast<const uint16_t *>(suffix_k);
    a.suffix_v = static_cast<const uint16_t *>(suffix_v);
    a.suffix_len = suffix_len;
    return run_decode(&p, a, suffix_len, out, out_lse, static_cast<hipStream_t>(stream));
}

fka_status fka_prefill(const fka_plan *p, const void *q, const void *prefix_k, const void *prefix_v,
                       const void *suffix_k, const void *suffix_v, const int32_t *suffix_len, float *out,
                       float *out_lse, void *stream)
{
    REQUIRE(p != nullptr, "plan is null");
    REQUIRE(p->prefill_n > 0, "plan is not an instruction-prefill plan (fka_plan_create_prefill)");
    REQUIRE(!p->paged, "plan is a paged prefill plan: use fka_prefill_paged");
    REQUIRE_PTR16(q);
    if (p->prefix_len > 0) {
        REQUIRE_PTR16(prefix_k);
        REQUIRE_PTR16(prefix_v);
    }
    REQUIRE_PTR16(suffix_k);
    REQUIRE_PTR16(suffix_v);
    REQUIRE_PTR4(suffix_len);
    REQUIRE_PTR16(out);
    REQUIRE_OPT4(out_lse);
    fka::AttnArgs a = attn_args(p);
    a.q = static_cast<const uint16_t *>(q);
    a.prefix_k = static_cast<const uint16_t *>(prefix_k);
    a.prefix_v = static_cast<const uint16_t *>(prefix_v);
    a.suffix_k = static_cast<const uint16_t *>(suffix_k);
    a.suffix_v = static_cast<const uint16_t *>(suffix_v);
    a.suffix_len = suffix_len;
    a.prefill_n = p->prefill_n;
    return run_prefill(p, a, out, out_lse, static_cast<hipStream_t>(stream));
}

fka_status fka_prefill_paged(const fka_plan *p, const void *q, const void *k_pool, const void *v_pool,
                             const int32_t *page_table, const int32_t *suffix_len, float *out, float *out_lse,
                             void *stream)
{
    REQUIRE(p != nullptr, "plan is null");
    REQUIRE(p->prefill_n > 0 && p->paged, "plan is not a paged instruction-prefill plan (fka_plan_create_prefill_paged)");
    REQUIRE_PTR16(q);
    REQUIRE_PTR16(k_pool);
    REQUIRE_PTR16(v_pool);
    REQUIRE_PTR4(page_table);
    REQUIRE_PTR4(suffix_len);
    REQUIRE_PTR16(out);
    REQUIRE_OPT4(out_lse);
    fka::AttnArgs a = attn_args(p);
    a.q = static_cast<const uint16_t *>(q);
    a.k_pool = static_cast<const uint16_t *>(k_pool);
    a.v_pool = static_cast<const uint16_t *>(v_pool);
    a.page_table = page_table;
    a.suffix_len = suffix_len;
    a.prefill_n = p->prefill_n;
    return run_prefill(p, a, out, out_lse, static_cast<hipStream_t>(stream));
}

fka_status fka_partials(const fka_plan *p, const void *q, const void *prefix_k, const void *prefix_v,
                        const void *suffix_k, const void *suffix_v, const int32_t *suffix_len, float *part_o,
                        float *part_lse, void *stream)
{
    REQUIRE(p != nullptr, "plan is null");
    REQUIRE(!p->prefill_n, "plan is an instruction-prefill plan: use fka_prefill");
    REQUIRE(!p->paged, "plan is paged: use fka_partials_paged");
    REQUIRE_PTR16(q);
    if (p->prefix_len > 0) {
        REQUIRE_PTR16(prefix_k);
        REQUIRE_PTR16(prefix_v);
    }
    REQUIRE_PTR16(suffix_k);
    REQUIRE_PTR16(suffix_v);
    REQUIRE_PTR4(suffix_len);
    REQUIRE_PTR16(part_o);
    REQUIRE_PTR4(part_lse);
    fka::AttnArgs a = attn_args(p);
    a.q = static_cast<const uint16_t *>(q);
    a.prefix_k = static_cast<const uint16_t *>(prefix_k);
    a.prefix_v = static_cast<const uint16_t *>(prefix_v);
    a.suffix_k = static_cast<const uint16_t *>(suffix_k);
    a.suffix_v = static_cast<const uint16_t *>(suffix_v);
    a.suffix_len = suffix_len;
    a.part_o = part_o;
    a.part_lse = part_lse;
    hipError_t e = fka::launch_partials(a, p->n_blocks * p->rounds, p->d, p->row_tiles, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "partials kernel launch");
    return ok();
}

fka_status fka_partials_paged(const fka_plan *p, const void *q, const void *k_pool, const void *v_pool,
                              const int32_t *page_table, const int32_t *suffix_len, float *part_o, float *part_lse,
                              void *stream)
{
    REQUIRE(p != nullptr, "plan is null");
    REQUIRE(p->paged, "plan is contiguous: use fka_partials");
    REQUIRE(!p->prefill_n, "plan is an instruction-prefill plan: use fka_prefill_paged");
    REQUIRE_PTR16(q);
    REQUIRE_PTR16(k_pool);
    REQUIRE_PTR16(v_pool);
    REQUIRE_PTR4(page_table);
    REQUIRE_PTR4(suffix_len);
    REQUIRE_PTR16(part_o);
    REQUIRE_PTR4(part_lse);
    fka::AttnArgs a = attn_args(p);
    a.q = static_cast<const uint16_t *>(q);
    a.k_pool = static_cast<const uint16_t *>(k_pool);
    a.v_pool = static_cast<const uint16_t *>(v_pool);
    a.page_table = page_table;
    a.suffix_len = suffix_len;
    a.part_o = part_o;
    a.part_lse = part_lse;
    hipError_t e = fka::launch_partials(a, p->n_blocks * p->rounds, p->d, p->row_tiles, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "partials kernel launch");
    return ok();
}

fka_status fka_append_kv(const fka_plan *p, const void *k_new, const void *v_new, void *suffix_k, void *suffix_v,
                         int32_t *suffix_len, void *stream)
{
    REQUIRE(p != nullptr, "plan is null");
    REQUIRE(!p->prefill_n, "plan is an instruction-prefill plan: use fka_prefill");
    REQUIRE(!p->paged, "plan is paged: use fka_append_kv_paged");
    REQUIRE_PTR16(k_new);
    REQUIRE_PTR16(v_new);
    REQUIRE_PTR16(suffix_k);
    REQUIRE_PTR16(suffix_v);
    REQUIRE_PTR4(suffix_len);
    fka::AppendArgs a{};
    a.k_new = static_cast<const uint16_t *>(k_new);
    a.v_new = static_cast<const uint16_t *>(v_new);
    a.k_dst = static_cast<uint16_t *>(suffix_k);
    a.v_dst = static_cast<uint16_t *>(suffix_v);
    a.suffix_len = suffix_len;
    a.suffix_cap = p->suffix_cap;
    a.max_suffix_len = p->max_suffix_len;
    a.n_kv_heads = p->Hkv;
    a.head_dim = p->d;
    a.paged = 0;
    a.err = p->err;
    hipError_t e = fka::launch_append(a, p->n_seqs, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "append kernel launch");
    return ok();
}

fka_status fka_fork_step(const fka_plan *p, const void *q, const void *k_new, const void *v_new,
                         const void *prefix_k, const void *prefix_v, void *suffix_k, void *suffix_v,
                         int32_t *suffix_len, float *out, float *out_lse, void *stream)
{
    REQUIRE(p != nullptr, "plan is null");
    REQUIRE(!p->prefill_n, "plan is an instruction-prefill plan: use fka_prefill");
    REQUIRE(!p->paged, "plan is paged: use fka_fork_step_paged");
    REQUIRE_PTR16(q);
    REQUIRE_PTR16(k_new);
    REQUIRE_PTR16(v_new);
    if (p->prefix_len > 0) {
        REQUIRE_PTR16(prefix_k);
        REQUIRE_PTR16(prefix_v);
    }
    REQUIRE_PTR16(suffix_k);
    REQUIRE_PTR16(suffix_v);
    REQUIRE_PTR4(suffix_len);
    REQUIRE_PTR16(out);
    REQUIRE_OPT4(out_lse);
    fka::AttnArgs a = attn_args(p);
    a.q = static_cast<const uint16_t *>(q);
    a.prefix_k = static_cast<const uint16_t *>(prefix_k);
    a.prefix_v = static_cast<const uint16_t *>(prefix_v);
    a.suffix_k = static_cast<const uint16_t *>(suffix_k);
    a.suffix_v = static_cast<const uint16_t *>(suffix_v);
    a.suffix_len = suffix_len;
    fka::MergeArgs m = merge_args(p, suffix_len, out, out_lse);
    m.step_mode = 1;
    m.q = a.q;
    m.k_new = static_cast<const uint16_t *>(k_new);
    m.v_new = static_cast<const uint16_t *>(v_new);
    m.k_dst = static_cast<uint16_t *>(suffix_k);
    m.v_dst = static_cast<uint16_t *>(suffix_v);
    return run_decode(p, a, suffix_len, out, out_lse, static_cast<hipStream_t>(stream), &m);
}

fka_status fka_fork_step_paged(const fka_plan *p, const void *q, const void *k_new, const void *v_new, void *k_pool,
                               void *v_pool, const int32_t *page_table, int32_t *suffix_len, float *out,
                               float *out_lse, void *stream)
{
    REQUIRE(p != nullptr, "plan is null");
    REQUIRE(p->paged, "plan is contiguous: use fka_fork_step");
    REQUIRE(!p->prefill_n, "plan is an instruction-prefill plan: use fka_prefill_paged");
    REQUIRE_PTR16(q);
    REQUIRE_PTR16(k_new);
    REQUIRE_PTR16(v_new);
    REQUIRE_PTR16(k_pool);
    REQUIRE_PTR16(v_pool);
    REQUIRE_PTR4(page_table);
    REQUIRE_PTR4(suffix_len);
    REQUIRE_PTR16(out);
    REQUIRE_OPT4(out_lse);
    fka::AttnArgs a = attn_args(p);
    a.q = static_cast<const uint16_t *>(q);
    a.k_pool = static_cast<const uint16_t *>(k_pool);
    a.v_pool = static_cast<const uint16_t *>(v_pool);
    a.page_table = page_table;
    a.suffix_len = suffix_len;
    fka::MergeArgs m = merge_args(p, suffix_len, out, out_lse);
    m.step_mode = 1;
    m.q = a.q;
    m.k_new = static_cast<const uint16_t *>(k_new);
    m.v_new = static_cast<const uint16_t *>(v_new);
    m.k_dst = static_cast<uint16_t *>(k_pool);
    m.v_dst = static_cast<uint16_t *>(v_pool);
    m.page_table = page_table;
    return run_decode(p, a, suffix_len, out, out_lse, static_cast<hipStream_t>(stream), &m);
}

fka_status fka_fork_decode_paged(const fka_plan *p, const void *q, const void *k_pool, const void *v_pool,
                                 const int32_t *page_table, const int32_t *suffix_len, float *out, float *out_lse,
                                 void *stream)
{
    REQUIRE(p != nullptr, "plan is null");
    REQUIRE(p->paged, "plan is contiguous: use fka_fork_decode");
    REQUIRE(!p->prefill_n, "plan is an instruction-prefill plan: use fka_prefill_paged");
    REQUIRE_PTR16(q);
    REQUIRE_PTR16(k_pool);
    REQUIRE_PTR16(v_pool);
    REQUIRE_PTR4(page_table);
    REQUIRE_PTR4(suffix_len);
    REQUIRE_PTR16(out);
    REQUIRE_OPT4(out_lse);
    fka::AttnArgs a = attn_args(p);
    a.q = static_cast<const uint16_t *>(q);
    a.k_pool = static_cast<const uint16_t *>(k_pool);
    a.v_pool = static_cast<const uint16_t *>(v_pool);
    a.page_table = page_table;
    a.suffix_len = suffix_len;
    return run_decode(p, a, suffix_len, out, out_lse, static_cast<hipStream_t>(stream));
}

fka_status fka_append_kv_paged(const fka_plan *p, const void *k_new, const void *v_new, void *k_pool, void *v_pool,
                               const int32_t *page_table, int32_t *suffix_len, void *stream)
{
    REQUIRE(p != nullptr, "plan is null");
    REQUIRE(p->paged, "plan is contiguous: use fka_append_kv");
    REQUIRE(!p->prefill_n, "plan is an instruction-prefill plan: use fka_prefill_paged");
    REQUIRE_PTR16(k_new);
    REQUIRE_PTR16(v_new);
    REQUIRE_PTR16(k_pool);
    REQUIRE_PTR16(v_pool);
    REQUIRE_PTR4(page_table);
    REQUIRE_PTR4(suffix_len);
    fka::AppendArgs a{};
    a.k_new = static_cast<const uint16_t *>(k_new);
    a.v_new = static_cast<const uint16_t *>(v_new);
    a.k_dst = static_cast<uint16_t *>(k_pool);
    a.v_dst = static_cast<uint16_t *>(v_pool);
    a.page_table = page_table;
    a.seq_prefix_len = p->d_seq_prefix_len;
    a.suffix_len = suffix_len;
    a.max_pages = p->max_pages;
    a.n_pool_pages = p->n_pool_pages;
    a.max_suffix_len = p->max_suffix_len;
    a.n_kv_heads = p->Hkv;
    a.head_dim = p->d;
    a.paged = 1;
    a.err = p->err;
    hipError_t e = fka::launch_append(a, p->n_seqs, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "append kernel launch");
    return ok();
}

fka_status fka_gather_paged(const fka_plan *p, int32_t seq, const void *k_pool, const void *v_pool,
                            const int32_t *page_table, int32_t out_len, void *k_out, void *v_out, void *stream)
{
    return fka_gather_paged_range(p, seq, 0, out_len, k_pool, v_pool, page_table, k_out, v_out, stream);
}

fka_status fka_gather_paged_range(const fka_plan *p, int32_t seq, int32_t begin, int32_t out_len, const void *k_pool,
                                  const void *v_pool, const int32_t *page_table, void *k_out, void *v_out,
                                  void *stream)
{
    REQUIRE(p != nullptr, "plan is null");
    REQUIRE(p->paged, "plan is contiguous");
    REQUIRE(!p->prefill_n, "plan is an instruction-prefill plan: use fka_prefill_paged");
    REQUIRE(seq >= 0 && seq < p->n_seqs, "seq %d out of range [0, %d)", seq, p->n_seqs);
    REQUIRE_PTR16(k_pool);
    REQUIRE_PTR16(v_pool);
    REQUIRE_PTR4(page_table);
    REQUIRE_PTR16(k_out);
    REQUIRE_PTR16(v_out);
    int t = 0;
    while (t + 1 < p->n_groups && p->group_start[t + 1] <= seq) ++t;
    const int lp = p->group_prefix_len[t];
    REQUIRE(out_len >= 0 && begin >= 0 && begin <= out_len, "need 0 <= begin <= out_len (begin %d, out_len %d)",
            begin, out_len);
    const int64_t pages = ceil_div(lp, fka::kPageSize) + (out_len > lp ? ceil_div(out_len - lp, fka::kPageSize) : 0);
    REQUIRE(pages <= p->max_pages, "out_len %d needs %lld pages, the table has %d", out_len, (long long)pages,
            p->max_pages);
    fka::GatherArgs a{};
    a.k_pool = static_cast<const uint16_t *>(k_pool);
    a.v_pool = static_cast<const uint16_t *>(v_pool);
    a.page_table = page_table;
    a.k_out = static_cast<uint16_t *>(k_out);
    a.v_out = static_cast<uint16_t *>(v_out);
    a.seq = seq;
    a.prefix_len = lp;
    a.begin = begin;
    a.out_len = out_len;
    a.max_pages = p->max_pages;
    a.n_pool_pages = p->n_pool_pages;
    a.n_kv_heads = p->Hkv;
    a.head_dim = p->d;
    a.err = p->err;
    hipError_t e = fka::launch_gather(a, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "gather kernel launch");
    return ok();
}

fka_status fka_lse_merge(int32_t rows, int32_t n_parts, int32_t head_dim, const float *part_o, const float *part_lse,
                         float *out, float *out_lse, void *stream)
{
    REQUIRE(rows >= 0 && n_parts >= 0, "rows and n_parts must be >= 0");
    if (head_dim != 64 && head_dim != 128)
        return fail(FKA_ERR_UNSUPPORTED, "head_dim %d not supported (64 or 128)", head_dim);
    if (rows == 0) return ok();
    if (n_parts > 0) {
        REQUIRE_PTR16(part_o);
        REQUIRE_PTR4(part_lse);
        // the merge addresses the parts with 32-bit byte offsets
        if ((int64_t)n_parts * rows * head_dim * 4 >= ((int64_t)1 << 31))
            return fail(FKA_ERR_UNSUPPORTED, "%d parts of %d rows exceed the 2 GiB the merge addresses", n_parts, rows);
    }
    REQUIRE_PTR16(out);
    REQUIRE_OPT4(out_lse);
    fka::MergeArgs m{};
    m.part_o = part_o;
    m.part_lse = part_lse;
    m.out = out;
    m.out_lse = out_lse;
    m.rows = rows;
    m.n_q_heads = 1;
    m.n_parts = n_parts;
    hipError_t e = fka::launch_merge(m, head_dim, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "merge kernel launch");
    return ok();
}

fka_status fka_read_probe(const void *buf, size_t bytes, int32_t blocks, int32_t threads, int32_t unroll,
                          uint32_t *sink, void *stream)
{
    REQUIRE_PTR16(buf);
    REQUIRE_PTR4(sink);
    REQUIRE(bytes > 0 && bytes % 16 == 0, "bytes (%zu) must be a positive multiple of 16", bytes);
    REQUIRE(blocks >= 1, "blocks (%d) must be >= 1", blocks);
    REQUIRE(threads >= 64 && threads <= 1024 && threads % 64 == 0, "threads (%d) must be a multiple of 64 in [64, 1024]",
            threads);
    REQUIRE(unroll == 4 || unroll == 8 || unroll == 16, "unroll (%d) must be 4, 8 or 16", unroll);
    hipError_t e = fka::launch_read_probe(buf, bytes, blocks, threads, unroll, sink, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "read probe launch");
    return ok();
}

fka_status fka_plan_device_error(const fka_plan *p, int32_t *flags)
{
    REQUIRE(p != nullptr && flags != nullptr, "null argument");
    int32_t v = 0;
    hipError_t e = hipMemcpy(&v, p->err, sizeof v, hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail(e, "hipMemcpy(error flag)");
    if ((e = hipMemset(p->err, 0, sizeof v)) != hipSuccess) return hip_fail(e, "hipMemset(error flag)");
    *flags = v;
    return ok();
}

void fka_plan_destroy(fka_plan *p)
{
    if (!p) return;
    if (p->mem) (void)hipFree(p->mem);
    delete p;
}

/* ------------------------------------------------------------------ page pool */

fka_status fka_pool_create(int32_t n_pages, fka_pool **out)
{
    REQUIRE(out != nullptr, "out is null");
    *out = nullptr;
    REQUIRE(n_pages >= 0, "n_pages must be >= 0");
    fka_pool *pool = new (std::nothrow) fka_pool;
    if (!pool) return fail(FKA_ERR_NOMEM, "pool: host allocation failed");
    try {
        pool->ref.assign(n_pages, 0);
        pool->pending.assign(n_pages, 0);
        for (int32_t i = 0; i < n_pages; ++i) pool->free_ids.insert(pool->free_ids.end(), i);
    } catch (...) {
        delete pool;
        return fail(FKA_ERR_NOMEM, "pool: host allocation failed");
    }
    *out = pool;
    return ok();
}

void fka_pool_destroy(fka_pool *pool) { delete pool; }

int32_t fka_pool_free_pages(const fka_pool *pool) { return pool ? (int32_t)pool->free_ids.size() : -1; }

int32_t fka_pool_refcount(const fka_pool *pool, int32_t page)
{
    if (!pool || page < 0 || page >= (int32_t)pool->ref.size()) return -1;
    return pool->ref[page];
}

}  // extern "C"

namespace {

void clear_drops(fka_pool *pool)
{
    for (int32_t id : pool->touched) pool->pending[id] = 0;
    pool->touched.clear();
}

// Counts the references to drop per page (ids[n], entries equal to -1 skipped) and checks them
// against the counts; nothing changes until apply_drops.
fka_status count_drops(fka_pool *pool, const int32_t *ids, int64_t n)
{
    clear_drops(pool);
    for (int64_t i = 0; i < n; ++i) {
        const int32_t id = ids[i];
        if (id == -1) continue;
        if (id < 0 || id >= (int32_t)pool->ref.size()) {
            clear_drops(pool);
            return fail(FKA_ERR_INVALID_ARG, "page id %d outside the pool", id);
        }
        if (pool->pending[id]++ == 0) pool->touched.push_back(id);
        if (pool->pending[id] > pool->ref[id]) {
            const int32_t r = pool->ref[id];
            clear_drops(pool);
            return fail(FKA_ERR_INVALID_ARG, "page %d has %d reference(s), more to drop", id, r);
        }
    }
    return FKA_OK;
}

void apply_drops(fka_pool *pool)
{
    for (int32_t id : pool->touched) {
        if ((pool->ref[id] -= pool->pending[id]) == 0) pool->free_ids.insert(id);
        pool->pending[id] = 0;
    }
    pool->touched.clear();
}

void take_pages(fka_pool *pool, int32_t n, int32_t *ids)  // n <= free pages
{
    for (int32_t i = 0; i < n; ++i) {
        const int32_t id = *pool->free_ids.begin();
        pool->free_ids.erase(pool->free_ids.begin());
        pool->ref[id] = 1;
        ids[i] = id;
    }
}

bool live(const fka_pool *pool, int32_t id) { return id >= 0 && id < (int32_t)pool->ref.size() && pool->ref[id] > 0; }

int32_t pages_for(int64_t tokens) { return (int32_t)((tokens + fka::kPageSize - 1) / fka::kPageSize); }

}  // namespace

extern "C" {

fka_status fka_pool_alloc(fka_pool *pool, int32_t n, int32_t *ids)
{
    REQUIRE(pool != nullptr, "pool is null");
    REQUIRE(n >= 0, "n must be >= 0");
    REQUIRE(n == 0 || ids != nullptr, "ids is null");
    if (n > (int32_t)pool->free_ids.size())
        return fail(FKA_ERR_NOMEM, "%d pages asked, %d free", n, (int32_t)pool->free_ids.size());
    take_pages(pool, n, ids);
    return ok();
}

fka_status fka_pool_retain(fka_pool *pool, int32_t n, const int32_t *ids)
{
    REQUIRE(pool != nullptr, "pool is null");
    REQUIRE(n >= 0, "n must be >= 0");
    REQUIRE(n == 0 || ids != nullptr, "ids is null");
    for (int32_t i = 0; i < n; ++i) REQUIRE(live(pool, ids[i]), "page id %d is not live", ids[i]);
    for (int32_t i = 0; i < n; ++i) ++pool->ref[ids[i]];
    return ok();
}

fka_status fka_pool_release(fka_pool *pool, int32_t n, const int32_t *ids)
{
    REQUIRE(pool != nullptr, "pool is null");
    REQUIRE(n >= 0, "n must be >= 0");
    REQUIRE(n == 0 || ids != nullptr, "ids is null");
    for (int32_t i = 0; i < n; ++i) REQUIRE(ids[i] != -1, "page id -1");
    fka_status st = count_drops(pool, ids, n);
    if (st != FKA_OK) return st;
    apply_drops(pool);
    return ok();
}

fka_status fka_pool_fork(fka_pool *pool, const int32_t *prefix_pages, int32_t n_prefix_pages, int32_t *page_table,
                         int32_t max_pages, int32_t first, int32_t n)
{
    REQUIRE(pool != nullptr && page_table != nullptr, "null argument");
    REQUIRE(max_pages > 0 && n_prefix_pages >= 0 && n_prefix_pages <= max_pages,
            "n_prefix_pages %d outside [0, max_pages %d]", n_prefix_pages, max_pages);
    REQUIRE(n_prefix_pages == 0 || prefix_pages != nullptr, "prefix_pages is null");
    REQUIRE(first >= 0 && n >= 0, "first and n must be >= 0");
    for (int32_t i = 0; i < n_prefix_pages; ++i)
        REQUIRE(live(pool, prefix_pages[i]), "snapshot page id %d is not live", prefix_pages[i]);
    for (int64_t r = first; r < (int64_t)first + n; ++r)
        for (int32_t i = 0; i < max_pages; ++i)
            REQUIRE(page_table[r * max_pages + i] == -1, "row %lld holds pages", (long long)r);
    for (int64_t r = first; r < (int64_t)first + n; ++r)
        for (int32_t i = 0; i < n_prefix_pages; ++i) {
            page_table[r * max_pages + i] = prefix_pages[i];
            ++pool->ref[prefix_pages[i]];
        }
    return ok();
}

fka_status fka_pool_reserve(fka_pool *pool, int32_t *page_table, int32_t max_pages, int32_t seq,
                            int32_t prefix_len, int32_t suffix_len, int32_t *n_new)
{
    REQUIRE(pool != nullptr && page_table != nullptr, "null argument");
    REQUIRE(max_pages > 0 && seq >= 0 && prefix_len >= 0 && suffix_len >= 0, "negative size or index");
    const int32_t a = pages_for(prefix_len), ns = pages_for(suffix_len);
    REQUIRE((int64_t)a + ns <= max_pages, "%d prefix and %d suffix pages exceed max_pages %d", a, ns, max_pages);
    int32_t *row = page_table + (int64_t)seq * max_pages;
    int32_t missing = 0;
    for (int32_t i = 0; i < a + ns; ++i) {
        if (row[i] == -1 && i >= a) {
            ++missing;
            continue;
        }
        REQUIRE(live(pool, row[i]), "row %d index %d: page id %d is not live", seq, i, row[i]);
    }
    if (missing > (int32_t)pool->free_ids.size())
        return fail(FKA_ERR_NOMEM, "%d pages needed, %d free", missing, (int32_t)pool->free_ids.size());
    for (int32_t i = a; i < a + ns; ++i)
        if (row[i] == -1) take_pages(pool, 1, &row[i]);
    if (n_new) *n_new = missing;
    return ok();
}

fka_status fka_pool_drop(fka_pool *pool, int32_t *page_table, int32_t max_pages, int32_t seq)
{
    REQUIRE(pool != nullptr && page_table != nullptr, "null argument");
    REQUIRE(max_pages > 0 && seq >= 0, "bad max_pages or seq");
    int32_t *row = page_table + (int64_t)seq * max_pages;
    fka_status st = count_drops(pool, row, max_pages);
    if (st != FKA_OK) return st;
    apply_drops(pool);
    for (int32_t i = 0; i < max_pages; ++i) row[i] = -1;
    return ok();
}

fka_status fka_pool_promote(fka_pool *pool, int32_t *page_table, int32_t max_pages, int32_t seq, int32_t prefix_len,
                            int32_t suffix_len, int32_t *dense, int32_t *from)
{
    REQUIRE(pool != nullptr && page_table != nullptr && dense != nullptr && from != nullptr, "null argument");
    REQUIRE(max_pages > 0 && seq >= 0 && prefix_len >= 0 && suffix_len >= 0, "negative size or index");
    const int32_t k0 = prefix_len / fka::kPageSize, a = pages_for(prefix_len), ns = pages_for(suffix_len);
    REQUIRE((int64_t)a + ns <= max_pages, "%d prefix and %d suffix pages exceed max_pages %d", a, ns, max_pages);
    const int32_t n_dense = pages_for((int64_t)prefix_len + suffix_len);
    int32_t *row = page_table + (int64_t)seq * max_pages;
    for (int32_t i = 0; i < a + ns; ++i)
        REQUIRE(live(pool, row[i]), "row %d index %d: page id %d is not live", seq, i, row[i]);
    fka_status st = count_drops(pool, row, max_pages);  // the row's references, checked
    if (st != FKA_OK) return st;
    // pages the row may refill: the partial prefix page, then the suffix pages (and any reserved
    // beyond them), each only where the row holds the page's one reference
    std::vector<int32_t> reuse, drop;
    for (int32_t i = k0; i < max_pages; ++i) {
        if (row[i] == -1) continue;
        if (pool->ref[row[i]] == 1 && pool->pending[row[i]] == 1)
            reuse.push_back(row[i]);
        else
            drop.push_back(row[i]);
    }
    clear_drops(pool);
    const int32_t need = n_dense - k0;
    const int32_t take = std::max(0, need - (int32_t)reuse.size());
    if (take > (int32_t)pool->free_ids.size())
        return fail(FKA_ERR_NOMEM, "%d pages needed, %d free", take, (int32_t)pool->free_ids.size());
    for (int32_t i = 0; i < k0; ++i) dense[i] = row[i];
    for (int32_t j = 0; j < (int32_t)reuse.size(); ++j) {
        if (j < need)
            dense[k0 + j] = reuse[j];
        else
            drop.push_back(reuse[j]);
    }
    if (count_drops(pool, drop.data(), (int64_t)drop.size()) == FKA_OK) apply_drops(pool);  // held: cannot fail
    if (take > 0) take_pages(pool, take, dense + k0 + (int32_t)reuse.size());
    for (int32_t i = 0; i < max_pages; ++i) row[i] = -1;
    *from = k0 * fka::kPageSize;
    return ok();
}

fka_status fka_scatter_pages(const void *k_src, const void *v_src, int32_t len, int32_t from, const int32_t *page_row,
                             int32_t n_kv_heads, int32_t head_dim, int32_t n_pool_pages, void *k_pool, void *v_pool,
                             int32_t *err, void *stream)
{
    REQUIRE(len >= 0 && from >= 0 && from <= len, "need 0 <= from <= len (from %d, len %d)", from, len);
    REQUIRE(head_dim == 64 || head_dim == 128, "head_dim %d: 64 or 128", head_dim);
    REQUIRE(n_kv_heads >= 1 && n_kv_heads <= 65535, "n_kv_heads %d outside [1, 65535]", n_kv_heads);
    REQUIRE(n_pool_pages >= 0, "n_pool_pages must be >= 0");
    if (len == from) return ok();
    REQUIRE_PTR16(k_src);
    REQUIRE_PTR16(v_src);
    REQUIRE_PTR16(k_pool);
    REQUIRE_PTR16(v_pool);
    REQUIRE_PTR4(page_row);
    REQUIRE_OPT4(err);
    fka::ScatterArgs s{};
    s.k_src = static_cast<const uint16_t *>(k_src);
    s.v_src = static_cast<const uint16_t *>(v_src);
    s.page_row = page_row;
    s.k_pool = static_cast<uint16_t *>(k_pool);
    s.v_pool = static_cast<uint16_t *>(v_pool);
    s.len = len;
    s.from = from;
    s.n_pool_pages = n_pool_pages;
    s.n_kv_heads = n_kv_heads;
    s.head_dim = head_dim;
    s.err = err;
    hipError_t e = fka::launch_scatter(s, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "scatter kernel launch");
    return ok();
}

}  // extern "C"
