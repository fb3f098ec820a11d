// C ABI of libforkattn.so: argument validation, plans (work lists and
// workspaces) and kernel launches.  Declared in include/forkattn.h.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>
#include <vector>

#include "forkattn.h"
#include "internal.h"

using fka::WorkItem;

struct fka_plan {
    bool paged = false;
    int32_t Hq = 0, Hkv = 0, d = 0, G = 0;
    float scale = 0.f;
    int32_t n_seqs = 0;
    int32_t share_prefix = 1;
    int32_t max_suffix_len = 0;
    // contiguous
    int32_t prefix_len = 0, suffix_cap = 0;
    // paged
    int32_t n_groups = 0, page_size = 0, max_pages = 0, n_pool_pages = 0;
    std::vector<int32_t> group_start, group_prefix_len;
    // split geometry
    int32_t split = 0, ssplit = 0, max_prefix_parts = 0, n_suffix_parts = 0, slots = 0;
    int32_t row_tiles = 1;
    int32_t n_items = 0;
    size_t workspace_bytes = 0;
    int device = 0;
    // device memory (one allocation, carved)
    void *mem = nullptr;
    WorkItem *items = nullptr;
    int32_t *seq_prefix_parts = nullptr;
    int32_t *seq_prefix_len = nullptr;
    int32_t *err = nullptr;
    int32_t *counter = nullptr;  // fused-step completion counter, zero between launches
    int32_t *queue = nullptr;    // work-queue head of the partial kernel, zero between launches
    int32_t *done = nullptr;     // finished blocks of the partial kernel, zero between launches
    void *zero_page = nullptr;   // 4 KiB of zeros
    int32_t n_blocks = 0;        // persistent blocks of the partial kernel
    float *part_o = nullptr;
    float *part_lse = nullptr;
};

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

#define REQUIRE(cond, ...)                                  \
    do {                                                    \
        if (!(cond)) return fail(FKA_ERR_INVALID_ARG, __VA_ARGS__); \
    } while (0)

#define REQUIRE_PTR16(p)                                                          \
    do {                                                                          \
        if (!(p)) return fail(FKA_ERR_INVALID_ARG, "%s is null", #p);             \
        if (!aligned16(p)) return fail(FKA_ERR_INVALID_ARG, "%s is not 16-byte aligned", #p); \
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

// Prefix tokens per work item: about one item per compute unit (256 on MI355X),
// in whole 128-token tiles, between 128 and 8192 tokens; the suffix items fill in
// behind them from the device queue.
int32_t auto_split(int64_t prefix_token_heads)
{
    const int64_t target_items = 256;
    int64_t s = (prefix_token_heads + target_items - 1) / target_items;
    s = ((s + fka::kTileTokens - 1) / fka::kTileTokens) * fka::kTileTokens;
    return (int32_t)std::min<int64_t>(8192, std::max<int64_t>(fka::kTileTokens, s));
}

int32_t auto_suffix_split(int32_t max_suffix_len)
{
    // whole tiles; short suffixes stay in one item
    if (max_suffix_len <= 512) return std::max(fka::kTileTokens, ceil_div(std::max(max_suffix_len, 1), 128) * 128);
    return 512;
}

// Allocate device memory for the work list, per-sequence tables, error flag and
// workspace, and upload the tables.
fka_status finish_plan(fka_plan *p, const std::vector<WorkItem> &items, const std::vector<int32_t> &spp,
                       const std::vector<int32_t> &spl)
{
    hipError_t e = hipGetDevice(&p->device);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    auto up = [](size_t x) { return (x + 255) & ~size_t(255); };
    const size_t n_rows = (size_t)p->n_seqs * p->Hq;
    const size_t b_items = up(std::max<size_t>(1, items.size()) * sizeof(WorkItem));
    const size_t b_spp = up(std::max<size_t>(1, spp.size()) * sizeof(int32_t));
    const size_t b_spl = up(std::max<size_t>(1, spl.size()) * sizeof(int32_t));
    const size_t b_err = 256;
    const size_t b_zero = 4096;
    const size_t b_po = up(std::max<size_t>(1, (size_t)p->slots * n_rows * p->d) * sizeof(float));
    const size_t b_pl = up(std::max<size_t>(1, (size_t)p->slots * n_rows) * sizeof(float));
    const size_t total = b_items + b_spp + b_spl + b_err + b_zero + b_po + b_pl;
    e = hipMalloc(&p->mem, total);
    if (e != hipSuccess) {
        p->mem = nullptr;
        (void)hipGetLastError();
        return fail(FKA_ERR_NOMEM, "hipMalloc(%zu) failed: %s", total, hipGetErrorString(e));
    }
    char *m = static_cast<char *>(p->mem);
    p->items = reinterpret_cast<WorkItem *>(m);
    m += b_items;
    p->seq_prefix_parts = reinterpret_cast<int32_t *>(m);
    m += b_spp;
    p->seq_prefix_len = reinterpret_cast<int32_t *>(m);
    m += b_spl;
    p->err = reinterpret_cast<int32_t *>(m);
    m += b_err;
    p->zero_page = m;
    m += b_zero;
    p->part_o = reinterpret_cast<float *>(m);
    m += b_po;
    p->part_lse = reinterpret_cast<float *>(m);
    p->workspace_bytes = total;
    p->n_items = (int32_t)items.size();
    if (!items.empty() && (e = hipMemcpy(p->items, items.data(), items.size() * sizeof(WorkItem),
                                         hipMemcpyHostToDevice)) != hipSuccess)
        return hip_fail(e, "hipMemcpy(work list)");
    if ((e = hipMemcpy(p->seq_prefix_parts, spp.data(), spp.size() * sizeof(int32_t), hipMemcpyHostToDevice)) !=
        hipSuccess)
        return hip_fail(e, "hipMemcpy(prefix parts)");
    if ((e = hipMemcpy(p->seq_prefix_len, spl.data(), spl.size() * sizeof(int32_t), hipMemcpyHostToDevice)) !=
        hipSuccess)
        return hip_fail(e, "hipMemcpy(prefix lengths)");
    if ((e = hipMemset(p->err, 0, b_err + b_zero)) != hipSuccess) return hip_fail(e, "hipMemset(flags)");
    p->counter = p->err + 16;
    p->queue = p->err + 32;
    p->done = p->err + 48;
    int cus = 0;
    if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, p->device)) != hipSuccess)
        return hip_fail(e, "hipDeviceGetAttribute");
    // one four-wave block per compute unit; never more blocks than items
    p->n_blocks = std::max(1, std::min<int32_t>(p->n_items, cus));
    return FKA_OK;
}

void init_heads(fka_plan *p, const fka_heads *h)
{
    p->Hq = h->n_q_heads;
    p->Hkv = h->n_kv_heads;
    p->d = h->head_dim;
    p->G = p->Hq / p->Hkv;
    p->scale = h->softmax_scale > 0.f ? h->softmax_scale : 1.0f / std::sqrt((float)h->head_dim);
}

fka_status check_split(int32_t split)
{
    REQUIRE(split >= 0 && split % fka::kTileTokens == 0, "split_tokens (%d) must be a non-negative multiple of %d",
            split, fka::kTileTokens);
    return FKA_OK;
}

fka::AttnArgs attn_args(const fka_plan *p)
{
    fka::AttnArgs a{};
    a.items = p->items;
    a.max_suffix_len = p->max_suffix_len;
    a.n_seqs = p->n_seqs;
    a.n_q_heads = p->Hq;
    a.n_kv_heads = p->Hkv;
    a.group = p->G;
    a.scale_log2 = p->scale * 1.4426950408889634f;
    a.part_o = p->part_o;
    a.part_lse = p->part_lse;
    a.err = p->err;
    a.prefix_len = p->prefix_len;
    a.suffix_cap = p->suffix_cap;
    a.max_pages = p->max_pages;
    a.n_pool_pages = p->n_pool_pages;
    a.paged = p->paged ? 1 : 0;
    a.n_items = p->n_items;
    a.queue = p->queue;
    a.done = p->done;
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
    m.seq_prefix_parts = p->seq_prefix_parts;
    m.max_prefix_parts = p->max_prefix_parts;
    m.suffix_len = const_cast<int32_t *>(suffix_len);  // only a fused step writes it
    m.suffix_split = p->ssplit;
    m.max_suffix_len = p->max_suffix_len;
    m.err = p->err;
    m.counter = p->counter;
    m.seq_prefix_len = p->seq_prefix_len;
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
    hipError_t e = fka::launch_partials(a, p->n_blocks, p->d, p->row_tiles, s);
    if (e != hipSuccess) return hip_fail(e, "partials kernel launch");
    e = fka::launch_merge(step ? *step : merge_args(p, suffix_len, out, out_lse), p->d, s);
    if (e != hipSuccess) return hip_fail(e, "merge kernel launch");
    return ok();
}

}  // namespace

extern "C" {

int fka_version(void) { return 10000; }

const char *fka_last_error(void) { return g_err; }

fka_status fka_plan_create_contig(const fka_heads *heads, const fka_contig_desc *desc, fka_plan **out)
{
    REQUIRE(out != nullptr, "out is null");
    *out = nullptr;
    fka_status st = check_heads(heads);
    if (st != FKA_OK) return st;
    REQUIRE(desc != nullptr, "desc is null");
    REQUIRE(desc->n_branches >= 1, "n_branches (%d) must be >= 1", desc->n_branches);
    REQUIRE(desc->prefix_len >= 0, "prefix_len (%d) must be >= 0", desc->prefix_len);
    REQUIRE(desc->suffix_cap >= 1, "suffix_cap (%d) must be >= 1", desc->suffix_cap);
    REQUIRE(desc->max_suffix_len >= 0 && desc->max_suffix_len <= desc->suffix_cap,
            "max_suffix_len (%d) must be in [0, suffix_cap=%d]", desc->max_suffix_len, desc->suffix_cap);
    REQUIRE(desc->share_prefix == 0 || desc->share_prefix == 1, "share_prefix must be 0 or 1");
    if ((st = check_split(desc->split_tokens)) != FKA_OK) return st;
    const int G = heads->n_q_heads / heads->n_kv_heads;
    const int rows = (desc->share_prefix ? desc->n_branches : 1) * G;
    if (G > fka::kMaxRows || rows > fka::kMaxRows)
        return fail(FKA_ERR_UNSUPPORTED, "%d query rows per KV head exceed the limit of %d", rows, fka::kMaxRows);

    fka_plan *p = new (std::nothrow) fka_plan();
    if (!p) return fail(FKA_ERR_NOMEM, "host allocation failed");
    init_heads(p, heads);
    p->n_seqs = desc->n_branches;
    p->share_prefix = desc->share_prefix;
    p->prefix_len = desc->prefix_len;
    p->suffix_cap = desc->suffix_cap;
    p->max_suffix_len = desc->max_suffix_len;
    const int64_t reads = (int64_t)desc->prefix_len * p->Hkv * (desc->share_prefix ? 1 : desc->n_branches);
    p->split = desc->split_tokens ? desc->split_tokens : auto_split(reads);
    p->ssplit = auto_suffix_split(desc->max_suffix_len);
    p->max_prefix_parts = desc->prefix_len > 0 ? ceil_div(desc->prefix_len, p->split) : 0;
    p->n_suffix_parts = desc->max_suffix_len > 0 ? ceil_div(desc->max_suffix_len, p->ssplit) : 0;
    p->slots = p->max_prefix_parts + p->n_suffix_parts;
    p->row_tiles = ceil_div(rows, 16);

    std::vector<WorkItem> items;
    const int N = desc->n_branches;
    for (int part = 0; part < p->max_prefix_parts; ++part)
        for (int g = 0; g < p->Hkv; ++g) {
            const int b0 = part * p->split, b1 = std::min(desc->prefix_len, b0 + p->split);
            if (desc->share_prefix)
                items.push_back({fka::kPrefix, 0, N, g, b0, b1, part, desc->prefix_len});
            else
                for (int b = 0; b < N; ++b) items.push_back({fka::kPrefix, b, 1, g, b0, b1, part, desc->prefix_len});
        }
    for (int s = 0; s < p->n_suffix_parts; ++s)
        for (int b = 0; b < N; ++b)
            for (int g = 0; g < p->Hkv; ++g)
                items.push_back({fka::kSuffix, b, 1, g, s * p->ssplit, (s + 1) * p->ssplit, p->max_prefix_parts + s,
                                 desc->prefix_len});
    std::vector<int32_t> spp(N, p->max_prefix_parts), spl(N, desc->prefix_len);
    st = finish_plan(p, items, spp, spl);
    if (st != FKA_OK) {
        fka_plan_destroy(p);
        return st;
    }
    *out = p;
    return ok();
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
    if ((st = check_split(desc->split_tokens)) != FKA_OK) return st;
    REQUIRE(host_group_start[0] == 0 && host_group_start[desc->n_groups] == desc->n_seqs,
            "group_start must begin at 0 and end at n_seqs");
    const int G = heads->n_q_heads / heads->n_kv_heads;
    int max_group = 0;
    int64_t reads = 0;
    for (int t = 0; t < desc->n_groups; ++t) {
        const int n = host_group_start[t + 1] - host_group_start[t];
        REQUIRE(n >= 1, "group %d is empty", t);
        const int lp = host_group_prefix_len[t];
        REQUIRE(lp >= 0, "group %d has a negative prefix length", t);
        const int64_t pages = ceil_div(lp, fka::kPageSize) + ceil_div(desc->max_suffix_len, fka::kPageSize);
        REQUIRE(pages <= desc->max_pages_per_seq, "group %d needs %lld pages, max_pages_per_seq is %d", t,
                (long long)pages, desc->max_pages_per_seq);
        max_group = std::max(max_group, n);
        reads += (int64_t)lp * heads->n_kv_heads * (desc->share_prefix ? 1 : n);
    }
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
    p->split = desc->split_tokens ? desc->split_tokens : auto_split(reads);
    p->ssplit = auto_suffix_split(desc->max_suffix_len);
    int maxp = 0;
    for (int t = 0; t < desc->n_groups; ++t)
        maxp = std::max(maxp, p->group_prefix_len[t] > 0 ? ceil_div(p->group_prefix_len[t], p->split) : 0);
    p->max_prefix_parts = maxp;
    p->n_suffix_parts = desc->max_suffix_len > 0 ? ceil_div(desc->max_suffix_len, p->ssplit) : 0;
    p->slots = p->max_prefix_parts + p->n_suffix_parts;
    p->row_tiles = ceil_div(rows, 16);

    std::vector<WorkItem> items;
    std::vector<int32_t> spp(desc->n_seqs), spl(desc->n_seqs);
    // prefix items, longest groups first so that the tail of the grid holds short items
    std::vector<int> order(desc->n_groups);
    for (int t = 0; t < desc->n_groups; ++t) order[t] = t;
    std::stable_sort(order.begin(), order.end(),
                     [&](int x, int y) { return p->group_prefix_len[x] > p->group_prefix_len[y]; });
    for (int part = 0; part < maxp; ++part)
        for (int t : order) {
            const int lp = p->group_prefix_len[t];
            const int b0 = part * p->split;
            if (b0 >= lp) continue;
            const int b1 = std::min(lp, b0 + p->split);
            const int s0 = p->group_start[t], s1 = p->group_start[t + 1];
            for (int g = 0; g < p->Hkv; ++g) {
                if (desc->share_prefix)
                    items.push_back({fka::kPrefix, s0, s1 - s0, g, b0, b1, part, lp});
                else
                    for (int i = s0; i < s1; ++i) items.push_back({fka::kPrefix, i, 1, g, b0, b1, part, lp});
            }
        }
    for (int t = 0; t < desc->n_groups; ++t)
        for (int i = p->group_start[t]; i < p->group_start[t + 1]; ++i) {
            const int lp = p->group_prefix_len[t];
            spp[i] = lp > 0 ? ceil_div(lp, p->split) : 0;
            spl[i] = lp;
        }
    for (int s = 0; s < p->n_suffix_parts; ++s)
        for (int t = 0; t < desc->n_groups; ++t)
            for (int i = p->group_start[t]; i < p->group_start[t + 1]; ++i)
                for (int g = 0; g < p->Hkv; ++g)
                    items.push_back({fka::kSuffix, i, 1, g, s * p->ssplit, (s + 1) * p->ssplit,
                                     p->max_prefix_parts + s, p->group_prefix_len[t]});
    st = finish_plan(p, items, spp, spl);
    if (st != FKA_OK) {
        fka_plan_destroy(p);
        return st;
    }
    *out = p;
    return ok();
}

fka_status fka_plan_get_info(const fka_plan *p, fka_plan_info *info)
{
    REQUIRE(p != nullptr && info != nullptr, "null argument");
    info->split_tokens = p->split;
    info->suffix_split_tokens = p->ssplit;
    info->max_prefix_parts = p->max_prefix_parts;
    info->n_suffix_parts = p->n_suffix_parts;
    info->n_items = p->n_items;
    info->workspace_bytes = p->workspace_bytes;
    return ok();
}

fka_status fka_fork_decode(const fka_plan *p, const void *q, const void *prefix_k, const void *prefix_v,
                           const void *suffix_k, const void *suffix_v, const int32_t *suffix_len, float *out,
                           float *out_lse, void *stream)
{
    REQUIRE(p != nullptr, "plan is null");
    REQUIRE(!p->paged, "plan is paged: use fka_fork_decode_paged");
    REQUIRE_PTR16(q);
    if (p->prefix_len > 0) {
        REQUIRE_PTR16(prefix_k);
        REQUIRE_PTR16(prefix_v);
    }
    REQUIRE_PTR16(suffix_k);
    REQUIRE_PTR16(suffix_v);
    REQUIRE(suffix_len != nullptr, "suffix_len is null");
    REQUIRE_PTR16(out);
    fka::AttnArgs a = attn_args(p);
    a.q = static_cast<const uint16_t *>(q);
    a.prefix_k = static_cast<const uint16_t *>(prefix_k);
    a.prefix_v = static_cast<const uint16_t *>(prefix_v);
    a.suffix_k = static_cast<const uint16_t *>(suffix_k);
    a.suffix_v = static_cast<const uint16_t *>(suffix_v);
    a.suffix_len = suffix_len;
    return run_decode(p, a, suffix_len, out, out_lse, static_cast<hipStream_t>(stream));
}

fka_status fka_partials(const fka_plan *p, const void *q, const void *prefix_k, const void *prefix_v,
                        const void *suffix_k, const void *suffix_v, const int32_t *suffix_len, float *part_o,
                        float *part_lse, void *stream)
{
    REQUIRE(p != nullptr, "plan is null");
    REQUIRE(!p->paged, "fka_partials takes a contiguous plan");
    REQUIRE_PTR16(q);
    if (p->prefix_len > 0) {
        REQUIRE_PTR16(prefix_k);
        REQUIRE_PTR16(prefix_v);
    }
    REQUIRE_PTR16(suffix_k);
    REQUIRE_PTR16(suffix_v);
    REQUIRE(suffix_len != nullptr, "suffix_len is null");
    REQUIRE_PTR16(part_o);
    REQUIRE(part_lse != nullptr, "part_lse is null");
    fka::AttnArgs a = attn_args(p);
    a.q = static_cast<const uint16_t *>(q);
    a.prefix_k = static_cast<const uint16_t *>(prefix_k);
    a.prefix_v = static_cast<const uint16_t *>(prefix_v);
    a.suffix_k = static_cast<const uint16_t *>(suffix_k);
    a.suffix_v = static_cast<const uint16_t *>(suffix_v);
    a.suffix_len = suffix_len;
    a.part_o = part_o;
    a.part_lse = part_lse;
    hipError_t e = fka::launch_partials(a, p->n_blocks, p->d, p->row_tiles, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "partials kernel launch");
    return ok();
}

fka_status fka_append_kv(const fka_plan *p, const void *k_new, const void *v_new, void *suffix_k, void *suffix_v,
                         int32_t *suffix_len, void *stream)
{
    REQUIRE(p != nullptr, "plan is null");
    REQUIRE(!p->paged, "plan is paged: use fka_append_kv_paged");
    REQUIRE_PTR16(k_new);
    REQUIRE_PTR16(v_new);
    REQUIRE_PTR16(suffix_k);
    REQUIRE_PTR16(suffix_v);
    REQUIRE(suffix_len != nullptr, "suffix_len is null");
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
    REQUIRE(suffix_len != nullptr, "suffix_len is null");
    REQUIRE_PTR16(out);
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
    REQUIRE_PTR16(q);
    REQUIRE_PTR16(k_new);
    REQUIRE_PTR16(v_new);
    REQUIRE_PTR16(k_pool);
    REQUIRE_PTR16(v_pool);
    REQUIRE(page_table != nullptr, "page_table is null");
    REQUIRE(suffix_len != nullptr, "suffix_len is null");
    REQUIRE_PTR16(out);
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
    REQUIRE_PTR16(q);
    REQUIRE_PTR16(k_pool);
    REQUIRE_PTR16(v_pool);
    REQUIRE(page_table != nullptr, "page_table is null");
    REQUIRE(suffix_len != nullptr, "suffix_len is null");
    REQUIRE_PTR16(out);
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
    REQUIRE_PTR16(k_new);
    REQUIRE_PTR16(v_new);
    REQUIRE_PTR16(k_pool);
    REQUIRE_PTR16(v_pool);
    REQUIRE(page_table != nullptr, "page_table is null");
    REQUIRE(suffix_len != nullptr, "suffix_len is null");
    fka::AppendArgs a{};
    a.k_new = static_cast<const uint16_t *>(k_new);
    a.v_new = static_cast<const uint16_t *>(v_new);
    a.k_dst = static_cast<uint16_t *>(k_pool);
    a.v_dst = static_cast<uint16_t *>(v_pool);
    a.page_table = page_table;
    a.seq_prefix_len = p->seq_prefix_len;
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
    REQUIRE(p != nullptr, "plan is null");
    REQUIRE(p->paged, "plan is contiguous");
    REQUIRE(seq >= 0 && seq < p->n_seqs, "seq %d out of range [0, %d)", seq, p->n_seqs);
    REQUIRE_PTR16(k_pool);
    REQUIRE_PTR16(v_pool);
    REQUIRE(page_table != nullptr, "page_table is null");
    REQUIRE_PTR16(k_out);
    REQUIRE_PTR16(v_out);
    int t = 0;
    while (t + 1 < p->n_groups && p->group_start[t + 1] <= seq) ++t;
    const int lp = p->group_prefix_len[t];
    REQUIRE(out_len >= 0, "out_len must be >= 0");
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
        REQUIRE(part_o != nullptr && part_lse != nullptr, "part arrays are null");
    }
    REQUIRE(out != nullptr, "out is null");
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

}  // extern "C"
