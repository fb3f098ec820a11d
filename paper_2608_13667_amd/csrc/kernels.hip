// HIP kernels for fork-aware decode attention on gfx950 (CDNA4, wave64).
//
// (the partial-attention kernel over key ranges lives in partials.hip)
// merge_kernel: log-sum-exp combination of the partials of each (sequence, head).
// append_kernel / gather_kernel: suffix append and paged gather (data movement).
#include "internal.h"
#include "merge_row.h"

namespace fka {
namespace {

template <int HD>
__global__ __launch_bounds__(256) void merge_kernel(MergeArgs a)
{
    __shared__ MergeLds<HD> lds;
    constexpr int APP = HD / 8;  // 16-byte chunks of one K/V row
    const int tid = threadIdx.x;
    const int row = blockIdx.x;

    // Everything this block reads is requested together: under a static split the row's parts
    // (their slots follow from the plan) with, in a fused step, the length, q and the appended
    // key and value; under a proportional split the row's record first.
    RowMerge m{};
    m.part_o = a.part_o;
    m.part_lse = a.part_lse;
    m.out_row = a.out + (size_t)row * HD;
    m.out_lse = a.out_lse ? a.out_lse + row : nullptr;
    int seq = 0;
    uint4 app_k = {0, 0, 0, 0}, app_v = {0, 0, 0, 0};  // fused step, block (s, 0): the token to store
    if (a.plan) {
        seq = row / a.n_q_heads;
        const int h = row % a.n_q_heads;
        const int g = h / a.group;
        m.p_step = a.slot_rows;
        if (a.static_split) {
            // item g owns workers [floor(g NV / Hkv), floor((g+1) NV / Hkv)); its blocks write
            // their partials to slots vb + g; the one unit starts at sequence 0
            const int ws0 = static_start(g, a.n_workers, a.n_kv_heads);
            const int ws1 = static_start(g + 1, a.n_workers, a.n_kv_heads);
            const int vb0 = ws0 / a.waves;
            m.n = ws1 > ws0 ? (ws1 - 1) / a.waves - vb0 + 1 : 0;
            m.p_first = (int64_t)(vb0 + g) * a.slot_rows + (int64_t)seq * a.group + (h - g * a.group);
        } else {
            const int2 rec = *reinterpret_cast<const int2 *>(a.rowrec + (size_t)row * kRowRec);
            // a record that points outside the workspace (it cannot, unless the workspace was
            // overwritten from outside) is dropped and flagged rather than followed
            const int64_t lim = (int64_t)a.n_slots * a.slot_rows;
            const bool ok = rec.y >= 0 && rec.x >= 0 && (int64_t)rec.x + (int64_t)max(rec.y - 1, 0) * a.slot_rows < lim;
            if (!ok && tid == 0) atomicOr(a.err, kErrBadSchedule);
            m.p_first = rec.x;
            m.n = ok ? rec.y : 0;
        }
        if (a.step_mode) {
            m.step = 1;
            m.L = a.lens[seq];
            m.max_len = a.max_suffix_len;
            m.q_row = a.q + (size_t)row * HD;
            m.k_row = a.k_new + ((size_t)seq * a.n_kv_heads + g) * HD;
            m.v_row = a.v_new + ((size_t)seq * a.n_kv_heads + g) * HD;
            m.scale = a.scale;
            if (h == 0 && tid < a.n_kv_heads * APP) {
                const size_t src = ((size_t)seq * a.n_kv_heads + tid / APP) * HD + 8 * (tid % APP);
                app_k = *reinterpret_cast<const uint4 *>(a.k_new + src);
                app_v = *reinterpret_cast<const uint4 *>(a.v_new + src);
            }
        }
    } else {
        m.n = a.n_parts;
        m.p_first = row;
        m.p_step = a.rows;
    }
    merge_row<HD>(m, lds);

    // Fused step: block (s, head 0) stores the token sequence s appended (already attended
    // to from k_new / v_new) and advances suffix_len[s].  No block of this kernel reads the
    // suffix cache or suffix_len (the lengths come from the partial kernel), so nothing races.
    if (!a.step_mode || row % a.n_q_heads != 0) return;
    const int L = m.L;
    bool ok = L < a.max_suffix_len;
    int page = 0;
    if (ok && a.paged) {
        const int pidx = (a.seq_prefix_len[seq] + kPageSize - 1) / kPageSize + L / kPageSize;
        page = pidx < a.max_pages ? a.page_table[(size_t)seq * a.max_pages + pidx] : -1;
        ok = page >= 0 && page < a.n_pool_pages;
    }
    if (ok) {
        for (int c = tid; c < a.n_kv_heads * APP; c += 256) {
            const int gg = c / APP, cc = c % APP;
            const size_t dst =
                a.paged ? (((size_t)page * a.n_kv_heads + gg) * kPageSize + L % kPageSize) * HD + 8 * cc
                        : (((size_t)seq * a.n_kv_heads + gg) * a.suffix_cap + L) * HD + 8 * cc;
            uint4 kk = app_k, vv = app_v;  // loaded at the start (the first 256 chunks)
            if (c >= 256) {
                const size_t src = ((size_t)seq * a.n_kv_heads + gg) * HD + 8 * cc;
                kk = *reinterpret_cast<const uint4 *>(a.k_new + src);
                vv = *reinterpret_cast<const uint4 *>(a.v_new + src);
            }
            *reinterpret_cast<uint4 *>(a.k_dst + dst) = kk;
            *reinterpret_cast<uint4 *>(a.v_dst + dst) = vv;
        }
    }
    if (tid == 0) {
        if (ok)
            a.suffix_len[seq] = L + 1;
        else
            atomicOr(a.err, kErrAppendNoRoom);
    }
}

__global__ __launch_bounds__(256) void append_kernel(AppendArgs a)
{
    const int seq = blockIdx.x;
    __shared__ int s_row, s_page;
    if (threadIdx.x == 0) {
        const int L = a.suffix_len[seq];
        bool ok = L >= 0 && L < a.max_suffix_len;
        int page = 0;
        if (ok && a.paged) {
            const int lp = a.seq_prefix_len[seq];
            const int pidx = (lp + kPageSize - 1) / kPageSize + L / kPageSize;
            page = pidx < a.max_pages ? a.page_table[(size_t)seq * a.max_pages + pidx] : -1;
            ok = page >= 0 && page < a.n_pool_pages;
        }
        if (!ok) atomicOr(a.err, kErrAppendNoRoom);
        s_row = ok ? L : -1;
        s_page = page;
    }
    __syncthreads();
    const int row = s_row;
    if (row < 0) return;
    const int cpr = a.head_dim / 8;
    const int chunks = a.n_kv_heads * cpr;
    for (int c = threadIdx.x; c < chunks; c += blockDim.x) {
        const int g = c / cpr, cc = c % cpr;
        const size_t src = ((size_t)seq * a.n_kv_heads + g) * a.head_dim + 8 * cc;
        size_t dst;
        if (a.paged)
            dst = (((size_t)s_page * a.n_kv_heads + g) * kPageSize + row % kPageSize) * a.head_dim + 8 * cc;
        else
            dst = (((size_t)seq * a.n_kv_heads + g) * a.suffix_cap + row) * a.head_dim + 8 * cc;
        *reinterpret_cast<uint4 *>(a.k_dst + dst) = *reinterpret_cast<const uint4 *>(a.k_new + src);
        *reinterpret_cast<uint4 *>(a.v_dst + dst) = *reinterpret_cast<const uint4 *>(a.v_new + src);
    }
    __syncthreads();
    if (threadIdx.x == 0) a.suffix_len[seq] = row + 1;
}

// grid (ceil((out_len - begin) / 16), Hkv): block copies 16 logical positions of one KV head.
__global__ __launch_bounds__(256) void gather_kernel(GatherArgs a)
{
    const int g = blockIdx.y;
    const int cpr = a.head_dim / 8;
    for (int i = threadIdx.x; i < kPageSize * cpr; i += blockDim.x) {
        const int pos = a.begin + blockIdx.x * kPageSize + i / cpr, c = i % cpr;
        if (pos >= a.out_len) continue;
        int pidx, slot;
        if (pos < a.prefix_len) {
            pidx = pos / kPageSize;
            slot = pos % kPageSize;
        } else {
            const int u = pos - a.prefix_len;
            pidx = (a.prefix_len + kPageSize - 1) / kPageSize + u / kPageSize;
            slot = u % kPageSize;
        }
        const int page = a.page_table[(size_t)a.seq * a.max_pages + pidx];
        const size_t dst = ((size_t)g * (a.out_len - a.begin) + (pos - a.begin)) * a.head_dim + 8 * c;
        uint4 kv = uint4{0, 0, 0, 0}, vv = uint4{0, 0, 0, 0};
        if (page >= 0 && page < a.n_pool_pages) {
            const size_t src = (((size_t)page * a.n_kv_heads + g) * kPageSize + slot) * a.head_dim + 8 * c;
            kv = *reinterpret_cast<const uint4 *>(a.k_pool + src);
            vv = *reinterpret_cast<const uint4 *>(a.v_pool + src);
        } else {
            atomicOr(a.err, kErrBadPage);
        }
        *reinterpret_cast<uint4 *>(a.k_out + dst) = kv;
        *reinterpret_cast<uint4 *>(a.v_out + dst) = vv;
    }
}

// grid (pages covering [from, len), Hkv): block copies the positions of one page of one KV head
// from the contiguous source into the pool's dense layout.
__global__ __launch_bounds__(256) void scatter_kernel(ScatterArgs a)
{
    const int g = blockIdx.y;
    const int pidx = a.from / kPageSize + blockIdx.x;
    const int page = a.page_row[pidx];
    if (page < 0 || page >= a.n_pool_pages) {
        if (threadIdx.x == 0 && a.err) atomicOr(a.err, kErrBadPage);
        return;
    }
    const int cpr = a.head_dim / 8;
    for (int i = threadIdx.x; i < kPageSize * cpr; i += blockDim.x) {
        const int slot = i / cpr, c = i % cpr, pos = pidx * kPageSize + slot;
        if (pos < a.from || pos >= a.len) continue;
        const size_t src = ((size_t)g * (a.len - a.from) + (pos - a.from)) * a.head_dim + 8 * c;
        const size_t dst = (((size_t)page * a.n_kv_heads + g) * kPageSize + slot) * a.head_dim + 8 * c;
        *reinterpret_cast<uint4 *>(a.k_pool + dst) = *reinterpret_cast<const uint4 *>(a.k_src + src);
        *reinterpret_cast<uint4 *>(a.v_pool + dst) = *reinterpret_cast<const uint4 *>(a.v_src + src);
    }
}

// Read-only streaming probe: block b reads the 16-byte words [b * chunk, (b + 1) * chunk) of the
// buffer, its threads interleaved, U loads in flight per thread, non-temporal like the K/V
// stream of the partial kernel; the words are folded into one value so the loads are kept.
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

template <int U>
__global__ void read_probe_kernel(const u32x4 *__restrict__ p, size_t n_vec, size_t chunk, uint32_t *sink)
{
    const size_t b0 = (size_t)blockIdx.x * chunk;
    const size_t e = b0 + chunk < n_vec ? b0 + chunk : n_vec;
    const size_t step = blockDim.x;
    uint32_t acc = 0;
    size_t i = b0 + threadIdx.x;
    for (; i + (U - 1) * step < e; i += U * step) {
        u32x4 v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) v[u] = __builtin_nontemporal_load(p + i + u * step);
#pragma unroll
        for (int u = 0; u < U; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
    }
    for (; i < e; i += step) {
        const u32x4 v = __builtin_nontemporal_load(p + i);
        acc ^= v.x ^ v.y ^ v.z ^ v.w;
    }
    if (acc == 0x9e3779b9u) sink[blockIdx.x % 64] = acc;  // practically never: keeps the loads alive
}

}  // namespace

hipError_t launch_read_probe(const void *buf, size_t bytes, int blocks, int threads, int unroll, uint32_t *sink,
                             hipStream_t s)
{
    const size_t n_vec = bytes / 16;
    const size_t chunk = (n_vec + blocks - 1) / blocks;
    const u32x4 *p = static_cast<const u32x4 *>(buf);
    switch (unroll) {
    case 4: read_probe_kernel<4><<<blocks, threads, 0, s>>>(p, n_vec, chunk, sink); break;
    case 8: read_probe_kernel<8><<<blocks, threads, 0, s>>>(p, n_vec, chunk, sink); break;
    case 16: read_probe_kernel<16><<<blocks, threads, 0, s>>>(p, n_vec, chunk, sink); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_scatter(const ScatterArgs &a, hipStream_t s)
{
    if (a.len <= a.from) return hipSuccess;
    const int blocks = (a.len + kPageSize - 1) / kPageSize - a.from / kPageSize;
    scatter_kernel<<<dim3(blocks, a.n_kv_heads), dim3(256), 0, s>>>(a);
    return hipGetLastError();
}

hipError_t launch_merge(const MergeArgs &a, int head_dim, hipStream_t s)
{
    if (a.rows <= 0) return hipSuccess;
    const dim3 grid(a.rows), block(256);
    if (head_dim == 128)
        merge_kernel<128><<<grid, block, 0, s>>>(a);
    else if (head_dim == 64)
        merge_kernel<64><<<grid, block, 0, s>>>(a);
    else
        return hipErrorInvalidValue;
    return hipGetLastError();
}

hipError_t launch_append(const AppendArgs &a, int n_seqs, hipStream_t s)
{
    if (n_seqs <= 0) return hipSuccess;
    append_kernel<<<dim3(n_seqs), dim3(256), 0, s>>>(a);
    return hipGetLastError();
}

hipError_t launch_gather(const GatherArgs &a, hipStream_t s)
{
    if (a.out_len <= a.begin) return hipSuccess;
    gather_kernel<<<dim3((a.out_len - a.begin + kPageSize - 1) / kPageSize, a.n_kv_heads), dim3(256), 0, s>>>(a);
    return hipGetLastError();
}

}  // namespace fka
