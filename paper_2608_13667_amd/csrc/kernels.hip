// HIP kernels for fork-aware decode attention on gfx950 (CDNA4, wave64).
//
// (the partial-attention kernel over key ranges lives in partials.hip)
// merge_kernel: log-sum-exp combination of the partials of each (sequence, head).
// append_kernel / gather_kernel: suffix append and paged gather (data movement).
#include "internal.h"

namespace fka {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.442695040888963407f;

// One candidate of the schedule cache for the next launch (internal.h), built by merge blocks
// that hold no row: block pb of npb handles items pb, pb + npb, ...  Candidate 0 is for this
// launch's lengths, candidate 1 for the lengths after this fused step's append (one longer where
// there is room).  The key is the lengths a candidate is built for, so lengths that differ at
// the next launch only cost the cache.
__device__ void build_next_schedule(const MergeArgs &a, int cand, int pb, int npb)
{
    constexpr int NTH = 256;
    __shared__ int32_t s_ln[kMaxSeqs], s_cs[kMaxSeqs], s_ne[kMaxSeqs];
    __shared__ int32_t s_sum[2][NTH / 64];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int N = a.n_seqs, Hkv = a.n_kv_heads, G = a.group, NW = a.waves;
    int carry_cs = 0, carry_ne = 0;
    for (int base = 0; base < N; base += NTH) {
        const int s = base + tid;
        int L = 0;
        if (s < N) {
            L = a.lens[s];
            if (cand == 1 && L < a.max_suffix_len) ++L;
            if (pb == 0) a.key_next[cand][s] = L;
        }
        const int xs = slices_of(L) * Hkv, xe = (L > 0) ? Hkv : 0;
        int x = xs, y = xe;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const int ux = __shfl_up(x, off), uy = __shfl_up(y, off);
            if (lane >= off) {
                x += ux;
                y += uy;
            }
        }
        if (lane == 63) {
            s_sum[0][wave] = x;
            s_sum[1][wave] = y;
        }
        __syncthreads();
        int px = carry_cs, py = carry_ne;
        for (int w = 0; w < NTH / 64; ++w) {
            if (w < wave) {
                px += s_sum[0][w];
                py += s_sum[1][w];
            }
            carry_cs += s_sum[0][w];
            carry_ne += s_sum[1][w];
        }
        if (s < N) {
            s_ln[s] = L;
            s_cs[s] = px + x - xs;
            s_ne[s] = py + y - xe;
        }
        __syncthreads();
    }
    const int T = a.pre_slices + carry_cs, NNE = a.pre_nonempty + carry_ne, NV = a.n_workers;
    const uint64_t R = T > 0 ? sched_ratio((int64_t)NV - NNE, T) : 0;
    const int n_items = a.n_pre + N * Hkv;
    // workers past the last item have no work
    const int ws_end = T > 0 ? worker_start(T, NNE, R) : 0;
    if (pb == 0)
        for (int gw = ws_end + tid; gw < NV; gw += NTH) a.tab_next[cand][(size_t)gw * kTabWords] = -1;
    for (int i = pb; i < n_items; i += npb) {
        int seq0, nseq, kvh, n_tok, size, C, K;
        if (i < a.n_pre) {
            const PrefixItem it = a.pre_items[i];
            seq0 = it.seq0;
            nseq = it.nseq;
            kvh = it.kv_head;
            n_tok = it.n_tok;
            size = slices_of(n_tok);
            C = it.c0;
            K = it.k0;
        } else {
            const int j = i - a.n_pre, sq = j / Hkv;
            seq0 = sq;
            nseq = 1;
            kvh = j % Hkv;
            n_tok = s_ln[sq];
            size = slices_of(n_tok);
            C = a.pre_slices + s_cs[sq] + kvh * size;
            K = a.pre_nonempty + s_ne[sq] + (size > 0 ? kvh : 0);
        }
        int ws0 = 0, ws1 = 0;
        if (size > 0 && T > 0) {
            ws0 = worker_start(C, K, R);
            ws1 = worker_start(C + size, K + 1, R);
        }
        // slot records of the item's rows
        const int field = i < a.n_pre ? 0 : 2;
        const int vb0 = ws0 / NW, count = ws1 > ws0 ? (ws1 - 1) / NW - vb0 + 1 : 0;
        for (int r = tid; r < nseq * G; r += NTH) {
            int32_t *rr = a.rowrec_next[cand] + ((size_t)(seq0 + r / G) * a.n_q_heads + kvh * G + r % G) * kRowRec + field;
            rr[0] = (vb0 + i) * a.slot_rows + r;
            rr[1] = count;
        }
        // table rows of the item's workers
        for (int gw = ws0 + tid; gw < ws1; gw += NTH) {
            const int vb = gw / NW;
            int lo, hi, glo, ghi;
            block_group(vb, NW, ws0, ws1, size, lo, hi, glo, ghi);
            int32_t *t = a.tab_next[cand] + (size_t)gw * kTabWords;
            t[0] = i;
            t[1] = seq0;
            t[2] = nseq;
            t[3] = kvh;
            t[4] = n_tok;
            t[5] = lo - vb * NW;
            t[6] = glo;
            t[7] = ghi;
            t[8] = hi - vb * NW;
        }
    }
}

template <int HD>
__global__ __launch_bounds__(256) void merge_kernel(MergeArgs a)
{
    constexpr int CH = HD / 4;    // float4 chunks per row
    constexpr int SL = 256 / CH;  // part slices: slice k takes parts k, k + SL, ...
    __shared__ float s_m[SL], s_w[SL];
    __shared__ f32x4 s_acc[SL][CH];
    __shared__ float s_new;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int chunk = tid % CH, slice = tid / CH;
    const int row = blockIdx.x;
    if (row >= a.rows) {  // the blocks past the rows build the schedule cache of the next launch
        const int per = a.step_mode ? ((int)gridDim.x - a.rows) / 2 : (int)gridDim.x - a.rows;
        const int pb = row - a.rows;
        if (pb < per) {
            if (!a.step_mode && pb == 0 && tid == 0) a.key_next[1][0] = -1;  // no candidate 1
            build_next_schedule(a, 0, pb, per);
        } else {
            build_next_schedule(a, 1, pb - per, per);
        }
        return;
    }

    // Everything this block reads first is requested together: the row's slot records and the
    // schedule choice (plan mode) and, in a fused step, q and the appended key and value.
    // Parts of this row, as offsets (part index * row stride + row) into part_o / part_lse:
    // parts [0, np) start at p_first with stride p_step; parts [np, n) at s_first.
    int np = 0, n = 0, L = 0, seq = 0, g = 0;
    int64_t p_first = 0, p_step = 0, s_first = 0;
    bool with_new = false;  // fused step: the appended token is one more part, read from k_new / v_new
    float dot = 0.f;
    uint4 app_k = {0, 0, 0, 0}, app_v = {0, 0, 0, 0};  // fused step, block (s, 0): the token to store
    uint2 new_v = {0, 0};                              // fused step: this thread's 4 values of v_new
    constexpr int APP = HD / 8;                        // 16-byte chunks of one K/V row
    if (a.rowrec[0]) {
        seq = row / a.n_q_heads;
        g = (row % a.n_q_heads) / a.group;
        // the records of the schedule the partial kernel used (loaded together, then chosen)
        const int sel = *a.sel;
        const int4 r0 = *reinterpret_cast<const int4 *>(a.rowrec[0] + (size_t)row * kRowRec);
        const int4 r1 = *reinterpret_cast<const int4 *>(a.rowrec[1] + (size_t)row * kRowRec);
        const int4 r2 = *reinterpret_cast<const int4 *>(a.rowrec[2] + (size_t)row * kRowRec);
        const int4 rec = sel == 0 ? r0 : sel == 1 ? r1 : r2;
        L = a.lens[seq];
        if (a.step_mode && row % a.n_q_heads == 0 && tid < a.n_kv_heads * APP) {
            const size_t src = ((size_t)seq * a.n_kv_heads + tid / APP) * HD + 8 * (tid % APP);
            app_k = *reinterpret_cast<const uint4 *>(a.k_new + src);
            app_v = *reinterpret_cast<const uint4 *>(a.v_new + src);
        }
        with_new = a.step_mode && L < a.max_suffix_len;
        if (a.step_mode && slice == 0)
            new_v = *reinterpret_cast<const uint2 *>(a.v_new + ((size_t)seq * a.n_kv_heads + g) * HD + 4 * chunk);
        if (with_new && wave == 0) {  // q . k_new, wave 0
            const uint16_t *qr = a.q + (size_t)row * HD;
            const uint16_t *kr = a.k_new + ((size_t)seq * a.n_kv_heads + g) * HD;
            for (int c = lane; c < HD; c += 64)
                dot += __uint_as_float((uint32_t)qr[c] << 16) * __uint_as_float((uint32_t)kr[c] << 16);
        }
        // a record that points outside the workspace (it cannot, unless the cache was
        // overwritten from outside) is dropped and flagged rather than followed
        const int64_t lim = (int64_t)a.n_slots * a.slot_rows;
        const bool p_ok = rec.y >= 0 && rec.x >= 0 && (int64_t)rec.x + (int64_t)max(rec.y - 1, 0) * a.slot_rows < lim;
        const bool s_ok = rec.w >= 0 && rec.z >= 0 && (int64_t)rec.z + (int64_t)max(rec.w - 1, 0) * a.slot_rows < lim;
        if ((!p_ok || !s_ok) && tid == 0) atomicOr(a.err, kErrBadSchedule);
        p_first = rec.x;
        np = p_ok ? rec.y : 0;
        s_first = rec.z;
        n = np + (s_ok ? rec.w : 0);
        p_step = a.slot_rows;
    } else {
        np = n = a.n_parts;
        p_first = row;
        p_step = a.rows;
    }
    auto part_off = [&](int j) -> int64_t { return j < np ? p_first + j * p_step : s_first + (j - np) * p_step; };

    // Online merge of this slice's parts: running max m, weight sum w and accumulator (each
    // part's lse and o are loaded together).  An empty part (lse = -inf) has weight 0; a NaN
    // lse propagates.
    float m = -INFINITY, w = 0.f;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    constexpr int U = 4;  // parts loaded ahead of their use
    for (int j0 = slice; j0 < n; j0 += U * SL) {
        float l[U];
        f32x4 o[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int j = j0 + u * SL;
            l[u] = -INFINITY;
            o[u] = f32x4{0.f, 0.f, 0.f, 0.f};
            if (j < n) {
                const int64_t off = part_off(j);
                l[u] = a.part_lse[off];
                o[u] = *reinterpret_cast<const f32x4 *>(a.part_o + (size_t)off * HD + 4 * chunk);
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (l[u] == -INFINITY) continue;
            const float mn = fmaxf(m, l[u]);
            const float sc = (m == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f((m - mn) * kLog2e);
            const float e = __builtin_amdgcn_exp2f((l[u] - mn) * kLog2e);
            w = w * sc + e;
            acc = acc * sc + e * o[u];
            m = mn;
        }
    }
    if (chunk == 0) {
        s_m[slice] = m;
        s_w[slice] = w;
    }
    s_acc[slice][chunk] = acc;
    if (with_new && wave == 0) {
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) dot += __shfl_xor(dot, off);
        if (lane == 0) s_new = dot * a.scale;
    }
    __syncthreads();
    const float lse_new = with_new ? s_new : -INFINITY;
    float M = lse_new;
#pragma unroll
    for (int k = 0; k < SL; ++k) M = fmaxf(M, s_m[k]);
    if (slice == 0) {
        f32x4 t = {0.f, 0.f, 0.f, 0.f};
        float W = 0.f;
        if (M != -INFINITY) {
#pragma unroll
            for (int k = 0; k < SL; ++k) {
                const float sc = (s_m[k] == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f((s_m[k] - M) * kLog2e);
                t += sc * s_acc[k][chunk];
                W += sc * s_w[k];
            }
            if (with_new) {
                const float e = __builtin_amdgcn_exp2f((lse_new - M) * kLog2e);
                W += e;
                t += e * f32x4{__uint_as_float(new_v.x << 16), __uint_as_float(new_v.x & 0xffff0000u),
                               __uint_as_float(new_v.y << 16), __uint_as_float(new_v.y & 0xffff0000u)};
            }
        }
        const f32x4 r = (W == 0.f) ? f32x4{0.f, 0.f, 0.f, 0.f} : t * __builtin_amdgcn_rcpf(W);
        *reinterpret_cast<f32x4 *>(a.out + (size_t)row * HD + 4 * chunk) = r;
        if (a.out_lse && chunk == 0) a.out_lse[row] = (W == 0.f) ? -INFINITY : M + logf(W);
    }

    // Fused step: block (s, head 0) stores the token sequence s appended (already attended
    // to from k_new / v_new) and advances suffix_len[s].  No block of this kernel reads the
    // suffix cache or suffix_len (the lengths come from the partial kernel), so nothing races.
    if (!a.step_mode || row % a.n_q_heads != 0) return;
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

}  // namespace

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
    const int n_items = a.n_pre + a.n_seqs * a.n_kv_heads;
    const int producers = a.tab_next[0] ? (n_items < 64 ? n_items : 64) * (a.step_mode ? 2 : 1) : 0;
    const dim3 grid(a.rows + producers), block(256);
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
