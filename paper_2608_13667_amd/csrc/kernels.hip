// HIP kernels for fork-aware decode attention on gfx950 (CDNA4, wave64).
//
// partials_kernel: one block per work item = (query-row set, KV head, key range).
//   The block streams its key range in tiles of 128 tokens: each tile of K and V
//   is read from HBM once with coalesced 16-byte loads, staged in LDS, and scored
//   against every query row of the item (for a shared-prefix item: all sequences
//   of the fork x the G query heads of the KV head, Sec. 3.3 of the paper).
//   Scores and the probability-weighted sum of values run on MFMA
//   (v_mfma_f32_16x16x32_bf16) with fp32 accumulation, tokens on the M side so
//   that each lane owns one query row of the softmax.  The online softmax keeps a
//   running max and sum per row; the block ends with a cross-wave combine and
//   writes one normalised partial (o, lse) per row.
// merge_kernel: log-sum-exp combination of the partials of each (sequence, head).
// append_kernel / gather_kernel: suffix append and paged gather (data movement).
#include "internal.h"

namespace fka {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef unsigned short u16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr float kLn2 = 0.693147180559945309f;
constexpr float kLog2e = 1.442695040888963407f;

__device__ inline f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ inline float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Where the rows of one work item live.
struct Source {
    const uint16_t *k;
    const uint16_t *v;
    const int32_t *pt;  // paged: page-table row of the item's sequence
    int32_t page_off;   // paged: page index of the item's position 0
    int32_t kvh;
    int32_t n_kv_heads;
    int32_t n_pool_pages;
    bool paged;
};

// Element offset of key/value row t of the source, or -1 if its page id is invalid.
template <int HD>
__device__ inline long long row_offset(const Source &s, int t)
{
    if (!s.paged) return (long long)t * HD;
    const int page = s.pt[s.page_off + t / kPageSize];
    if (page < 0 || page >= s.n_pool_pages) return -1;
    return ((long long)(page * s.n_kv_heads + s.kvh) * kPageSize + (t % kPageSize)) * HD;
}

template <int HD, int NT>
__global__ __launch_bounds__(kThreads) void partials_kernel(AttnArgs a)
{
    constexpr int CPR = HD / 8;                           // 16-byte chunks per K/V row
    constexpr int LOADS = kTileTokens * CPR / kThreads;   // 16-byte loads per thread per tensor per tile
    constexpr int NC = HD / 32;                           // MFMA k-steps of q.k
    constexpr int NE = HD / 16;                           // MFMA d-tiles of p.v
    constexpr int OSTRIDE = HD + 4;                       // padded fp32 row stride of the output staging
    static_assert(kWaves * 16 * OSTRIDE * 4 <= kTileTokens * CPR * 16 * 2, "staging fits in the tile buffer");

    // K tile at [0, T*CPR), V tile at [T*CPR, 2*T*CPR); chunk c of token t sits at
    // t*CPR + (c ^ (t % CPR)) so that column reads by 16 lanes hit distinct banks.
    __shared__ uint4 lds[2 * kTileTokens * CPR];
    __shared__ float red_m[kWaves][NT][16];
    __shared__ float red_l[kWaves][NT][16];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int l16 = lane & 15, q4 = lane >> 4;

    const WorkItem it = a.items[blockIdx.x];
    const int G = a.group, kvh = it.kv_head;
    const int rows = it.nseq * G;

    Source src;
    src.paged = a.paged != 0;
    src.kvh = kvh;
    src.n_kv_heads = a.n_kv_heads;
    src.n_pool_pages = a.n_pool_pages;
    src.pt = nullptr;
    src.page_off = 0;
    int tok_end = it.tok_end;
    if (it.kind == kSuffix) {
        const int L = min(max(a.suffix_len[it.seq0], 0), a.max_suffix_len);
        tok_end = min(tok_end, L);
        if (src.paged) {
            src.k = a.k_pool;
            src.v = a.v_pool;
            src.pt = a.page_table + (size_t)it.seq0 * a.max_pages;
            src.page_off = (it.prefix_len + kPageSize - 1) / kPageSize;
        } else {
            const size_t base = ((size_t)it.seq0 * a.n_kv_heads + kvh) * (size_t)a.suffix_cap * HD;
            src.k = a.suffix_k + base;
            src.v = a.suffix_v + base;
        }
    } else {
        if (src.paged) {
            src.k = a.k_pool;
            src.v = a.v_pool;
            src.pt = a.page_table + (size_t)it.seq0 * a.max_pages;
        } else {
            const size_t base = (size_t)kvh * (size_t)a.prefix_len * HD;
            src.k = a.prefix_k + base;
            src.v = a.prefix_v + base;
        }
    }
    const int n_tok = tok_end - it.tok_begin;
    if (n_tok <= 0) return;  // a suffix part past the branch's length: the merge does not read it

    // query rows as the B operand of S^T = K Q^T: lane holds row 16t + l16, d = 32c + 8*q4 .. +7
    bf16x8 qb[NT][NC];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        const int r = 16 * t + l16;
        if (r < rows) {
            const int seq = it.seq0 + r / G, h = kvh * G + r % G;
            const uint16_t *qp = a.q + ((size_t)seq * a.n_q_heads + h) * HD + 8 * q4;
#pragma unroll
            for (int c = 0; c < NC; ++c) qb[t][c] = *reinterpret_cast<const bf16x8 *>(qp + 32 * c);
        } else {
#pragma unroll
            for (int c = 0; c < NC; ++c) qb[t][c] = bf16x8{};
        }
    }

    f32x4 acc[NT][NE];
    float m_run[NT], l_run[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        m_run[t] = -INFINITY;
        l_run[t] = 0.f;
#pragma unroll
        for (int e = 0; e < NE; ++e) acc[t][e] = f32x4{0.f, 0.f, 0.f, 0.f};
    }

    uint4 kr[LOADS], vr[LOADS];
    bool bad_page = false;
    auto load_tile = [&](int ti) {
        const int t0 = it.tok_begin + ti * kTileTokens;
#pragma unroll
        for (int r = 0; r < LOADS; ++r) {
            const int p = r * kThreads + tid;
            const int t = t0 + p / CPR, c = p % CPR;
            uint4 kv = uint4{0, 0, 0, 0}, vv = uint4{0, 0, 0, 0};
            if (t < tok_end) {
                const long long off = row_offset<HD>(src, t);
                if (off >= 0) {
                    kv = *reinterpret_cast<const uint4 *>(src.k + off + 8 * c);
                    vv = *reinterpret_cast<const uint4 *>(src.v + off + 8 * c);
                } else {
                    bad_page = true;
                }
            }
            kr[r] = kv;
            vr[r] = vv;
        }
    };

    const int n_tiles = (n_tok + kTileTokens - 1) / kTileTokens;
    load_tile(0);
    for (int ti = 0; ti < n_tiles; ++ti) {
        __syncthreads();  // every wave is done reading the previous tile
#pragma unroll
        for (int r = 0; r < LOADS; ++r) {
            const int p = r * kThreads + tid;
            const int tt = p / CPR, c = p % CPR;
            const int slot = tt * CPR + (c ^ (tt % CPR));
            lds[slot] = kr[r];
            lds[kTileTokens * CPR + slot] = vr[r];
        }
        __syncthreads();
        if (ti + 1 < n_tiles) load_tile(ti + 1);  // in flight while this tile is scored

        const int valid = n_tok - ti * kTileTokens - 32 * wave;  // keys present in this wave's 32-token slice
        if (valid > 0) {
            // K as the A operand: lane holds token 16u + l16 of the slice, d = 32c + 8*q4 .. +7
            bf16x8 ka[2][NC];
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                const int T = 32 * wave + 16 * u + l16;
#pragma unroll
                for (int c = 0; c < NC; ++c) {
                    const int cc = 4 * c + q4;
                    ka[u][c] = *reinterpret_cast<const bf16x8 *>(&lds[T * CPR + (cc ^ (T % CPR))]);
                }
            }
            bf16x8 ph[NT], pl[NT];
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int c = 0; c < NC; ++c) {
                    s0 = mfma16(ka[0][c], qb[t][c], s0);
                    s1 = mfma16(ka[1][c], qb[t][c], s1);
                }
                // lane holds scores of row 16t + l16 for slice tokens 4*q4 + j and 16 + 4*q4 + j
                float x[8];
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    x[j] = (4 * q4 + j < valid) ? s0[j] * a.scale_log2 : -INFINITY;
                    x[4 + j] = (16 + 4 * q4 + j < valid) ? s1[j] * a.scale_log2 : -INFINITY;
                }
                float mx = x[0];
#pragma unroll
                for (int i = 1; i < 8; ++i) mx = fmaxf(mx, x[i]);
                mx = fmaxf(mx, __shfl_xor(mx, 16));
                mx = fmaxf(mx, __shfl_xor(mx, 32));
                const float m_new = fmaxf(m_run[t], mx);
                const float m_use = (m_new == -INFINITY) ? 0.f : m_new;
                const float alpha = fast_exp2(m_run[t] - m_use);
                m_run[t] = m_new;
                float ps = 0.f;
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    const float p = fast_exp2(x[i] - m_use);
                    ps += p;
                    // p = hi + lo in two bf16 terms keeps the p.v product accurate to ~2^-16
                    const __bf16 hi = (__bf16)p;
                    ph[t][i] = hi;
                    pl[t][i] = (__bf16)(p - (float)hi);
                }
                l_run[t] = l_run[t] * alpha + ps;
#pragma unroll
                for (int e = 0; e < NE; ++e) acc[t][e] *= alpha;
            }
            // V^T as the A operand of O^T = V^T P^T: lane holds d = 16e + l16 and the
            // slice tokens 16*(i/4) + 4*q4 + i%4, the same token order as the P operand.
            const unsigned short *lv = reinterpret_cast<const unsigned short *>(&lds[kTileTokens * CPR]);
#pragma unroll
            for (int e = 0; e < NE; ++e) {
                const int d = 16 * e + l16;
                u16x8 vv;
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    const int T = 32 * wave + 16 * (i >> 2) + 4 * q4 + (i & 3);
                    vv[i] = lv[(T * CPR + ((d >> 3) ^ (T % CPR))) * 8 + (d & 7)];
                }
                const bf16x8 va = __builtin_bit_cast(bf16x8, vv);
#pragma unroll
                for (int t = 0; t < NT; ++t) {
                    acc[t][e] = mfma16(va, ph[t], acc[t][e]);
                    acc[t][e] = mfma16(va, pl[t], acc[t][e]);
                }
            }
        }
    }
    if (bad_page) atomicOr(a.err, kErrBadPage);

    // combine the four waves' (max, sum, accumulator) per row and write the partial
    __syncthreads();
    float *lds_o = reinterpret_cast<float *>(lds);  // [kWaves][16][OSTRIDE]
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        float ls = l_run[t];
        ls += __shfl_xor(ls, 16);
        ls += __shfl_xor(ls, 32);
        if (q4 == 0) {
            red_m[wave][t][l16] = m_run[t];
            red_l[wave][t][l16] = ls;
        }
    }
    __syncthreads();
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        float M = -INFINITY;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) M = fmaxf(M, red_m[w][t][l16]);
        const float Mu = (M == -INFINITY) ? 0.f : M;
        float L = 0.f;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) L += red_l[w][t][l16] * fast_exp2(red_m[w][t][l16] - Mu);
        const float f = (L > 0.f) ? fast_exp2(m_run[t] - Mu) / L : 0.f;
#pragma unroll
        for (int e = 0; e < NE; ++e)
            *reinterpret_cast<f32x4 *>(&lds_o[(wave * 16 + l16) * OSTRIDE + 16 * e + 4 * q4]) = acc[t][e] * f;
        __syncthreads();
        {
            constexpr int PER = HD / 16;  // floats per thread: 16 threads cover one row
            const int r = tid >> 4, d0 = (tid & 15) * PER;
            const int row = 16 * t + r;
            if (row < rows) {
                const int seq = it.seq0 + row / G, h = kvh * G + row % G;
                float o[PER];
#pragma unroll
                for (int k = 0; k < PER; ++k) o[k] = 0.f;
#pragma unroll
                for (int w = 0; w < kWaves; ++w)
#pragma unroll
                    for (int k = 0; k < PER; ++k) o[k] += lds_o[(w * 16 + r) * OSTRIDE + d0 + k];
                float *dst = a.part_o + (((size_t)it.part * a.n_seqs + seq) * a.n_q_heads + h) * HD + d0;
#pragma unroll
                for (int k = 0; k < PER; k += 4)
                    *reinterpret_cast<f32x4 *>(dst + k) = f32x4{o[k], o[k + 1], o[k + 2], o[k + 3]};
                if ((tid & 15) == 0) {
                    float Mr = -INFINITY;
#pragma unroll
                    for (int w = 0; w < kWaves; ++w) Mr = fmaxf(Mr, red_m[w][t][r]);
                    const float Mru = (Mr == -INFINITY) ? 0.f : Mr;
                    float Lr = 0.f;
#pragma unroll
                    for (int w = 0; w < kWaves; ++w) Lr += red_l[w][t][r] * fast_exp2(red_m[w][t][r] - Mru);
                    a.part_lse[((size_t)it.part * a.n_seqs + seq) * a.n_q_heads + h] =
                        (Lr > 0.f) ? (Mru + log2f(Lr)) * kLn2 : -INFINITY;
                }
            }
        }
        __syncthreads();
    }
}

// One wave per output row (sequence, query head).
template <int HD>
__global__ __launch_bounds__(256) void merge_kernel(MergeArgs a)
{
    constexpr int PER = HD / 64;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int row = blockIdx.x * 4 + wave;
    if (row >= a.rows) return;

    int npre, nsuf, suf0;
    if (a.seq_prefix_parts) {
        const int seq = row / a.n_q_heads;
        npre = a.seq_prefix_parts[seq];
        const int Lraw = a.suffix_len[seq];
        const int L = min(max(Lraw, 0), a.max_suffix_len);
        if (L != Lraw && lane == 0 && row % a.n_q_heads == 0) atomicOr(a.err, kErrSuffixClamped);
        nsuf = (L + a.suffix_split - 1) / a.suffix_split;
        suf0 = a.max_prefix_parts;
    } else {
        npre = a.n_parts;
        nsuf = 0;
        suf0 = 0;
    }
    const int n = npre + nsuf;
    const size_t rows = (size_t)a.rows;

    float M = -INFINITY;
    for (int i = lane; i < n; i += 64) {
        const int p = i < npre ? i : suf0 + (i - npre);
        M = fmaxf(M, a.part_lse[(size_t)p * rows + row]);
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) M = fmaxf(M, __shfl_xor(M, off));

    float acc[PER];
#pragma unroll
    for (int k = 0; k < PER; ++k) acc[k] = 0.f;
    float wsum = 0.f;
    if (M != -INFINITY) {
        for (int base = 0; base < n; base += 64) {
            const int i = base + lane;
            int p = 0;
            float w = 0.f;
            if (i < n) {
                p = i < npre ? i : suf0 + (i - npre);
                const float l = a.part_lse[(size_t)p * rows + row];
                w = (l == -INFINITY) ? 0.f : exp2f((l - M) * kLog2e);
            }
            float ws = w;
#pragma unroll
            for (int off = 32; off >= 1; off >>= 1) ws += __shfl_xor(ws, off);
            wsum += ws;
            const int cnt = min(64, n - base);
            for (int j = 0; j < cnt; ++j) {
                const float wj = __shfl(w, j);
                const int pj = __shfl(p, j);
                if (wj != 0.f) {
                    const float *src = a.part_o + ((size_t)pj * rows + row) * HD + lane * PER;
#pragma unroll
                    for (int k = 0; k < PER; ++k) acc[k] += wj * src[k];
                }
            }
        }
    }
    float *dst = a.out + (size_t)row * HD + lane * PER;
#pragma unroll
    for (int k = 0; k < PER; ++k) dst[k] = (wsum > 0.f) ? acc[k] / wsum : 0.f;
    if (a.out_lse && lane == 0) a.out_lse[row] = (wsum > 0.f) ? M + logf(wsum) : -INFINITY;
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

// grid (ceil(out_len / 16), Hkv): block copies 16 logical positions of one KV head.
__global__ __launch_bounds__(256) void gather_kernel(GatherArgs a)
{
    const int g = blockIdx.y;
    const int cpr = a.head_dim / 8;
    for (int i = threadIdx.x; i < kPageSize * cpr; i += blockDim.x) {
        const int pos = blockIdx.x * kPageSize + i / cpr, c = i % cpr;
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
        const size_t dst = ((size_t)g * a.out_len + pos) * a.head_dim + 8 * c;
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

template <int HD>
hipError_t launch_partials_hd(const AttnArgs &a, int n_items, int row_tiles, hipStream_t s)
{
    const dim3 grid(n_items), block(kThreads);
    switch (row_tiles) {
    case 1: partials_kernel<HD, 1><<<grid, block, 0, s>>>(a); break;
    case 2: partials_kernel<HD, 2><<<grid, block, 0, s>>>(a); break;
    case 3: partials_kernel<HD, 3><<<grid, block, 0, s>>>(a); break;
    case 4: partials_kernel<HD, 4><<<grid, block, 0, s>>>(a); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_partials(const AttnArgs &a, int n_items, int head_dim, int row_tiles, hipStream_t s)
{
    if (n_items <= 0) return hipSuccess;
    if (head_dim == 128) return launch_partials_hd<128>(a, n_items, row_tiles, s);
    if (head_dim == 64) return launch_partials_hd<64>(a, n_items, row_tiles, s);
    return hipErrorInvalidValue;
}

hipError_t launch_merge(const MergeArgs &a, int head_dim, hipStream_t s)
{
    if (a.rows <= 0) return hipSuccess;
    const dim3 grid((a.rows + 3) / 4), block(256);
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
    if (a.out_len <= 0) return hipSuccess;
    gather_kernel<<<dim3((a.out_len + kPageSize - 1) / kPageSize, a.n_kv_heads), dim3(256), 0, s>>>(a);
    return hipGetLastError();
}

}  // namespace fka
