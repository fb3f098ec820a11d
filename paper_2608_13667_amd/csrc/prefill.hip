// Instruction prefill at the fork as a tiled multi-query attention kernel (gfx950, wave64).
//
// After a fork every branch b takes n instruction tokens at once (paper Sec. 3.3: the snapshot
// of the shared context followed by a short branch-specific instruction; Sec. 4.4: a branch's
// load is dominated by prefill over the cached prefix).  Token t of branch b is virtual sequence
// s = b n + t; its G query rows (one per query head of a KV head) attend to the whole shared
// prefix and to b's suffix positions [0, L_b + t] (causal within the instruction).  With N n G
// query rows per KV head sharing one prefix, this stage is a dense contraction: every prefix
// key is scored against hundreds of rows, so it runs on the matrix cores and is bound by their
// rate and by the vector work of the online softmax, not by HBM.
//
// Work: the rows of KV head g are cut into units of 32 consecutive rows (row i of the head is
// query head g G + i mod G of sequence i / G), one unit per wave.  A block of eight waves takes
// up to eight units of one KV head (the units spread evenly over the blocks of a range) over one
// range of prefix tiles (64 keys each); the prefix is split into R ranges so that the blocks fill
// the device, and the block of the last range also takes the suffix keys.  Each wave writes one normalised partial (o, lse) per row for its range, and
// the merge kernel combines a row's R partials (its explicit mode).
//   * K and V tiles go from HBM (or L2: the blocks of one KV head and range run on one XCD when
//     the KV heads are a multiple of 8 apart in the grid order) into LDS by DMA
//     (buffer_load_dwordx4 ... lds) into four tile buffers (two read while two load), each
//     tile loaded once by the block (every wave moves 8 of its 64 rows) and read by all eight
//     waves;
//   * the two waves of a SIMD alternate between matrix and vector work, in two phases per tile
//     with a block barrier between them: while one takes p.v of the previous tile and q.k of
//     this one (at raised priority), the other takes a softmax, and then the roles swap;
//   * S^T = K Q^T and O^T += V^T P^T run on v_mfma_f32_16x16x32_bf16 with keys on M, so each
//     lane owns two query rows of the online softmax (rows l16 and 16 + l16 of the unit) and
//     16 keys of each per tile; P enters the second product as two bf16 terms (hi + lo);
//   * K is read from LDS in the A-operand layout (16-byte chunks xor-swizzled by row, so a
//     16-lane read touches every bank once), V transposed with ds_read_b64_tr_b16;
//   * the running maximum moves only when a score exceeds it by more than 2^8;
//   * suffix keys (the instruction and any suffix before it) are read per wave after the prefix
//     range, 32 keys at a time, K straight into registers and V through a wave-private LDS
//     area, with each row masked to its own branch and causal limit.  A non-finite value there
//     is replaced by zero for the product and the rows that read its key are made NaN, so that
//     it reaches no row of another branch or of an earlier token.
#include <type_traits>
#include <utility>

#include "internal.h"

namespace fka {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(4))) const int32_t const_i32;

constexpr int HD = 128;            // head dimension of this kernel
constexpr int ROWB = HD * 2;       // bytes per key row
constexpr int NC = HD / 32;        // k-steps of the q.k product
constexpr int NE = HD / 16;        // 16-wide d tiles of the output
constexpr int KT = 64;             // keys per prefix tile
constexpr int NW = 8;              // waves per block (two per SIMD)
constexpr int STAGES = 4;          // prefix tile buffers: two read, two loading
constexpr int KBYTES = KT * ROWB;  // 16 KiB of K (or V) per tile
constexpr int K_LDS = 0;           // K buffers at [0, 64 KiB)
constexpr int V_LDS = STAGES * KBYTES;  // V buffers at [64, 128 KiB)
constexpr int LDS_BYTES = 2 * STAGES * KBYTES;
constexpr int ST = 32;             // keys per suffix tile
constexpr int SUF_LDS = ST * ROWB; // per-wave V area for a suffix tile (8 KiB), reusing the stages
constexpr float kLn2 = 0.693147180559945309f;
constexpr float kRescaleGap = 8.0f;  // log2 units

static_assert(NW * SUF_LDS <= LDS_BYTES, "suffix areas fit the stage buffers");
static_assert(STAGES == 4, "the tile loop is unrolled over its four buffers");
static_assert((STAGES - 1) * KBYTES + 3 * 16 * ROWB < 65536, "LDS offsets fit the immediate field");

__device__ inline f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ inline float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ inline int uni(int x) { return __builtin_amdgcn_readfirstlane(x); }

// Raw buffer resource over [base, base + bytes), built from wave-uniform values.
__device__ inline __amdgpu_buffer_rsrc_t make_rsrc(const char *base, int bytes)
{
    const uint64_t b = (uint64_t)base;
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)b);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(b >> 32));
    const int n = __builtin_amdgcn_readfirstlane(bytes);
    return __builtin_amdgcn_make_buffer_rsrc((void *)(((uint64_t)hi << 32) | lo), 0, n, 0x00020000);
}

// 16 bytes per lane into LDS at dst + 16 * lane (LDS DMA), default cache policy: the other
// blocks of the KV head read the same tile from L2.  Kept outside the kernel template (used
// there directly, the builtin stops the host compiler from emitting the launch stub).
template <int OFFSET>
__device__ inline void dma16(__amdgpu_buffer_rsrc_t r, lds_void *dst, uint32_t voff)
{
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, dst, 16, voff, 0, OFFSET, 0);
}

__device__ inline int32_t scalar_load(const int32_t *p) { return *(const_i32 *)p; }

template <int N>
__device__ inline void wait_vm()
{
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

template <typename F, int... I>
__device__ inline void static_for_impl(F &&f, std::integer_sequence<int, I...>)
{
    (f(std::integral_constant<int, I>{}), ...);
}
template <int N, typename F>
__device__ inline void static_for(F &&f)
{
    static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// max(a, b) in one instruction, for values that hold no signalling NaN (see max3 below).
__device__ inline float max2(float a, float b)
{
    float r;
    asm("v_max_f32 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
    return r;
}

// Reductions over lanes l, l ^ 16, l ^ 32, l ^ 48 (the four lanes holding one query row).  The
// maximum's inputs are maxima of matrix-core results (no signalling NaN).
__device__ inline float max_over_rows(float x)
{
    const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    x = max2(__uint_as_float(a[0]), __uint_as_float(a[1]));
    const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return max2(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

__device__ inline float sum_over_rows(float x)
{
    const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    x = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// LDS reads as inline assembly (the builtins make the compiler wait for every LDS DMA in
// flight, which would drain the tiles being prefetched); valid after lds_wait().
template <int OFFSET>
__device__ inline u32x4 ds_read_b128_at(uint32_t addr)
{
    static_assert(OFFSET >= 0 && OFFSET < 65536, "ds offset field");
    u32x4 r;
    asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "i"(OFFSET) : "memory");
    return r;
}

// ds_read_b64_tr_b16: within each group of 16 lanes, lane i receives element i % 4 of the rows
// addressed by lanes i / 4, 4 + i / 4, 8 + i / 4 and 12 + i / 4 (the transpose of a 16 x 4 block).
typedef long vtr_t;
template <int OFFSET>
__device__ inline vtr_t ds_read_tr16(uint32_t addr)
{
    static_assert(OFFSET >= 0 && OFFSET < 65536, "ds offset field");
    vtr_t r;
    asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "i"(OFFSET) : "memory");
    return r;
}

__device__ inline void lds_wait() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// Block barrier after this wave's LDS reads have returned (global loads stay in flight).
__device__ inline void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// Sixteen wait states between matrix-core ops and the first vector read of their results (the
// toolchain's own count for this op on gfx950 was seen to fall short in the decode kernel).
__device__ inline void xdl_result_wait()
{
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("s_nop 7\n\ts_nop 7" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
}

// max(a, b, c) in one instruction.  fmaxf on a matrix-core result makes the compiler quiet a
// possible signalling NaN first (one more instruction per value); the matrix cores produce
// only quiet NaNs, which v_max3_f32 ignores as fmaxf does.
__device__ inline float max3(float a, float b, float c)
{
    float r;
    asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
    return r;
}

// Maximum of n values as a tree of v_max3_f32.
template <int N>
__device__ inline float max_of(const float (&v)[N])
{
    static_assert(N >= 3, "at least three values");
    if constexpr (N == 3) {
        return max3(v[0], v[1], v[2]);
    } else {
        constexpr int M = (N + 2) / 3;
        float w[M];
#pragma unroll
        for (int i = 0; i < M; ++i) {
            const int k = 3 * i;
            w[i] = (k + 2 < N) ? max3(v[k], v[k + 1], v[k + 2]) : (k + 1 < N) ? max2(v[k], v[k + 1]) : v[k];
        }
        if constexpr (M < 3)
            return max2(w[0], w[M - 1]);
        else
            return max_of(w);
    }
}

__device__ inline int opaque_lane_id()
{
    int v;
    asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(v));
    return v;
}

__device__ inline bf16x8 join_tr16(vtr_t lo, vtr_t hi)
{
    const s16x4 a = __builtin_bit_cast(s16x4, lo), b = __builtin_bit_cast(s16x4, hi);
    const short __attribute__((ext_vector_type(8))) v = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
    return __builtin_bit_cast(bf16x8, v);
}

// Splits p into hi + lo, both bf16: hi keeps the top 16 bits of p, lo is the rest rounded.
// Packs the values of two key groups (four each) into the B operand of one p.v product.
__device__ inline void split_p(const float (&p)[8], bf16x8 &hi, bf16x8 &lo)
{
    uint32_t hw[4];
    float r[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) r[i] = p[i] - __uint_as_float(__float_as_uint(p[i]) & 0xffff0000u);
#pragma unroll
    for (int k = 0; k < 4; ++k) hw[k] = __builtin_amdgcn_perm(__float_as_uint(p[2 * k + 1]), __float_as_uint(p[2 * k]), 0x07060302u);
    hi = __builtin_bit_cast(bf16x8, hw);
#pragma unroll
    for (int i = 0; i < 8; ++i) lo[i] = (__bf16)r[i];
}

template <bool PAGED>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(2))) void prefill_tiles_kernel(PrefillArgs a)
{
    __shared__ __attribute__((aligned(1024))) char lds[LDS_BYTES];

    const int tid = threadIdx.x;
    const int lane = tid & 63, l16 = lane & 15, q4 = lane >> 4;
    const int wave = uni(tid >> 6);
    const int Hkv = a.n_kv_heads, G = a.group, Hq = a.n_q_heads;
    const int n = a.n_tokens, N = a.n_branches;
    const int S = N * n, rows_head = S * G;
    const int Lp = a.prefix_len;

    // block -> (KV head, unit group, range); the KV head varies fastest so that with Hkv a
    // multiple of 8 a head's blocks all land on one XCD (block b runs on XCD b mod 8)
    const int vb = blockIdx.x;
    const int g = vb % Hkv, rest = vb / Hkv;
    const int ug = rest % a.unit_groups, r = rest / a.unit_groups;
    // the units spread evenly over the groups (at most eight each): blocks of one range then
    // stream its tiles at the same pace, so each tile is fetched once into the XCD's L2 for all
    const int u = mul_div(ug, a.n_units, a.unit_groups) + wave;
    const bool active = u < mul_div(ug + 1, a.n_units, a.unit_groups);
    const int R = a.ranges;
    const int PT = a.prefix_tiles;
    const int total = PT + a.tail_reserve;
    const int t0 = min(PT, mul_div(r, total, R)), t1 = (r == R - 1) ? PT : min(PT, mul_div(r + 1, total, R));
    const int ntile = t1 - t0;

    // ---- per-lane constants
    // DMA: this wave moves tile rows [8 wave, 8 wave + 8): instruction ii writes rows
    // 8 wave + 4 ii + lane / 16, lane's LDS chunk position lane % 16, which holds the row's
    // global chunk position ^ swizzle(row) (K: row mod 16, V: 2 row mod 16)
    uint32_t koff[2], voff[2];
#pragma unroll
    for (int ii = 0; ii < 2; ++ii) {
        const int tl = 4 * ii + (lane >> 4), pos = lane & 15, T = 8 * wave + tl;
        koff[ii] = tl * ROWB + 16 * (pos ^ (T & 15));
        voff[ii] = tl * ROWB + 16 * (pos ^ ((2 * T) & 15));
    }
    const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char *)&lds[0];
    // K A-operand reads: row 16 i + l16 (i = M tile, an immediate 4096 i), chunk 4 c + q4
    uint32_t kaddr[NC];
#pragma unroll
    for (int c = 0; c < NC; ++c) kaddr[c] = lds0 + K_LDS + l16 * ROWB + 16 * ((4 * c + q4) ^ l16);
    // V^T reads (transposed): lane (q4, l16) addresses row 4 q4 + l16 / 4, d = 16 e + 4 (l16 % 4);
    // rows 16 m further are at + 4096 m with the same swizzle
    uint32_t vaddr[NE];
    {
        const int jt = l16 >> 2, m4 = l16 & 3, T = 4 * q4 + jt;
#pragma unroll
        for (int e = 0; e < NE; ++e) {
            const int slot = (2 * e + (m4 >> 1)) ^ ((2 * T) & 15);
            vaddr[e] = lds0 + V_LDS + T * ROWB + slot * 16 + (m4 & 1) * 8;
        }
    }

    // ---- query rows (B operand of S^T): lane holds unit row 16 t + l16, d = 32 c + 8 q4 .. +7
    bf16x8 qb[2][NC];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
        const int lr = u * 32 + 16 * t + l16;
#pragma unroll
        for (int c = 0; c < NC; ++c) qb[t][c] = bf16x8{};
        if (active && lr < rows_head) {
            const int s = lr / G, h = g * G + lr % G;
            const uint16_t *qp = a.q + ((size_t)s * Hq + h) * HD + 8 * q4;
#pragma unroll
            for (int c = 0; c < NC; ++c) qb[t][c] = *reinterpret_cast<const bf16x8 *>(qp + 32 * c);
        }
    }

    // ---- prefix tile loads: this wave's 8 rows of tile `tile` into stage `st`
    bool bad_page = false;
    const char *const pk = reinterpret_cast<const char *>(PAGED ? a.k_pool : a.prefix_k);
    const char *const pv = reinterpret_cast<const char *>(PAGED ? a.v_pool : a.prefix_v);
    auto issue_prefix = [&](int tile, int st) {
        const int row0 = tile * KT + 8 * wave;
        int rows_ok = max(0, min(8, Lp - row0));
        size_t off;
        if constexpr (PAGED) {
            // prefix pages: the same ids in every branch's row (branch 0's row is read)
            const int32_t page = scalar_load(a.page_table + uni(min(row0 / kPageSize, a.max_pages - 1)));
            const bool bad = rows_ok > 0 && (page < 0 || page >= a.n_pool_pages);
            bad_page |= bad;
            rows_ok = bad ? 0 : rows_ok;
            off = rows_ok > 0 ? (((size_t)page * Hkv + g) * kPageSize + (row0 % kPageSize)) * ROWB : 0;
        } else {
            off = rows_ok > 0 ? ((size_t)g * Lp + row0) * ROWB : 0;
        }
        const __amdgpu_buffer_rsrc_t rk = make_rsrc(pk + off, rows_ok * ROWB);
        const __amdgpu_buffer_rsrc_t rv = make_rsrc(pv + off, rows_ok * ROWB);
        char *kd = &lds[K_LDS + st * KBYTES + 8 * wave * ROWB];
        char *vd = &lds[V_LDS + st * KBYTES + 8 * wave * ROWB];
        dma16<0>(rk, (lds_void *)(__attribute__((address_space(3))) char *)kd, koff[0]);
        dma16<0>(rk, (lds_void *)(__attribute__((address_space(3))) char *)(kd + 4 * ROWB), koff[1]);
        dma16<0>(rv, (lds_void *)(__attribute__((address_space(3))) char *)vd, voff[0]);
        dma16<0>(rv, (lds_void *)(__attribute__((address_space(3))) char *)(vd + 4 * ROWB), voff[1]);
    };

    // ---- online softmax state: lane owns unit rows l16 (t = 0) and 16 + l16 (t = 1)
    f32x4 acc[2][NE];
    float m_ref[2], l_run[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
        m_ref[t] = -INFINITY;
        l_run[t] = 0.f;
#pragma unroll
        for (int e = 0; e < NE; ++e) acc[t][e] = f32x4{0.f, 0.f, 0.f, 0.f};
    }

    // Softmax of NM M tiles of scores (x[t][i][j]: row 16 t + l16, key 16 i + 4 q4 + j of the
    // tile, raw q.k or -inf) into the two bf16 terms of P per k-step of 32 keys.
    // Row tile t's maximum over NM M tiles of scores (xt[i][j]: key 16 i + 4 q4 + j of the tile,
    // raw q.k or -inf), moving the running maximum (and rescaling) when it grows by over 2^8.
    auto row_max = [&](auto NMc, int t, const float (&xt)[decltype(NMc)::value][4]) {
        constexpr int NM = decltype(NMc)::value;
        float v[4 * NM];
#pragma unroll
        for (int i = 0; i < NM; ++i)
#pragma unroll
            for (int j = 0; j < 4; ++j) v[4 * i + j] = xt[i][j];
        const float mx = max_over_rows(max_of(v)) * a.scale_log2;  // the scale is positive: the order is kept
        const bool move = mx > m_ref[t] + kRescaleGap;
        if (__builtin_expect(__builtin_amdgcn_ballot_w64(move) != 0, 0)) {
            const float m_new = move ? mx : m_ref[t];
            // exactly 1 for a row that keeps its max; 0 when the row's max was -inf
            const float alpha = move ? fast_exp2(m_ref[t] - m_new) : 1.f;
            l_run[t] *= alpha;
            xdl_result_wait();
#pragma unroll
            for (int e = 0; e < NE; ++e) acc[t][e] *= alpha;
            m_ref[t] = m_new;
        }
    };
    // Row tile t's p = 2^(scale q.k - max) into the two bf16 terms per k-step of 32 keys.
    auto row_exp = [&](auto NMc, int t, const float (&xt)[decltype(NMc)::value][4],
                       bf16x8 (&pht)[decltype(NMc)::value / 2], bf16x8 (&plt)[decltype(NMc)::value / 2]) {
        constexpr int NM = decltype(NMc)::value;
        const float nm = (m_ref[t] == -INFINITY) ? 0.f : -m_ref[t];
        float ps = 0.f;
#pragma unroll
        for (int kk = 0; kk < NM / 2; ++kk) {
            float p[8];
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                p[j] = fast_exp2(__builtin_fmaf(xt[2 * kk][j], a.scale_log2, nm));
                p[4 + j] = fast_exp2(__builtin_fmaf(xt[2 * kk + 1][j], a.scale_log2, nm));
            }
#pragma unroll
            for (int j = 0; j < 8; ++j) ps += p[j];
            split_p(p, pht[kk], plt[kk]);
        }
        l_run[t] += ps;
    };
    auto softmax = [&](auto NMc, auto &x, auto &ph, auto &pl) {
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            row_max(NMc, t, x[t]);
            row_exp(NMc, t, x[t], ph[t], pl[t]);
        }
    };

    // p.v of one k-step (32 keys: tile keys 32 kk + 4 q4 + j and 32 kk + 16 + 4 q4 + j)
    auto pv_step = [&](const vtr_t (&vr)[NE][2], const bf16x8 (&ph)[2], const bf16x8 (&pl)[2]) {
#pragma unroll
        for (int e = 0; e < NE; ++e) {
            const bf16x8 va = join_tr16(vr[e][0], vr[e][1]);
#pragma unroll
            for (int t = 0; t < 2; ++t) {
                acc[t][e] = mfma16(va, ph[t], acc[t][e]);
                acc[t][e] = mfma16(va, pl[t], acc[t][e]);
            }
        }
    };

    // ---- the prefix range: tiles [t0, t1), two loading ahead, in two phases per tile.  The two
    // waves of a SIMD alternate between matrix and vector work: in phase 1 of step i the first
    // wave (waves 0..3) takes p.v of tile i - 1 and q.k of tile i while the second (waves 4..7)
    // takes the softmax of tile i - 1; in phase 2 the first takes the softmax of tile i while the
    // second takes p.v of tile i - 1 and q.k of tile i (p.v first, so that p and the new scores
    // are not live together).  A block barrier separates the phases; the
    // wave in its matrix phase runs at raised priority.  Four tile buffers: tiles i - 1 and i are
    // read during step i while i + 1 and i + 2 load.
    using nm4_t = std::integral_constant<int, 4>;
    // q.k of the tile at buffer offset SO: each M tile's K operands are read one M tile ahead of
    // its MFMAs (LDS reads return in order, so "at most 4 outstanding" means the earlier M tile's
    // four reads are in)
    auto qk = [&](auto SOc, f32x4 (&sc)[4][2]) {
        constexpr int SO = decltype(SOc)::value;
        bf16x8 ka[2][NC];
        auto rd = [&](auto MIc) {
            constexpr int mi = decltype(MIc)::value;
#pragma unroll
            for (int c = 0; c < NC; ++c)
                ka[mi & 1][c] = __builtin_bit_cast(bf16x8, ds_read_b128_at<SO + mi * 16 * ROWB>(kaddr[c]));
        };
        rd(std::integral_constant<int, 0>{});
        static_for<4>([&](auto MIc) {
            constexpr int mi = decltype(MIc)::value;
            if constexpr (mi + 1 < 4) {
                rd(std::integral_constant<int, mi + 1>{});
                asm volatile("s_waitcnt lgkmcnt(4)" ::: "memory");
            } else {
                lds_wait();
            }
#pragma unroll
            for (int c = 0; c < NC; ++c) asm volatile("" : "+v"(ka[mi & 1][c]));
#pragma unroll
            for (int t = 0; t < 2; ++t) {
                f32x4 v = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int c = 0; c < NC; ++c) v = mfma16(ka[mi & 1][c], qb[t][c], v);
                sc[mi][t] = v;
            }
        });
    };
    // (every tile here is whole: no key mask, which would make the compiler copy the scores
    // into the masked path's registers, 32 moves per tile)
    auto sm = [&](const f32x4 (&sc)[4][2], bf16x8 (&ph)[2][2], bf16x8 (&pl)[2][2]) {
        xdl_result_wait();
        float x[2][4][4];
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
            for (int mi = 0; mi < 4; ++mi)
#pragma unroll
                for (int j = 0; j < 4; ++j) x[t][mi][j] = sc[mi][t][j];
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            row_max(nm4_t{}, t, x[t]);
            row_exp(nm4_t{}, t, x[t], ph[t], pl[t]);
        }
    };
    auto pv_tile = [&](auto SOc, const bf16x8 (&ph)[2][2], const bf16x8 (&pl)[2][2]) {
        constexpr int SO = decltype(SOc)::value;
        static_for<2>([&](auto KKc) {
            constexpr int kk = decltype(KKc)::value;
            vtr_t vr[NE][2];
#pragma unroll
            for (int e = 0; e < NE; ++e) {
                vr[e][0] = ds_read_tr16<SO + (2 * kk) * 16 * ROWB>(vaddr[e]);
                vr[e][1] = ds_read_tr16<SO + (2 * kk + 1) * 16 * ROWB>(vaddr[e]);
            }
            lds_wait();
#pragma unroll
            for (int e = 0; e < NE; ++e) asm volatile("" : "+v"(vr[e][0]), "+v"(vr[e][1]));
            const bf16x8 h2[2] = {ph[0][kk], ph[1][kk]}, l2[2] = {pl[0][kk], pl[1][kk]};
            pv_step(vr, h2, l2);
        });
    };
    f32x4 sc[4][2];
    bf16x8 ph[2][2], pl[2][2];
    // step i (0 <= i <= ntile; the last one only finishes tile ntile - 1), tile i in buffer B.  The
    // two roles run in loops of their own (a role test in each phase would keep both roles'
    // values live at once); both pass the same barriers.
    auto step = [&](int i, auto Bc, auto LEADc) {
        constexpr int B = decltype(Bc)::value;
        constexpr bool LEAD = decltype(LEADc)::value;
        constexpr int SO = B * KBYTES, SOP = ((B + STAGES - 1) % STAGES) * KBYTES;
        using so_t = std::integral_constant<int, SO>;
        using sop_t = std::integral_constant<int, SOP>;
        if (i < ntile) {
            if (i + 1 < ntile)
                wait_vm<4>();
            else
                wait_vm<0>();
        }
        lds_barrier();  // tile i is in LDS; every wave is done with tile i - 2
        if (i + 2 < ntile) issue_prefix(t0 + i + 2, (i + 2) % STAGES);
        if (active) {
            if constexpr (LEAD) {
                __builtin_amdgcn_s_setprio(1);
                if (i > 0) pv_tile(sop_t{}, ph, pl);
                if (i < ntile) qk(so_t{}, sc);
                __builtin_amdgcn_s_setprio(0);
            } else {
                if (i > 0) sm(sc, ph, pl);
            }
        }
        lds_barrier();
        if (active) {
            if constexpr (LEAD) {
                if (i < ntile) sm(sc, ph, pl);
            } else {
                __builtin_amdgcn_s_setprio(1);
                if (i > 0) pv_tile(sop_t{}, ph, pl);
                if (i < ntile) qk(so_t{}, sc);
                __builtin_amdgcn_s_setprio(0);
            }
        }
    };
    auto run = [&](auto LEADc) {
        for (int i = 0; i <= ntile; i += STAGES) {
            step(i, std::integral_constant<int, 0>{}, LEADc);
            if (i + 1 <= ntile) step(i + 1, std::integral_constant<int, 1>{}, LEADc);
            if (i + 2 <= ntile) step(i + 2, std::integral_constant<int, 2>{}, LEADc);
            if (i + 3 <= ntile) step(i + 3, std::integral_constant<int, 3>{}, LEADc);
        }
    };
    if (ntile > 0) issue_prefix(t0, 0);
    if (ntile > 1) issue_prefix(t0 + 1, 1);
    if (ntile > 0) {
        if (wave < 4)
            run(std::true_type{});
        else
            run(std::false_type{});
    }

    // ---- keys outside the whole prefix tiles (last range only), per wave: the prefix's last
    // Lp mod 64 keys (every row reads them), then the suffix keys branch by branch of the unit's
    // rows (the waves of a block hold different branches)
    if (r == R - 1) {
        lds_barrier();  // every wave is done with the stage buffers (no DMA in flight: all waited)
        if (active) {
            const int lr0 = u * 32, lr1 = min(rows_head, lr0 + 32);
            const int s_lo = lr0 / G, s_hi = (lr1 - 1) / G;
            const int b_lo = s_lo / n, b_hi = s_hi / n;
            // this lane's rows: sequence (or -1 past the head's rows)
            int srow[2];
#pragma unroll
            for (int t = 0; t < 2; ++t) {
                const int lr = lr0 + 16 * t + l16;
                srow[t] = lr < rows_head ? lr / G : -1;
            }
            const int max_L = a.max_suffix_len - n;  // clamp bound of suffix_len[b]
            const uint32_t vw = lds0 + wave * SUF_LDS;  // this wave's V area
            char *vwp = &lds[wave * SUF_LDS];
            // V DMA offsets for a 32-row suffix tile: instruction ii writes rows 4 ii + lane / 16
            // (the parity of ii decides the swizzle); rows 16 m further are one page further
            uint32_t svoff[2];
#pragma unroll
            for (int par = 0; par < 2; ++par) {
                const int T = 4 * par + (lane >> 4), pos = lane & 15;
                svoff[par] = (lane >> 4) * ROWB + 16 * (pos ^ ((2 * T) & 15));
            }
            const char *const sk = reinterpret_cast<const char *>(PAGED ? a.k_pool : a.suffix_k);
            const char *const sv = reinterpret_cast<const char *>(PAGED ? a.v_pool : a.suffix_v);
            const int pre_pages = (Lp + kPageSize - 1) / kPageSize;
            // One 32-key tile [p0, p0 + 32) of a key run whose 16-row groups `grp` addresses (K from
            // srck, V from srcv), row t of this lane masked to the run's keys <= lim[t] (-1: none).
            // CHECK: a non-finite value is zeroed for the product and the first key holding one
            // is kept in kbad.
            auto key_tile = [&](auto CHECKc, auto &grp, const char *srck, const char *srcv, int p0, const int (&lim)[2],
                                int &kbad) {
                constexpr bool CHECK = decltype(CHECKc)::value;
                // K rows straight into registers (A operand): M tile mi = rows 16 mi + l16
                bf16x8 ka[2][NC];
#pragma unroll
                for (int mi = 0; mi < 2; ++mi) {
                    const __amdgpu_buffer_rsrc_t rk = grp(srck, p0 + 16 * mi);
#pragma unroll
                    for (int c = 0; c < NC; ++c)
                        ka[mi][c] = __builtin_bit_cast(
                            bf16x8, __builtin_amdgcn_raw_buffer_load_b128(rk, l16 * ROWB + 16 * (4 * c + q4), 0, 0));
                }
                // V rows into this wave's LDS area
                {
                    const __amdgpu_buffer_rsrc_t r0 = grp(srcv, p0), r1 = grp(srcv, p0 + 16);
                    static_for<8>([&](auto I) {
                        constexpr int ii = decltype(I)::value;
                        constexpr int imm = 1024 * (ii % 4);
                        dma16<imm>(ii < 4 ? r0 : r1,
                                   (lds_void *)((__attribute__((address_space(3))) char *)vwp + 1024 * ii - imm),
                                   svoff[ii & 1]);
                    });
                }
                wait_vm<0>();
                f32x4 sc[2][2];
#pragma unroll
                for (int mi = 0; mi < 2; ++mi)
#pragma unroll
                    for (int t = 0; t < 2; ++t) {
                        f32x4 s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                        for (int c = 0; c < NC; ++c) s = mfma16(ka[mi][c], qb[t][c], s);
                        sc[mi][t] = s;
                    }
                xdl_result_wait();
                float x[2][2][4];
                {
                    const int kq = p0 + 4 * (opaque_lane_id() >> 4);  // key of j = 0 in M tile 0
#pragma unroll
                    for (int t = 0; t < 2; ++t)
#pragma unroll
                        for (int mi = 0; mi < 2; ++mi)
#pragma unroll
                            for (int j = 0; j < 4; ++j)
                                x[t][mi][j] = (kq + 16 * mi + j <= lim[t]) ? sc[mi][t][j] : -INFINITY;
                }
                bf16x8 ph[2][1], pl[2][1];
                softmax(std::integral_constant<int, 2>{}, x, ph, pl);
                vtr_t vr[NE][2];
#pragma unroll
                for (int e = 0; e < NE; ++e) {
                    const uint32_t ad = vaddr[e] - (lds0 + V_LDS) + vw;
                    vr[e][0] = ds_read_tr16<0>(ad);
                    vr[e][1] = ds_read_tr16<16 * ROWB>(ad);
                }
                lds_wait();
#pragma unroll
                for (int e = 0; e < NE; ++e) asm volatile("" : "+v"(vr[e][0]), "+v"(vr[e][1]));
                if constexpr (CHECK) {
                    // non-finite values: zero for the product, remember the first such key
                    uint32_t bits = 0;
#pragma unroll
                    for (int e = 0; e < NE; ++e)
#pragma unroll
                        for (int h = 0; h < 2; ++h) {
                            const uint64_t w = (uint64_t)vr[e][h];
                            bits |= (((uint32_t)w & 0x7f807f80u) + 0x00800080u) |
                                    ((((uint32_t)(w >> 32)) & 0x7f807f80u) + 0x00800080u);
                        }
                    if (__builtin_expect(__builtin_amdgcn_ballot_w64((bits & 0x80008000u) != 0) != 0, 0)) {
                        // lane (q4, l16) holds keys p0 + 16 h + 4 q4 + k (k = 0..3) of column 16 e + l16
                        int first = 0x7fffffff;
                        const int kq = p0 + 4 * (opaque_lane_id() >> 4);
#pragma unroll
                        for (int e = 0; e < NE; ++e)
#pragma unroll
                            for (int h = 0; h < 2; ++h) {
                                uint64_t w = (uint64_t)vr[e][h];
#pragma unroll
                                for (int k = 0; k < 4; ++k) {
                                    const uint32_t v16 = (uint32_t)(w >> (16 * k)) & 0xffffu;
                                    if ((v16 & 0x7f80u) == 0x7f80u) {
                                        first = min(first, kq + 16 * h + k);
                                        w &= ~((uint64_t)0xffffu << (16 * k));
                                    }
                                }
                                vr[e][h] = (vtr_t)w;
                            }
#pragma unroll
                        for (int off = 1; off < 64; off <<= 1) first = min(first, __shfl_xor(first, off));
                        kbad = min(kbad, first);
                    }
                }
                const bf16x8 h2[2] = {ph[0][0], ph[1][0]}, l2[2] = {pl[0][0], pl[1][0]};
                pv_step(vr, h2, l2);
                // the next tile's V overwrites this area: the transposed reads are done
                // (waited above) before its DMA is issued
            };
            // the prefix keys past its whole tiles: rows of KV head g, or the prefix pages (the
            // same ids in every branch's row: branch 0's row is read)
            const int tail0 = PT * KT, tl = Lp - tail0;
            if (tl > 0) {
                auto grp_pre = [&](const char *src, int p) -> __amdgpu_buffer_rsrc_t {
                    int rows_ok = max(0, min(kPageSize, tl - p));
                    size_t off;
                    if constexpr (PAGED) {
                        const int32_t page = scalar_load(a.page_table + uni(min((tail0 + p) / kPageSize, a.max_pages - 1)));
                        const bool bad = rows_ok > 0 && (page < 0 || page >= a.n_pool_pages);
                        bad_page |= bad;
                        rows_ok = bad ? 0 : rows_ok;
                        off = rows_ok > 0 ? ((size_t)page * Hkv + g) * kPageSize * ROWB : 0;
                    } else {
                        off = rows_ok > 0 ? ((size_t)g * Lp + tail0 + p) * ROWB : 0;
                    }
                    return make_rsrc(src + off, rows_ok * ROWB);
                };
                int lim[2];
#pragma unroll
                for (int t = 0; t < 2; ++t) lim[t] = srow[t] >= 0 ? tl - 1 : -1;
                int unused = 0x7fffffff;
                for (int p0 = 0; p0 < tl; p0 += ST) key_tile(std::false_type{}, grp_pre, pk, pv, p0, lim, unused);
            }
            for (int b = b_lo; b <= b_hi; ++b) {
                const int lraw = scalar_load(a.suffix_len + b);
                const int L = min(max(lraw, 0), max_L);
                if (L != lraw && lane == 0) atomicOr(a.err, kErrSuffixClamped);
                const int tmax = min(n - 1, s_hi - b * n);
                const int klim = L + tmax + 1;  // keys of b's suffix this unit reads
                // the last key each of this lane's rows reads, or -1 for a row of another branch
                int lim[2];
#pragma unroll
                for (int t = 0; t < 2; ++t) lim[t] = (srow[t] >= 0 && srow[t] / n == b) ? L + srow[t] % n : -1;
                int kbad = 0x7fffffff;  // first key of b holding a non-finite value
                // 16-row group resource of b's suffix positions [p, p + 16)
                auto grp = [&](const char *src, int p) -> __amdgpu_buffer_rsrc_t {
                    int rows_ok = max(0, min(kPageSize, klim - p));
                    size_t off;
                    if constexpr (PAGED) {
                        const int32_t page = scalar_load(
                            a.page_table + (size_t)b * a.max_pages + uni(min(pre_pages + p / kPageSize, a.max_pages - 1)));
                        const bool bad = rows_ok > 0 && (page < 0 || page >= a.n_pool_pages);
                        bad_page |= bad;
                        rows_ok = bad ? 0 : rows_ok;
                        off = rows_ok > 0 ? ((size_t)page * Hkv + g) * kPageSize * ROWB : 0;
                    } else {
                        off = rows_ok > 0 ? (((size_t)b * Hkv + g) * a.suffix_cap + p) * ROWB : 0;
                    }
                    return make_rsrc(src + off, rows_ok * ROWB);
                };
                for (int p0 = 0; p0 < klim; p0 += ST) key_tile(std::true_type{}, grp, sk, sv, p0, lim, kbad);
#pragma unroll
                for (int t = 0; t < 2; ++t) l_run[t] = (lim[t] >= kbad) ? __builtin_nanf("") : l_run[t];
            }
        }
    }
    if (PAGED && __builtin_amdgcn_ballot_w64(bad_page) != 0 && lane == 0) atomicOr(a.err, kErrBadPage);

    // ---- one normalised partial per row of the unit for range r
    if (!active) return;
    const int lane_c = opaque_lane_id();
    const int l16c = lane_c & 15, q4c = lane_c >> 4;
    const size_t rows_total = (size_t)S * Hq;
    xdl_result_wait();
#pragma unroll
    for (int t = 0; t < 2; ++t) {
        const float l = sum_over_rows(l_run[t]);
        const int lr = u * 32 + 16 * t + l16c;
        if (lr >= rows_head) continue;
        const int s = lr / G, h = g * G + lr % G;
        const size_t orow = (size_t)r * rows_total + (size_t)s * Hq + h;
        // a row with no keys in this range: o = 0, lse = -inf (weight 0 in the merge)
        const bool empty = !(l > 0.f) && !(l != l);
        const float inv = empty ? 0.f : 1.f / l;
        float *dst = a.part_o + orow * HD + 4 * q4c;
#pragma unroll
        for (int e = 0; e < NE; ++e) *reinterpret_cast<f32x4 *>(dst + 16 * e) = acc[t][e] * inv;
        if (q4c == 0) a.part_lse[orow] = empty ? -INFINITY : (m_ref[t] + __log2f(l)) * kLn2;
    }
}

}  // namespace

int prefill_tiles_unit_rows() { return 32; }
int prefill_tiles_waves() { return NW; }

int prefill_tiles_blocks_per_cu(bool paged)
{
    int n = 0;
    const void *f = paged ? reinterpret_cast<const void *>(&prefill_tiles_kernel<true>)
                          : reinterpret_cast<const void *>(&prefill_tiles_kernel<false>);
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, f, 64 * NW, 0) != hipSuccess) return 0;
    return n;
}

hipError_t launch_prefill_tiles(const PrefillArgs &a, int n_blocks, hipStream_t s)
{
    if (n_blocks <= 0) return hipSuccess;
    if (a.paged)
        prefill_tiles_kernel<true><<<n_blocks, 64 * NW, 0, s>>>(a);
    else
        prefill_tiles_kernel<false><<<n_blocks, 64 * NW, 0, s>>>(a);
    return hipGetLastError();
}

}  // namespace fka
