// Partial attention over key ranges: the streaming stage of fork-aware decode
// attention on gfx950 (CDNA4, wave64).
//
// Work items (see WorkItem) are pulled from a device queue by persistent blocks of
// four waves.  An item covers one KV head and one key range and holds every query
// row that reads those keys: for a shared-prefix item, all sequences of the fork x
// the G query heads of the KV head, so each prefix K/V byte is fetched from HBM
// once for all branches (paper, Sec. 3.3: the prefix cache is reused by all
// decoding streams).  The block's four waves split the item into 32-token slices
// and stream them independently:
//   * K rows are loaded straight into registers in the MFMA A-operand layout
//     (16 tokens x 4 lanes x 16 bytes per instruction) one slice ahead;
//   * V rows are copied by LDS DMA (buffer_load_dwordx4 ... lds) into a wave-private
//     ring of four slices, three slices ahead, and read back transposed with
//     ds_read_b64_tr_b16;
//   * loads go through buffer resources sized to the rows that exist, so rows past the
//     end of a key range read as zeros without any per-lane test;
//   * S^T = K Q^T and O^T += V^T P^T run on v_mfma_f32_16x16x32_bf16 with tokens
//     on M, so each lane owns one query row of the online softmax; P enters the
//     second product as two bf16 terms (hi + lo), which keeps it accurate to ~2^-16;
//   * the running maximum is only moved when a score exceeds it by more than 2^8,
//     so the accumulator is rarely rescaled.
// The waves' (max, sum, accumulator) are combined through LDS at the end of the
// item and one normalised partial (o, lse) per row is written.
#include <type_traits>
#include <utility>

#include "internal.h"

namespace fka {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
typedef __attribute__((address_space(4))) const int32_t const_i32;

constexpr int kThreads = 256;
constexpr int kWaves = 4;
constexpr int kSlice = 32;      // tokens per wave step
#ifndef FKA_PIPELINE_DEPTH
#define FKA_PIPELINE_DEPTH 1
#endif
constexpr int kDepth = FKA_PIPELINE_DEPTH;  // K and V slices in flight ahead of the one being scored
constexpr int kStages = kDepth + 1;         // V ring stages and K register sets per wave
constexpr float kLn2 = 0.693147180559945309f;
constexpr float kRescaleGap = 8.0f;  // log2 units: accumulate with p <= 2^8 before moving the max

__device__ inline f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ inline float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Raw buffer resource over [base, base + bytes); every input is made wave-uniform so the
// descriptor lives in scalar registers (a per-lane descriptor would force a waterfall loop).
__device__ inline __amdgpu_buffer_rsrc_t make_rsrc(const char *base, int bytes)
{
    const uint64_t b = (uint64_t)base;
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)b);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(b >> 32));
    const int n = __builtin_amdgcn_readfirstlane(bytes);
    // word 3 0x00020000: raw 32-bit access (gfx9 family)
    return __builtin_amdgcn_make_buffer_rsrc((void *)(((uint64_t)hi << 32) | lo), 0, n, 0x00020000);
}

// 16 bytes per lane from a buffer into LDS at dst + 16 * lane (LDS DMA).  Kept outside
// the kernel template: used directly there, the builtin stops the host compiler from
// emitting the kernel's launch stub.
__device__ inline void buffer_to_lds16(__amdgpu_buffer_rsrc_t r, lds_void *dst, uint32_t voff)
{
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, dst, 16, voff, 0, 0, 0);
}

// Uniform (scalar-unit) load of a value that no kernel in flight writes.
__device__ inline int32_t scalar_load(const int32_t *p)
{
    return *(const_i32 *)p;
}

// s_waitcnt with vmcnt = n and the other counters left alone (gfx9 encoding).
template <int N>
__device__ inline void wait_vm()
{
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Calls f(std::integral_constant<int, i>{}) for i = 0 .. N-1 (compile-time unrolled).
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

// Reductions over the four lanes l, l ^ 16, l ^ 32, l ^ 48 (the four 16-lane rows of
// the wave) with v_permlane32_swap / v_permlane16_swap: VALU only, no LDS traffic.
__device__ inline float max_over_rows(float x)
{
    const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    x = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
    const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}

__device__ inline float sum_over_rows(float x)
{
    const auto a = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    x = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    const auto b = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// ds_read_b64_tr_b16: within each group of 16 lanes the 16 addressed 4-element rows
// are read as a 16 x 4 matrix M, and lane i receives M[i/4][i%4], M[4 + i/4][i%4],
// M[8 + i/4][i%4], M[12 + i/4][i%4].  Issued as inline assembly: the builtin makes the
// compiler wait for every LDS DMA in flight, which would drain the prefetch ring.
// The result is only valid after lds_wait_all().
typedef long vtr_t;
template <int OFFSET>
__device__ inline vtr_t ds_read_tr16(uint32_t lds_addr)
{
    static_assert(OFFSET >= 0 && OFFSET < 65536, "ds offset field");
    vtr_t r;
    asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(r) : "v"(lds_addr), "i"(OFFSET) : "memory");
    return r;
}

// Wait for the outstanding LDS reads; routing the values through the asm keeps their
// uses after the wait.
template <int NE>
__device__ inline void lds_wait_all(vtr_t (&v)[NE][2])
{
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
    for (int e = 0; e < NE; ++e) asm volatile("" : "+v"(v[e][0]), "+v"(v[e][1]));
}

__device__ inline bf16x8 join_tr16(vtr_t lo, vtr_t hi)
{
    const s16x4 a = __builtin_bit_cast(s16x4, lo), b = __builtin_bit_cast(s16x4, hi);
    const short __attribute__((ext_vector_type(8))) v = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
    return __builtin_bit_cast(bf16x8, v);
}

template <int HD, int NT, bool PAGED>
__global__ __launch_bounds__(kThreads) void partials_kernel(AttnArgs a)
{
    constexpr int CPR = HD / 8;                 // 16-byte chunks per K/V row
    constexpr int NC = HD / 32;                 // MFMA k-steps of q.k
    constexpr int NE = HD / 16;                 // MFMA d-tiles of p.v
    constexpr int SLICE_CHUNKS = kSlice * CPR;  // 16-byte chunks of one V slice
    constexpr int VDMA = SLICE_CHUNKS / 64;     // LDS DMA instructions per V slice
    constexpr int KLOADS = 2 * NC;              // K loads per lane per slice
    static_assert(VDMA == KLOADS, "one wait count per slice");
    constexpr int OSTRIDE = HD + 4;             // padded row stride of the output staging (floats)
    static_assert(kWaves * 16 * OSTRIDE * 4 <= kWaves * kStages * SLICE_CHUNKS * 16, "staging fits");

    // per wave: kStages V slices; chunk c of slice token T sits at T*CPR + (c ^ swz(T))
    __shared__ uint4 vring[kWaves][kStages][SLICE_CHUNKS];
    __shared__ float red_m[kWaves][NT][16];
    __shared__ float red_l[kWaves][NT][16];
    __shared__ int s_item;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform per wave
    const int l16 = lane & 15, q4 = lane >> 4;
    const int G = a.group;

    for (;;) {
        if (tid == 0) s_item = atomicAdd(a.queue, 1);
        __syncthreads();
        const int item = __builtin_amdgcn_readfirstlane(s_item);
        __syncthreads();  // s_item is rewritten at the next fetch
        if (item >= a.n_items) break;

        WorkItem it;  // scalar loads: every field is uniform across the block
        {
            const int32_t *ip = reinterpret_cast<const int32_t *>(a.items + item);
            it.kind = scalar_load(ip + 0);
            it.seq0 = scalar_load(ip + 1);
            it.nseq = scalar_load(ip + 2);
            it.kv_head = scalar_load(ip + 3);
            it.tok_begin = scalar_load(ip + 4);
            it.tok_end = scalar_load(ip + 5);
            it.part = scalar_load(ip + 6);
            it.prefix_len = scalar_load(ip + 7);
        }
        const int kvh = it.kv_head;
        const int rows = it.nseq * G;
        const int nt_act = (rows + 15) >> 4;

        // key source of the item
        const char *kbase, *vbase;
        const int32_t *ptab = nullptr;
        int page_off = 0;
        int tok_end = it.tok_end;
        if (it.kind == kSuffix) {
            tok_end = min(tok_end, min(max(scalar_load(a.suffix_len + it.seq0), 0), a.max_suffix_len));
            if (PAGED) {
                kbase = reinterpret_cast<const char *>(a.k_pool);
                vbase = reinterpret_cast<const char *>(a.v_pool);
                ptab = a.page_table + (size_t)it.seq0 * a.max_pages;
                page_off = (it.prefix_len + kPageSize - 1) / kPageSize;
            } else {
                const size_t base = ((size_t)it.seq0 * a.n_kv_heads + kvh) * (size_t)a.suffix_cap * HD * 2;
                kbase = reinterpret_cast<const char *>(a.suffix_k) + base;
                vbase = reinterpret_cast<const char *>(a.suffix_v) + base;
            }
        } else {
            if (PAGED) {
                kbase = reinterpret_cast<const char *>(a.k_pool);
                vbase = reinterpret_cast<const char *>(a.v_pool);
                ptab = a.page_table + (size_t)it.seq0 * a.max_pages;
            } else {
                const size_t base = (size_t)kvh * (size_t)a.prefix_len * HD * 2;
                kbase = reinterpret_cast<const char *>(a.prefix_k) + base;
                vbase = reinterpret_cast<const char *>(a.prefix_v) + base;
            }
        }
        const int n_tok = tok_end - it.tok_begin;
        if (n_tok <= 0) continue;  // a suffix part past the branch's length: the merge does not read it

        // this wave's slices: w, w + 4, w + 8, ... of the item
        const int n_slices = (n_tok + kSlice - 1) / kSlice;
        const int ns = n_slices > wave ? (n_slices - wave + kWaves - 1) / kWaves : 0;
        auto slice_tok0 = [&](int k) { return it.tok_begin + (wave + kWaves * k) * kSlice; };
        constexpr int ROWB = HD * 2;  // bytes per K/V row

        // Buffer resource over the 16-row group holding item positions [t, t + 16) (t is a
        // multiple of 16, so a group never straddles a page).  Its size covers only the rows
        // below tok_end, so loads of rows past the end (or of a group wholly past it, or behind
        // an out-of-range page id) return zeros.  Uniform.
        bool bad_page = false;
        auto group_rsrc = [&](const char *src, int t) -> __amdgpu_buffer_rsrc_t {
            const int rows_ok = max(0, min(kPageSize, tok_end - t));
            const char *base = src;
            if (!PAGED) {
                base = src + (size_t)t * ROWB;
            } else if (rows_ok > 0) {
                const int32_t page = scalar_load(ptab + min(page_off + t / kPageSize, a.max_pages - 1));
                if (page < 0 || page >= a.n_pool_pages) {
                    bad_page = true;
                    return make_rsrc(src, 0);
                }
                base = src + ((size_t)page * a.n_kv_heads + kvh) * (kPageSize * ROWB);
            }
            return make_rsrc(base, rows_ok * ROWB);
        };

        // query rows (B operand of S^T = K Q^T): lane holds row 16t + l16, d = 32c + 8*q4 .. +7
        bf16x8 qb[NT][NC];
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const int r = 16 * t + l16;
#pragma unroll
            for (int c = 0; c < NC; ++c) qb[t][c] = bf16x8{};
            if (r < rows) {
                const int seq = it.seq0 + r / G, h = kvh * G + r % G;
                const uint16_t *qp = a.q + ((size_t)seq * a.n_q_heads + h) * HD + 8 * q4;
#pragma unroll
                for (int c = 0; c < NC; ++c) qb[t][c] = *reinterpret_cast<const bf16x8 *>(qp + 32 * c);
            }
        }

        // K slice k into registers (the A operand of S^T): lane holds slice token 16u + l16,
        // bytes 16*q4 + 64c of its row, i.e. d = 32c + 8*q4 .. +7, the k-slots of q above.
        const uint32_t koff = l16 * ROWB + 16 * q4;
        auto load_k = [&](int k, bf16x8 (&kr)[2][NC]) {
            const int t0 = slice_tok0(k);
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                const __amdgpu_buffer_rsrc_t r = group_rsrc(kbase, t0 + 16 * u);
#pragma unroll
                for (int c = 0; c < NC; ++c)
                    kr[u][c] = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(r, koff + 64 * c, 0, 0));
            }
        };

        // V slice k -> ring stage ST by LDS DMA.  Instruction i moves 1 KiB: slice tokens
        // T = (64i + lane) / CPR (within one 16-row group), chunk ((64i + lane) % CPR) ^ swz(T),
        // where swz(T) = 2T mod CPR spreads a column read by ds_read_b64_tr_b16 over all banks.
        uint32_t voff[VDMA];
#pragma unroll
        for (int i = 0; i < VDMA; ++i) {
            const int p = 64 * i + lane;
            const int T = p / CPR, sl = p % CPR;
            voff[i] = (T % kPageSize) * ROWB + 16 * (sl ^ ((2 * T) & (CPR - 1)));
        }
        auto issue_v = [&](int k, auto ST) {
            constexpr int st = decltype(ST)::value;
            const int t0 = slice_tok0(k);
            lds_void *dst = (lds_void *)&vring[wave][st][0];
            const __amdgpu_buffer_rsrc_t r0 = group_rsrc(vbase, t0), r1 = group_rsrc(vbase, t0 + 16);
#pragma unroll
            for (int i = 0; i < VDMA; ++i)
                buffer_to_lds16(((64 * i) / CPR < 16) ? r0 : r1,
                                (lds_void *)((__attribute__((address_space(3))) char *)dst + 1024 * i), voff[i]);
        };

        // LDS byte addresses, relative to the wave's ring, of the transposed V reads: for d-tile
        // e and token half h, lane (q4, 4j + m) reads slice token T = 16h + 4*q4 + j, d = 16e + 4m.
        const uint32_t ring0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char *)&vring[wave][0][0];
        uint32_t traddr[NE][2];
        {
            const int jt = l16 >> 2, m4 = l16 & 3;
#pragma unroll
            for (int e = 0; e < NE; ++e)
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const int T = 16 * h + 4 * q4 + jt;
                    const int slot = (2 * e + (m4 >> 1)) ^ ((2 * T) & (CPR - 1));
                    traddr[e][h] = ring0 + T * CPR * 16 + slot * 16 + (m4 & 1) * 8;
                }
        }

        f32x4 acc[NT][NE];
        float m_ref[NT], l_run[NT];
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            m_ref[t] = -INFINITY;
            l_run[t] = 0.f;
#pragma unroll
            for (int e = 0; e < NE; ++e) acc[t][e] = f32x4{0.f, 0.f, 0.f, 0.f};
        }

        auto compute = [&](int k, const bf16x8 (&kr)[2][NC], auto ST) {
            constexpr int st = decltype(ST)::value;
            // V^T operands (issued first so the LDS latency overlaps the score MFMAs): the
            // transposed read hands lane l16 column d = 16e + l16 of four slice tokens
            vtr_t vr[NE][2];
#pragma unroll
            for (int e = 0; e < NE; ++e)
#pragma unroll
                for (int h = 0; h < 2; ++h) vr[e][h] = ds_read_tr16<st * SLICE_CHUNKS * 16>(traddr[e][h]);

            const int valid = tok_end - slice_tok0(k);  // keys of this slice that exist (may exceed 32)
            const bool full = valid >= kSlice;
            bf16x8 ph[NT], pl[NT];
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                ph[t] = bf16x8{};
                pl[t] = bf16x8{};
                if (t >= nt_act) continue;
                f32x4 s0 = {0.f, 0.f, 0.f, 0.f}, s1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int c = 0; c < NC; ++c) {
                    s0 = mfma16(kr[0][c], qb[t][c], s0);
                    s1 = mfma16(kr[1][c], qb[t][c], s1);
                }
                // lane: row 16t + l16, slice tokens 4*q4 + j (s0) and 16 + 4*q4 + j (s1); raw q.k
                float x[8] = {s0[0], s0[1], s0[2], s0[3], s1[0], s1[1], s1[2], s1[3]};
                if (__builtin_expect(!full, 0)) {
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        x[j] = (4 * q4 + j < valid) ? x[j] : -INFINITY;
                        x[4 + j] = (16 + 4 * q4 + j < valid) ? x[4 + j] : -INFINITY;
                    }
                }
                float mx = fmaxf(fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3])), fmaxf(fmaxf(x[4], x[5]), fmaxf(x[6], x[7])));
                mx = max_over_rows(mx) * a.scale_log2;  // the scale is positive: the order is kept
                const bool move = mx > m_ref[t] + kRescaleGap;
                if (__builtin_expect(__builtin_amdgcn_ballot_w64(move) != 0, 0)) {
                    const float m_new = move ? mx : m_ref[t];
                    const float alpha = fast_exp2(m_ref[t] - m_new);  // 0 when m_ref was -inf
                    l_run[t] *= alpha;
#pragma unroll
                    for (int e = 0; e < NE; ++e) acc[t][e] *= alpha;
                    m_ref[t] = m_new;
                }
                const float nm = (m_ref[t] == -INFINITY) ? 0.f : -m_ref[t];
                float p[8];
                float ps = 0.f;
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    p[i] = fast_exp2(__builtin_fmaf(x[i], a.scale_log2, nm));
                    ps += p[i];
                }
                l_run[t] += ps;
                // p = hi + lo: hi keeps the top 16 bits (a bf16), lo is the rest rounded to bf16
                uint32_t hw[4];
                float lo[8];
#pragma unroll
                for (int i = 0; i < 8; ++i) lo[i] = p[i] - __uint_as_float(__float_as_uint(p[i]) & 0xffff0000u);
#pragma unroll
                for (int w = 0; w < 4; ++w)
                    hw[w] = __builtin_amdgcn_perm(__float_as_uint(p[2 * w + 1]), __float_as_uint(p[2 * w]), 0x07060302u);
                ph[t] = __builtin_bit_cast(bf16x8, hw);
#pragma unroll
                for (int i = 0; i < 8; ++i) pl[t][i] = (__bf16)lo[i];
            }
            lds_wait_all(vr);
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                if (t >= nt_act) break;
#pragma unroll
                for (int e = 0; e < NE; ++e) {
                    const bf16x8 va = join_tr16(vr[e][0], vr[e][1]);
                    acc[t][e] = mfma16(va, ph[t], acc[t][e]);
                    acc[t][e] = mfma16(va, pl[t], acc[t][e]);
                }
            }
        };

        // Pipeline: K and V kDepth slices ahead, slice k in V ring stage and K register set
        // k % kStages.  Loads are issued for every step (slices past this wave's last one have
        // empty buffer resources and move no data), so the issue order is fixed:
        // V0 K0 V1 K1 ... | V(k+kDepth) K(k+kDepth) before computing slice k.  The loads issued
        // after K(k) are then V(k+1), K(k+1), ..., V(k+kDepth), K(k+kDepth); V(k) precedes K(k).
        bf16x8 kbuf[kStages][2][NC];
        static_for<kDepth>([&](auto J) {
            constexpr int j = decltype(J)::value;
            issue_v(j, std::integral_constant<int, j>{});
            load_k(j, kbuf[j]);
        });
        for (int k = 0; k < ns; k += kStages) {
            static_for<kStages>([&](auto PH) {
                constexpr int ph = decltype(PH)::value;
                constexpr int ahead = (ph + kDepth) % kStages;
                issue_v(k + ph + kDepth, std::integral_constant<int, ahead>{});
                load_k(k + ph + kDepth, kbuf[ahead]);
                wait_vm<2 * kDepth * KLOADS>();
                if (ph == 0 || k + ph < ns) compute(k + ph, kbuf[ph], PH);
            });
        }

        // combine the four waves' (max, sum, accumulator) per row and write the partial
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const float ls = sum_over_rows(l_run[t]);
            if (q4 == 0) {
                red_m[wave][t][l16] = m_ref[t];
                red_l[wave][t][l16] = ls;
            }
        }
        wait_vm<0>();
        __syncthreads();  // every wave is done with its ring: it becomes the output staging
        float *lds_o = reinterpret_cast<float *>(&vring[0][0][0]);  // [kWaves][16][OSTRIDE]
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            if (t >= nt_act) break;
            float M = -INFINITY;
#pragma unroll
            for (int w = 0; w < kWaves; ++w) M = fmaxf(M, red_m[w][t][l16]);
            const float Mu = (M == -INFINITY) ? 0.f : M;
            float L = 0.f;
#pragma unroll
            for (int w = 0; w < kWaves; ++w) L += red_l[w][t][l16] * fast_exp2(red_m[w][t][l16] - Mu);
            // L == 0 only when the item saw no keys; a NaN input keeps propagating
            const float mine = (m_ref[t] == -INFINITY) ? 0.f : fast_exp2(m_ref[t] - Mu);
            const float f = (L == 0.f) ? 0.f : mine / L;
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
                    for (int k2 = 0; k2 < PER; ++k2) o[k2] = 0.f;
#pragma unroll
                    for (int w = 0; w < kWaves; ++w)
#pragma unroll
                        for (int k2 = 0; k2 < PER; ++k2) o[k2] += lds_o[(w * 16 + r) * OSTRIDE + d0 + k2];
                    float *dst = a.part_o + (((size_t)it.part * a.n_seqs + seq) * a.n_q_heads + h) * HD + d0;
#pragma unroll
                    for (int k2 = 0; k2 < PER; k2 += 4)
                        *reinterpret_cast<f32x4 *>(dst + k2) = f32x4{o[k2], o[k2 + 1], o[k2 + 2], o[k2 + 3]};
                    if ((tid & 15) == 0) {
                        float Mr = -INFINITY;
#pragma unroll
                        for (int w = 0; w < kWaves; ++w) Mr = fmaxf(Mr, red_m[w][t][r]);
                        const float Mru = (Mr == -INFINITY) ? 0.f : Mr;
                        float Lr = 0.f;
#pragma unroll
                        for (int w = 0; w < kWaves; ++w) Lr += red_l[w][t][r] * fast_exp2(red_m[w][t][r] - Mru);
                        a.part_lse[((size_t)it.part * a.n_seqs + seq) * a.n_q_heads + h] =
                            (Lr == 0.f) ? -INFINITY : (Mru + log2f(Lr)) * kLn2;
                    }
                }
            }
            __syncthreads();
        }
        wait_vm<0>();
        if (bad_page) atomicOr(a.err, kErrBadPage);
    }

    // the last block out re-arms the queue for the next launch
    if (tid == 0) {
        __threadfence();
        if (atomicAdd(a.done, 1) == (int)gridDim.x - 1) {
            *a.queue = 0;
            *a.done = 0;
        }
    }
}

template <int HD, bool PAGED>
hipError_t launch_hd(const AttnArgs &a, int n_blocks, int row_tiles, hipStream_t s)
{
    const dim3 grid(n_blocks), block(kThreads);
    switch (row_tiles) {
    case 1: partials_kernel<HD, 1, PAGED><<<grid, block, 0, s>>>(a); break;
    case 2: partials_kernel<HD, 2, PAGED><<<grid, block, 0, s>>>(a); break;
    case 3: partials_kernel<HD, 3, PAGED><<<grid, block, 0, s>>>(a); break;
    case 4: partials_kernel<HD, 4, PAGED><<<grid, block, 0, s>>>(a); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace

hipError_t launch_partials(const AttnArgs &a, int n_blocks, int head_dim, int row_tiles, hipStream_t s)
{
    if (a.n_items <= 0 || n_blocks <= 0) return hipSuccess;
    if (head_dim == 128) return a.paged ? launch_hd<128, true>(a, n_blocks, row_tiles, s)
                                        : launch_hd<128, false>(a, n_blocks, row_tiles, s);
    if (head_dim == 64) return a.paged ? launch_hd<64, true>(a, n_blocks, row_tiles, s)
                                       : launch_hd<64, false>(a, n_blocks, row_tiles, s);
    return hipErrorInvalidValue;
}

}  // namespace fka
