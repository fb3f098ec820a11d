// Partial attention over key ranges: the streaming stage of fork-aware decode
// attention on gfx950 (CDNA4, wave64).
//
// Every launch first rebuilds the work schedule (internal.h) from the suffix lengths on
// the device: the 32-token slices of the shared prefix items and of the suffix items are
// spread evenly over all waves of the grid.  The waves of a block that share an item deal
// the slices of their joint range among themselves in turn, so the block streams one
// contiguous region and its waves finish together.  An item holds every query row that reads its keys: for a
// shared-prefix item, all sequences of the fork x the G query heads of the KV head, so
// each prefix K/V byte is fetched from HBM once for all branches (paper, Sec. 3.3: the
// prefix cache is reused by all decoding streams).  Within a wave:
//   * K rows are loaded straight into registers in the MFMA A-operand layout
//     (16 tokens x 4 lanes x 16 bytes per instruction) one slice ahead;
//   * V rows are copied by LDS DMA (buffer_load_dwordx4 ... lds) into a wave-private
//     ring of two slices, one slice ahead, and read back transposed with
//     ds_read_b64_tr_b16;
//   * loads go through buffer resources sized to the rows that exist, so rows past the
//     end of a key range read as zeros without any per-lane test;
//   * S^T = K Q^T and O^T += V^T P^T run on v_mfma_f32_16x16x32_bf16 with tokens
//     on M, so each lane owns one query row of the online softmax; P enters the
//     second product as two bf16 terms (hi + lo), which keeps it accurate to ~2^-16;
//   * the running maximum is only moved when a score exceeds it by more than 2^8,
//     so the accumulator is rarely rescaled.
// At the end the waves of a block that worked on the same item combine their
// (max, sum, accumulator) through LDS and write one normalised partial (o, lse) per row.
// Blocks of eight waves (two per SIMD) where the registers allow it: d = 64, or at most
// 32 query rows of d = 128; four waves otherwise.
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

constexpr int kStages = 2;  // V ring stages and K register sets per wave: one slice ahead
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

// Cache policy of the K/V stream: non-temporal (each byte is read once; measured 6% faster on
// the 32k-prefix workload and 13% on the 128k one), except paged K.  A K load instruction reads
// 64 bytes of each of 16 rows (the MFMA operand layout), so with 4 KiB (page, head) blocks in
// page-table order the halves of a 128-byte line come from different instructions; without
// the line kept in the cache that measured 12% slower on the paged workload, the default policy
// is kept there.  V arrives by LDS DMA, 1 KiB contiguous per instruction: non-temporal in both
// layouts (5% faster on the paged workload than the default).
template <bool PAGED>
constexpr int k_policy()
{
    return PAGED ? 0 : 2;
}
constexpr int kVPolicy = 2;

// 16 bytes per lane from a buffer into LDS at dst + 16 * lane (LDS DMA).  Kept outside
// the kernel template: used directly there, the builtin stops the host compiler from
// emitting the kernel's launch stub.
template <int POLICY>
__device__ inline void buffer_to_lds16(__amdgpu_buffer_rsrc_t r, lds_void *dst, uint32_t voff)
{
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, dst, 16, voff, 0, 0, POLICY);
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

// Lane id computed at the point of use (the asm cannot be hoisted or merged with an
// earlier copy).
__device__ inline int opaque_lane_id()
{
    int v;
    asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(v));
    return v;
}

// Sixteen wait states between MFMAs and the first VALU read of their results.  The wait
// states the compiler counts before such a read on gfx950 can fall short: the first score
// registers read after the q.k MFMAs were seen to hold the previous slice's values (the row
// maximum then came out of stale scores, which showed as rounding-level differences between
// identical rows of different tiles).  Sixteen covers a 4-pass XDL result with margin; the
// scheduling barriers keep the MFMAs above the wait and the reads below it.
__device__ inline void xdl_result_wait()
{
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("s_nop 7\n\ts_nop 7" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
}

// Block barrier for LDS hand-offs: waits for this wave's LDS operations only, so global
// stores and prefetches in flight stay in flight (__syncthreads would wait for them too).
__device__ inline void lds_barrier()
{
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

__device__ inline bf16x8 join_tr16(vtr_t lo, vtr_t hi)
{
    const s16x4 a = __builtin_bit_cast(s16x4, lo), b = __builtin_bit_cast(s16x4, hi);
    const short __attribute__((ext_vector_type(8))) v = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
    return __builtin_bit_cast(bf16x8, v);
}

// Waves per SIMD (and so per block: four times as many, one block per compute unit).  d = 128:
// one wave per SIMD with the whole register file (three or four 16-row tiles need it; with one
// or two, contiguous K/V measured 1% faster on the 32k-prefix workload and 5% on the 8k one
// than two waves of <= 256 VGPRs, whose older wave finishes well before the younger), except
// paged K/V with one or two tiles, where two waves per SIMD measured 11% faster.  d = 64: two.
template <int HD, int NT, bool PAGED>
constexpr int waves_per_simd()
{
    return (HD <= 64 || (PAGED && NT <= 2)) ? 2 : 1;
}

template <int HD, int NT, bool PAGED>
__global__ __launch_bounds__((256 * waves_per_simd<HD, NT, PAGED>()))
__attribute__((amdgpu_waves_per_eu(waves_per_simd<HD, NT, PAGED>()))) void partials_kernel(AttnArgs a)
{
    constexpr int NW = 4 * waves_per_simd<HD, NT, PAGED>();  // waves per block
    constexpr int NTH = 64 * NW;
    constexpr int CPR = HD / 8;                 // 16-byte chunks per K/V row
    constexpr int NC = HD / 32;                 // MFMA k-steps of q.k
    constexpr int NE = HD / 16;                 // MFMA d-tiles of p.v
    constexpr int SLICE_CHUNKS = kSlice * CPR;  // 16-byte chunks of one V slice
    constexpr int VDMA = SLICE_CHUNKS / 64;     // LDS DMA instructions per V slice
    constexpr int KLOADS = 2 * NC;              // K loads per lane per slice
    static_assert(VDMA == KLOADS, "one wait count per slice");
    constexpr int ROWB = HD * 2;                // bytes per K/V row
    static_assert(2 * 16 * HD * 4 <= kStages * SLICE_CHUNKS * 16, "two tiles fit in a wave's ring");
    // 16-row tiles the combine stages per pass: all of them for d = 128 (one block per CU, so
    // the LDS is there), else the two that fit in a wave's ring
    constexpr int TPP = (HD == 128 && NT > 2) ? NT : 2;
    constexpr int NPASS = (NT + TPP - 1) / TPP;

    // per wave: kStages V slices; chunk c of slice token T sits at T*CPR + (c ^ swz(T))
    __shared__ uint4 vring[NW][kStages][SLICE_CHUNKS];
    __shared__ __attribute__((aligned(16))) float red_m[NT][16][NW];  // per row, the waves side by side
    __shared__ __attribute__((aligned(16))) float red_l[NT][16][NW];
    // staging of 16-row tiles past the first two when one pass holds them all
    __shared__ __attribute__((aligned(16))) float stg_x[NW][TPP > 2 ? (TPP - 2) * 16 * HD : 4];
    __shared__ int32_t s_len[kMaxSeqs], s_cs[kMaxSeqs], s_ne[kMaxSeqs];
    __shared__ int32_t s_wsum[2][NW];
    __shared__ int32_t s_spl[PAGED ? kMaxSeqs : 1];  // prefix length of each sequence's unit
    // each wave's item: item, seq0, nseq, kv head, keys, and its group (the block's waves on the
    // same item): first wave, first slice, end slice, end wave
    __shared__ int32_t s_wfc[2][NW][9];  // per candidate schedule (the built one goes to [0])
    __shared__ __attribute__((aligned(16))) int32_t s_grp[NW][4];  // the block's groups: first wave, end wave, rows, item
    __shared__ int32_t s_ngrp;
    __shared__ int32_t s_stale[NW];   // bit c: a wave saw a suffix length that differs from key c

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform per wave
    const int l16 = lane & 15, q4 = lane >> 4;
    const int G = a.group, Hkv = a.n_kv_heads, N = a.n_seqs;

    // ---- the schedule.  One round trip brings the suffix lengths (and, paged, the prefix
    // lengths of the sequences' units), the cached candidates' keys and this block's table rows
    // and the static prefix item of this thread's first item.  The first candidate whose key
    // equals the clamped lengths is taken; otherwise the block builds the schedule (internal.h).
    const int vb = (int)blockIdx.x;
    const int w_lo = vb * NW;
    // the kernel arguments this needs, all read before the first branch: the compiler would
    // otherwise fetch them one branch at a time, a scalar round trip each
    const int32_t *tab0 = a.tab[0] + (size_t)w_lo * kTabWords, *tab1 = a.tab[1] + (size_t)w_lo * kTabWords;
    const int32_t *key0 = a.key[0], *key1 = a.key[1], *sl = a.suffix_len, *spl = a.seq_prefix_len;
    const int32_t *pre = reinterpret_cast<const int32_t *>(a.pre_items);
    int32_t *lens = a.lens;
    const int n_pre = a.n_pre, max_len = a.max_suffix_len;
    asm volatile("" ::"s"(tab0), "s"(tab1), "s"(key0), "s"(key1), "s"(sl), "s"(spl), "s"(pre), "s"(lens),
                 "s"(n_pre), "s"(max_len));
    int32_t tab_v[2] = {0, 0};
    if (tid < NW * kTabWords) {
        tab_v[0] = tab0[tid];
        tab_v[1] = tab1[tid];
    }
    int32_t my_pre[6] = {0, 0, 0, 0, 0, 0};  // seq0, nseq, kv_head, n_tok, c0, k0
    if (tid < n_pre) {
#pragma unroll
        for (int f = 0; f < 6; ++f) my_pre[f] = pre[tid * 8 + f];
    }
    bool clamped = false, stale0 = false, stale1 = false;
    for (int s = tid; s < N; s += NTH) {
        const int raw = sl[s];
        const int k0 = key0[s], k1 = key1[s];
        const int L = min(max(raw, 0), max_len);
        clamped |= (L != raw);
        stale0 |= (k0 != L);
        stale1 |= (k1 != L);
        s_len[s] = L;
        if (PAGED) s_spl[s] = spl[s];
        if (vb == 0) lens[s] = L;  // what the merge appends at
    }
    if (vb == 0 && clamped) atomicOr(a.err, kErrSuffixClamped);
    const int wave_stale = (__builtin_amdgcn_ballot_w64(stale0) != 0 ? 1 : 0) |
                           (__builtin_amdgcn_ballot_w64(stale1) != 0 ? 2 : 0);
    if (lane == 0) s_stale[wave] = wave_stale;
    if (tid < NW * kTabWords) {  // both candidates' rows; the chosen one is used below
        const int w = tid / kTabWords, f = tid % kTabWords;
        s_wfc[0][w][f] = tab_v[0];
        s_wfc[1][w][f] = tab_v[1];
    }
    lds_barrier();
    int any_stale = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) any_stale |= s_stale[w];
    any_stale = __builtin_amdgcn_readfirstlane(any_stale);
    const int choice = !(any_stale & 1) ? 0 : !(any_stale & 2) ? 1 : 2;
    if (vb == 0 && tid == 0) *a.sel = choice;
    int32_t(*s_wf)[9] = s_wfc[choice == 1 ? 1 : 0];
    if (choice == 2) {
        if (tid < NW) s_wf[tid][0] = -1;  // waves the placement below does not reach have no item
        // per-sequence suffix tables: CS(s), NE(s) (exclusive scans)
        int carry_cs = 0, carry_ne = 0;
        for (int base = 0; base < N; base += NTH) {
            const int s = base + tid;
            const int L = s < N ? s_len[s] : 0;
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
                s_wsum[0][wave] = x;
                s_wsum[1][wave] = y;
            }
            lds_barrier();
            int px = carry_cs, py = carry_ne;
            for (int w = 0; w < NW; ++w) {
                if (w < wave) {
                    px += s_wsum[0][w];
                    py += s_wsum[1][w];
                }
                carry_cs += s_wsum[0][w];
                carry_ne += s_wsum[1][w];
            }
            if (s < N) {
                s_cs[s] = px + x - xs;
                s_ne[s] = py + y - xe;
            }
            lds_barrier();
        }
        const int T = __builtin_amdgcn_readfirstlane(a.pre_slices + carry_cs);      // total slices
        const int NNE = __builtin_amdgcn_readfirstlane(a.pre_nonempty + carry_ne);  // non-empty items
        const int NV = (int)gridDim.x * NW;  // workers: every block is one virtual block
        const uint64_t R = T > 0 ? sched_ratio((int64_t)NV - NNE, T) : 0;
        const int n_items = a.n_pre + N * Hkv;
        // every thread places its items' workers of this block; the block holding an item's
        // first worker writes the item's slot records for the merge (block 0 those of empty items)
        for (int i = tid; i < n_items; i += NTH) {
            int f[6];
            int size, C, K;
            if (i < a.n_pre) {
                if (i == tid) {  // loaded at the start
#pragma unroll
                    for (int k = 0; k < 6; ++k) f[k] = my_pre[k];
                } else {
                    const int32_t *ip = reinterpret_cast<const int32_t *>(a.pre_items + i);
#pragma unroll
                    for (int k = 0; k < 6; ++k) f[k] = ip[k];
                }
                size = slices_of(f[3]);
                C = f[4];
                K = f[5];
            } else {
                const int j = i - a.n_pre, sq = j / Hkv, g = j % Hkv;
                f[0] = sq;
                f[1] = 1;
                f[2] = g;
                f[3] = s_len[sq];
                size = slices_of(f[3]);
                C = a.pre_slices + s_cs[sq] + g * size;
                K = a.pre_nonempty + s_ne[sq] + (size > 0 ? g : 0);
            }
            if (size == 0 || T == 0) {
                if (vb == 0) write_rowrecs(a.rowrec_live, i, a.n_pre, f[0], f[1], f[2], G, a.n_q_heads, a.slot_rows, 0, 0);
                continue;
            }
            const int ws0 = worker_start(C, K, R), ws1 = worker_start(C + size, K + 1, R);
            if (ws0 >= w_lo && ws0 < w_lo + NW)
                write_rowrecs(a.rowrec_live, i, a.n_pre, f[0], f[1], f[2], G, a.n_q_heads, a.slot_rows, vb,
                              (ws1 - 1) / NW - vb + 1);
            if (ws1 <= w_lo || ws0 >= w_lo + NW) continue;
            // the block's workers [lo, hi) of this item form one group over the union of
            // their slice ranges; its waves deal the slices in turn
            int lo, hi, glo, ghi;
            block_group(vb, NW, ws0, ws1, size, lo, hi, glo, ghi);
            for (int gw = lo; gw < hi; ++gw) {
                int32_t *d = s_wf[gw - w_lo];
                d[0] = i;
                d[1] = f[0];
                d[2] = f[1];
                d[3] = f[2];
                d[4] = f[3];
                d[5] = lo - w_lo;
                d[6] = glo;
                d[7] = ghi;
                d[8] = hi - w_lo;
            }
        }
        lds_barrier();
    }

    {
        const int item = __builtin_amdgcn_readfirstlane(s_wf[wave][0]);
        if (wave == 0) {  // the block's groups, in wave order (read after the combine barrier)
            const int w = lane < NW ? lane : 0;  // lane w looks at wave w
            const bool lead = lane < NW && s_wf[w][0] >= 0 && s_wf[w][5] == w;
            const uint64_t m = __builtin_amdgcn_ballot_w64(lead);
            if (lead) {
                const int n = __builtin_popcountll(m & ((uint64_t(1) << w) - 1));
                s_grp[n][0] = w;
                s_grp[n][1] = s_wf[w][8];
                s_grp[n][2] = s_wf[w][2] * G;
                s_grp[n][3] = s_wf[w][0];
            }
            if (lane == 0) s_ngrp = __builtin_popcountll(m);
        }

        // ---- this wave's item and group (all values uniform)
        bool suffix = false;
        int seq0 = 0, nseq = 0, kvh = 0, tok_end = 0, unit_prefix = 0;
        int wa = wave, ghi = 0;
        if (item >= 0) {
            seq0 = __builtin_amdgcn_readfirstlane(s_wf[wave][1]);
            nseq = __builtin_amdgcn_readfirstlane(s_wf[wave][2]);
            kvh = __builtin_amdgcn_readfirstlane(s_wf[wave][3]);
            tok_end = __builtin_amdgcn_readfirstlane(s_wf[wave][4]);
            wa = __builtin_amdgcn_readfirstlane(s_wf[wave][5]);
            ghi = __builtin_amdgcn_readfirstlane(s_wf[wave][7]);
            suffix = item >= a.n_pre;
            if (PAGED && suffix) unit_prefix = __builtin_amdgcn_readfirstlane(s_spl[seq0]);
        }
        const int rows = nseq * G;
        const int nt_act = (rows + 15) >> 4;
        // keys of the group end at tok_lim: loads past it (the prefetch beyond the last slice)
        // move no data, and scores past it are masked
        const int tok_lim = min(tok_end, ghi * kSlice);
        // next slice of this wave: wave j of the group's g waves takes glo + j, glo + j + g, ...
        // (a fixed assignment, so results repeat bit for bit; it also measured faster than
        // taking slices from a shared LDS counter, whose round trip delayed each slice's loads)
        const int g_waves = item >= 0 ? __builtin_amdgcn_readfirstlane(s_wf[wave][8]) - wa : 1;
        int next_slice = (item >= 0 ? __builtin_amdgcn_readfirstlane(s_wf[wave][6]) : 0) + (wave - wa);
        auto grab = [&]() -> int {
            const int k = next_slice;
            next_slice += g_waves;
            return k;
        };

        // key source of the item
        const char *kbase = reinterpret_cast<const char *>(a.q), *vbase = kbase;
        const int32_t *ptab = a.page_table;
        int page_off = 0;
        if (item >= 0) {
            if (PAGED) {
                kbase = reinterpret_cast<const char *>(a.k_pool);
                vbase = reinterpret_cast<const char *>(a.v_pool);
                ptab = a.page_table + (size_t)seq0 * a.max_pages;
                if (suffix) page_off = (unit_prefix + kPageSize - 1) / kPageSize;
            } else if (suffix) {
                const size_t base = ((size_t)seq0 * Hkv + kvh) * (size_t)a.suffix_cap * HD * 2;
                kbase = reinterpret_cast<const char *>(a.suffix_k) + base;
                vbase = reinterpret_cast<const char *>(a.suffix_v) + base;
            } else {
                const size_t base = (size_t)kvh * (size_t)a.prefix_len * HD * 2;
                kbase = reinterpret_cast<const char *>(a.prefix_k) + base;
                vbase = reinterpret_cast<const char *>(a.prefix_v) + base;
            }
        }
        auto slice_tok0 = [&](int k) { return k * kSlice; };

        // Buffer resource over the 16-row group holding positions [t, t + 16) (t is a
        // multiple of 16, so a group never straddles a page).  Its size covers only the rows
        // below tok_lim, so loads of rows past the end (or of a group wholly past it, or behind
        // an out-of-range page id) return zeros.  Uniform.
        bool bad_page = false;
        auto group_rsrc = [&](const char *src, int t) -> __amdgpu_buffer_rsrc_t {
            const int rows_ok = max(0, min(kPageSize, tok_lim - t));
            const char *base = src;
            if (!PAGED) {
                base = src + (size_t)t * ROWB;
            } else if (rows_ok > 0) {
                const int32_t page = scalar_load(ptab + min(page_off + t / kPageSize, a.max_pages - 1));
                if (page < 0 || page >= a.n_pool_pages) {
                    bad_page = true;
                    return make_rsrc(src, 0);
                }
                base = src + ((size_t)page * Hkv + kvh) * (kPageSize * ROWB);
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
                const int seq = seq0 + r / G, h = kvh * G + r % G;
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
                    kr[u][c] = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(r, koff + 64 * c, 0, k_policy<PAGED>()));
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
                buffer_to_lds16<kVPolicy>(((64 * i) / CPR < 16) ? r0 : r1,
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

            const int valid = tok_lim - slice_tok0(k);  // keys of this slice in range (may exceed 32)
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
                xdl_result_wait();
                // lane: row 16t + l16, slice tokens 4*q4 + j (s0) and 16 + 4*q4 + j (s1); raw q.k
                float x[8] = {s0[0], s0[1], s0[2], s0[3], s1[0], s1[1], s1[2], s1[3]};
                if (__builtin_expect(!full, 0)) {
                    const int v4 = valid - 4 * q4;  // keys left from this lane's first token
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        x[j] = (j < v4) ? x[j] : -INFINITY;
                        x[4 + j] = (16 + j < v4) ? x[4 + j] : -INFINITY;
                    }
                }
                float mx = fmaxf(fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3])), fmaxf(fmaxf(x[4], x[5]), fmaxf(x[6], x[7])));
                mx = max_over_rows(mx) * a.scale_log2;  // the scale is positive: the order is kept
                const bool move = mx > m_ref[t] + kRescaleGap;
                if (__builtin_expect(__builtin_amdgcn_ballot_w64(move) != 0, 0)) {
                    const float m_new = move ? mx : m_ref[t];
                    // exactly 1 for a row that keeps its max (the hardware exp2 of 0 need not be),
                    // so a row's result does not depend on the other rows of its tile; 0 when
                    // the row's max was -inf
                    const float alpha = move ? fast_exp2(m_ref[t] - m_new) : 1.f;
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

        // Pipeline, one slice ahead: slice kc sits in V ring stage 0 / K registers 0 while the
        // next one loads into stage 1, then the roles swap.  Loads are issued at every step
        // (slices past the group's end have empty buffer resources and move no data), so the
        // wait count is fixed: V(k), K(k) precede the two loads of the slice behind them.  The
        // loop is tested at the top (a test in the middle costs the allocator registers).
        if (item >= 0) {
            bf16x8 kbuf[kStages][2][NC];
            int kc = grab();
            issue_v(kc, std::integral_constant<int, 0>{});
            load_k(kc, kbuf[0]);
            while (kc < ghi) {
                const int kn = grab();
                issue_v(kn, std::integral_constant<int, 1>{});
                load_k(kn, kbuf[1]);
                wait_vm<2 * KLOADS>();
                compute(kc, kbuf[0], std::integral_constant<int, 0>{});
                kc = grab();
                issue_v(kc, std::integral_constant<int, 0>{});
                load_k(kc, kbuf[0]);
                wait_vm<2 * KLOADS>();
                if (kn < ghi)
                    compute(kn, kbuf[1], std::integral_constant<int, 1>{});
                else
                    kc = ghi;
            }
        }

        // ---- combine the (max, sum, accumulator) of the waves that worked on this item.
        // Lane-derived values are recomputed here from an opaque lane id: values kept from the
        // kernel start would have been spilled, and their reloads wait for every load in flight.
        const int lane_c = opaque_lane_id();
        const int l16c = lane_c & 15, q4c = lane_c >> 4, tid_c = wave * 64 + lane_c;
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const float ls = sum_over_rows(l_run[t]);
            if (q4c == 0) {
                red_m[t][l16c][wave] = m_ref[t];
                red_l[t][l16c][wave] = ls;
            }
        }
        wait_vm<0>();  // this wave's ring is idle: it takes the wave's raw accumulators
        // Staging: wave w writes [tile][row][d] of its own accumulator (the 16-float blocks of a
        // row XOR-permuted by the row, for the banks): tiles 0 and 1 into its ring, further tiles
        // into stg_x when a pass holds them, else in later passes.  After one barrier, threads own
        // (row, unit) pieces of each group: they weigh the group's waves by exp(max_w - max), sum,
        // and normalise; the unit holding the row's first floats also stores its lse.  (A separate
        // step computing the weights once per row cost more than it saved: one wave ran it alone
        // behind a second barrier.)  All global stores of a pass follow its LDS work.
        // A unit is UQ 16-byte chunks of one row: 16 floats with four waves to sum (measured
        // 0.3-0.5 us faster per launch than 8), else 8.
        constexpr int UQ = NW == 4 ? 4 : 2;
        constexpr int CHU = HD / (4 * UQ);  // units per row
        auto stg = [&](int w, int tt) -> const float * {
            if (TPP <= 2 || tt < 2) return reinterpret_cast<const float *>(&vring[w][0][0]) + tt * 16 * HD;
            return &stg_x[w][(tt - 2) * 16 * HD];
        };
        auto stg_off = [&](int r, int c4) {  // float offset of chunk c4 (4 floats) of row r in a tile
            return r * HD + 16 * ((c4 >> 2) ^ (r & (NE - 1))) + 4 * (c4 & 3);
        };
#pragma unroll
        for (int pass = 0; pass < NPASS; ++pass) {
            if (pass > 0) lds_barrier();  // the previous pass has read the staging
#pragma unroll
            for (int tt = 0; tt < TPP; ++tt) {
                const int t = TPP * pass + tt;
                if (t >= NT) break;
                if (item >= 0 && t < nt_act) {
                    float *dst = const_cast<float *>(stg(wave, tt));
#pragma unroll
                    for (int e = 0; e < NE; ++e)
                        *reinterpret_cast<f32x4 *>(&dst[stg_off(l16c, 4 * e + q4c)]) = acc[t][e];
                }
            }
            lds_barrier();  // also orders the group table (written by wave 0 before streaming)
            const int n_grp = min(s_ngrp, NW);
            for (int g = 0; g < n_grp; ++g) {
                const int4 gi = *reinterpret_cast<const int4 *>(&s_grp[g][0]);
                asm volatile("" ::"v"(gi.x), "v"(gi.y), "v"(gi.z), "v"(gi.w));  // one LDS read, not four
                const int lw = gi.x, ge = gi.y, it = gi.w;
                if (vb + it >= a.n_slots || it < 0) continue;  // never store outside the workspace
                const int r0 = 16 * TPP * pass, r1 = min(gi.z, r0 + 16 * TPP);
                const bool whole = lw == 0 && ge == NW;  // the usual case: one group, all waves
                for (int u = tid_c; u < (r1 - r0) * CHU; u += NTH) {
                    const int row = r0 + u / CHU, cu = u % CHU;
                    const int t = row >> 4, tt = t - TPP * pass, r = row & 15;
                    // a wave of the group that saw no keys has max -inf, weight 0 and a zero
                    // accumulator; waves outside the group are never read (their staging may
                    // hold another item's NaN)
                    float M = -INFINITY, L = 0.f;
                    f32x4 o[UQ];
#pragma unroll
                    for (int q = 0; q < UQ; ++q) o[q] = f32x4{0.f, 0.f, 0.f, 0.f};
                    if (whole) {
                        float mw[NW], lw_[NW];
                        f32x4 v[NW][UQ];
#pragma unroll
                        for (int w = 0; w < NW; ++w) {
                            mw[w] = red_m[t][r][w];
                            lw_[w] = red_l[t][r][w];
#pragma unroll
                            for (int q = 0; q < UQ; ++q)
                                v[w][q] = *reinterpret_cast<const f32x4 *>(&stg(w, tt)[stg_off(r, UQ * cu + q)]);
                        }
#pragma unroll
                        for (int w = 0; w < NW; ++w) M = fmaxf(M, mw[w]);
                        const float Mu = (M == -INFINITY) ? 0.f : M;
#pragma unroll
                        for (int w = 0; w < NW; ++w) {
                            const float wt = fast_exp2(mw[w] - Mu);  // 0 for max -inf
                            L = __builtin_fmaf(wt, lw_[w], L);
#pragma unroll
                            for (int q = 0; q < UQ; ++q) o[q] += wt * v[w][q];
                        }
                    } else {
                        for (int w = lw; w < ge; ++w) M = fmaxf(M, red_m[t][r][w]);
                        const float Mu = (M == -INFINITY) ? 0.f : M;
                        for (int w = lw; w < ge; ++w) {
                            const float wt = fast_exp2(red_m[t][r][w] - Mu);
                            L = __builtin_fmaf(wt, red_l[t][r][w], L);
#pragma unroll
                            for (int q = 0; q < UQ; ++q)
                                o[q] += wt * *reinterpret_cast<const f32x4 *>(&stg(w, tt)[stg_off(r, UQ * cu + q)]);
                        }
                    }
                    // L == 0 only when the group saw no keys: its accumulators are zero and so is
                    // o; a NaN input keeps propagating
                    const float inv = (L == 0.f) ? 0.f : __builtin_amdgcn_rcpf(L);
                    const size_t so = (size_t)(vb + it) * a.slot_rows + row;
                    float *dst = a.part_o + so * HD + 4 * UQ * cu;
#pragma unroll
                    for (int q = 0; q < UQ; ++q) *reinterpret_cast<f32x4 *>(dst + 4 * q) = o[q] * inv;
                    if (cu == 0) a.part_lse[so] = (L == 0.f) ? -INFINITY : (((M == -INFINITY) ? 0.f : M) + log2f(L)) * kLn2;
                }
            }
        }
        if (bad_page) atomicOr(a.err, kErrBadPage);
    }
}

template <int HD, bool PAGED>
int blocks_per_cu_hd(int row_tiles)
{
    const void *f = nullptr;
    int threads = 0;
    switch (row_tiles) {
    case 1: f = reinterpret_cast<const void *>(&partials_kernel<HD, 1, PAGED>); threads = 256 * waves_per_simd<HD, 1, PAGED>(); break;
    case 2: f = reinterpret_cast<const void *>(&partials_kernel<HD, 2, PAGED>); threads = 256 * waves_per_simd<HD, 2, PAGED>(); break;
    case 3: f = reinterpret_cast<const void *>(&partials_kernel<HD, 3, PAGED>); threads = 256 * waves_per_simd<HD, 3, PAGED>(); break;
    case 4: f = reinterpret_cast<const void *>(&partials_kernel<HD, 4, PAGED>); threads = 256 * waves_per_simd<HD, 4, PAGED>(); break;
    default: return 0;
    }
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, f, threads, 0) != hipSuccess) return 0;
    return n;
}

template <int HD, bool PAGED>
hipError_t launch_hd(const AttnArgs &a, int n_blocks, int row_tiles, hipStream_t s)
{
    const dim3 grid(n_blocks);
    switch (row_tiles) {
    case 1: partials_kernel<HD, 1, PAGED><<<grid, 256 * waves_per_simd<HD, 1, PAGED>(), 0, s>>>(a); break;
    case 2: partials_kernel<HD, 2, PAGED><<<grid, 256 * waves_per_simd<HD, 2, PAGED>(), 0, s>>>(a); break;
    case 3: partials_kernel<HD, 3, PAGED><<<grid, 256 * waves_per_simd<HD, 3, PAGED>(), 0, s>>>(a); break;
    case 4: partials_kernel<HD, 4, PAGED><<<grid, 256 * waves_per_simd<HD, 4, PAGED>(), 0, s>>>(a); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace

int partials_blocks_per_cu(int head_dim, int row_tiles, bool paged)
{
    if (head_dim == 128) return paged ? blocks_per_cu_hd<128, true>(row_tiles) : blocks_per_cu_hd<128, false>(row_tiles);
    if (head_dim == 64) return paged ? blocks_per_cu_hd<64, true>(row_tiles) : blocks_per_cu_hd<64, false>(row_tiles);
    return 0;
}

template <bool PAGED>
int waves_per_block_hd128(int row_tiles)
{
    switch (row_tiles) {
    case 1: return 4 * waves_per_simd<128, 1, PAGED>();
    case 2: return 4 * waves_per_simd<128, 2, PAGED>();
    case 3: return 4 * waves_per_simd<128, 3, PAGED>();
    case 4: return 4 * waves_per_simd<128, 4, PAGED>();
    default: return 0;
    }
}

int partials_waves_per_block(int head_dim, int row_tiles, bool paged)
{
    if (head_dim == 64) return 4 * waves_per_simd<64, 1, false>();
    return paged ? waves_per_block_hd128<true>(row_tiles) : waves_per_block_hd128<false>(row_tiles);
}

hipError_t launch_partials(const AttnArgs &a, int n_blocks, int head_dim, int row_tiles, hipStream_t s)
{
    if (n_blocks <= 0) return hipSuccess;
    if (head_dim == 128) return a.paged ? launch_hd<128, true>(a, n_blocks, row_tiles, s)
                                        : launch_hd<128, false>(a, n_blocks, row_tiles, s);
    if (head_dim == 64) return a.paged ? launch_hd<64, true>(a, n_blocks, row_tiles, s)
                                       : launch_hd<64, false>(a, n_blocks, row_tiles, s);
    return hipErrorInvalidValue;
}

}  // namespace fka
