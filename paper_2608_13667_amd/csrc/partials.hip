// Partial attention over key ranges: the streaming stage of fork-aware decode
// attention on gfx950 (CDNA4, wave64).
//
// Work items (internal.h): one per (prefix-sharing unit, KV head).  An item's rows are all the
// unit's sequences x the G query heads of its KV head, and its keys are the unit's prefix
// followed by each sequence's own suffix; every prefix slice is scored against all rows, so
// each prefix K/V byte is fetched from HBM once for all branches (paper, Sec. 3.3: the prefix
// cache is reused by all decoding streams), and a suffix slice only against its sequence's G
// rows.  With one unit (a single fork) the items split the grid statically: each wave's
// prefix slices are known from the plan alone, so their loads are issued before the suffix
// lengths arrive.  The waves of a block that share an item deal the slices of their joint
// range among themselves in turn, so the block streams one contiguous region and its waves
// finish together.  Within a wave:
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
//     so the accumulator is rarely rescaled;
//   * a suffix slice updates only its sequence's rows: the other rows' scores are -inf and
//     their accumulators are left as they were (so not even a non-finite value of another
//     branch's suffix reaches them).
// At the end the waves of a block that worked on the same item combine their
// (max, sum, accumulator) through LDS and write one normalised partial (o, lse) per row.
// Blocks of eight waves (two per SIMD) where the registers allow it: d = 64, or at most
// 32 query rows of paged d = 128; four waves otherwise.
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
// The instruction prefill reads every prefix tile once per unit, the units of a KV head together
// on one XCD: there the default policy keeps the tile in L2 for the other units.
template <bool PAGED, bool PREFILL>
constexpr int k_policy()
{
    return (PAGED || PREFILL) ? 0 : 2;
}
template <bool PREFILL>
constexpr int v_policy()
{
    return PREFILL ? 0 : 2;
}

// 16 bytes per lane from a buffer into LDS at dst + 16 * lane (LDS DMA).  Kept outside
// the kernel template: used directly there, the builtin stops the host compiler from
// emitting the kernel's launch stub.
template <int POLICY, int OFFSET>
__device__ inline void buffer_to_lds16(__amdgpu_buffer_rsrc_t r, lds_void *dst, uint32_t voff)
{
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, dst, 16, voff, 0, OFFSET, POLICY);
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

// A value the whole wave agrees on, moved to a scalar register (the compiler does not always
// see that a value is uniform; a pointer or a count held in vector registers turns scalar loads
// into vector ones and branches into divergent ones).
__device__ inline int uni(int x) { return __builtin_amdgcn_readfirstlane(x); }
template <typename T>
__device__ inline T *uni_ptr(T *p)
{
    const uint64_t b = (uint64_t)p;
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)b);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(b >> 32));
    return (T *)(((uint64_t)hi << 32) | lo);
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
// paged K/V with one or two tiles, where two waves per SIMD measured 11% faster, and the
// instruction prefill with one or two tiles, which is bound by instruction issue rather than
// bytes: there the second wave's matrix and vector work fills the first one's stalls (32-row
// units at two waves per SIMD measured 4-11% faster at the 32k shape than 64-row units at one).
// d = 64: two.
template <int HD, int NT, bool PAGED, bool PREFILL>
constexpr int waves_per_simd()
{
    return (HD <= 64 || ((PAGED || PREFILL) && NT <= 2)) ? 2 : 1;
}

// Where the keys of one slice come from (every field uniform over the wave).
struct SliceSrc {
    const char *kb, *vb;  // contiguous: K and V rows of the slice's segment; paged: the pools
    const int32_t *ptab;  // paged: page row of the segment's sequence
    int32_t page_off;     // paged: page index of the segment's position 0
    int32_t tok0;         // first position of the slice within its segment
    int32_t tok_lim;      // positions in the segment (a key at or past it does not exist)
    int32_t r_lo, r_hi;   // the query rows that read these keys
    int32_t suffix;       // 1: a suffix slice, read by rows [r_lo, r_hi) only
};

template <int HD, int NT, bool PAGED, bool PREFILL>
__global__ __launch_bounds__((256 * waves_per_simd<HD, NT, PAGED, PREFILL>()))
__attribute__((amdgpu_waves_per_eu(waves_per_simd<HD, NT, PAGED, PREFILL>()))) void partials_kernel(AttnArgs a)
{
    constexpr int NW = 4 * waves_per_simd<HD, NT, PAGED, PREFILL>();  // waves per block
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
    // proportional split only: per-sequence clamped lengths and slice scan, the units, and the
    // scan of non-empty units
    __shared__ int32_t s_len[kMaxSeqs], s_cs[kMaxSeqs + 1], s_ne[kMaxSeqs + 1];
    __shared__ int32_t s_u0[kMaxSeqs], s_un[kMaxSeqs], s_ul[kMaxSeqs], s_up[kMaxSeqs];
    __shared__ int32_t s_wsum[NW];
    // per wave: item (-1: none), unit, item workers W, the group's first and end worker within
    // the item, the group's first and end wave within the block
    __shared__ int32_t s_wf[NW][7];
    __shared__ __attribute__((aligned(16))) int32_t s_grp[NW][4];  // the block's groups: first wave, end wave, rows, item
    __shared__ int32_t s_ngrp;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    // Wave w runs on SIMD w mod 4, and of the two waves of a SIMD the older (w < 4) runs ahead.
    // When an eight-wave prefill block takes two units (prefill_groups 2), the waves are numbered
    // so that both units' groups hold two older waves at positions 0-1 and two younger ones at
    // positions 2-3 (group 0: waves 0, 1, 6, 7; group 1: 2, 3, 4, 5): a prefix slice is then read
    // by waves of the same age in both groups, so the units stay together on the prefix and share
    // its tiles through L2 (with one group of older and one of younger waves, the younger group
    // fell behind and a quarter of the prefix was fetched from HBM twice).
    const int hw_wave = tid >> 6;
    const int wave = __builtin_amdgcn_readfirstlane(
        (PREFILL && NW == 8 && a.prefill_groups == 2) ? (hw_wave < 2 ? hw_wave : hw_wave < 6 ? hw_wave + 2 : hw_wave - 4)
                                                      : hw_wave);  // uniform per wave
    const int l16 = lane & 15, q4 = lane >> 4;
    const int G = a.group, Hkv = a.n_kv_heads, N = a.n_seqs;
    const int vb = (int)blockIdx.x;
    const int NV = (int)gridDim.x * NW;
    const int w_lo = vb * NW;
    const int max_len = a.max_suffix_len;
    const bool static_split = a.static_split != 0;

    // ---- this wave's item, its unit and the group (uniform)
    int item = -1, unit = 0, Wi = 1, jg0 = 0, jg1 = 0, wa = wave, we = wave + 1;
    int seq0 = 0, nseq = 0, plen = 0;
    int lraw = 0;  // static split: lane s < N loads suffix_len[s]
    if (static_split) {
        // the item and group follow from the plan; the lengths are requested now and waited for
        // only after the first prefix loads are issued
        if (lane < N) lraw = a.suffix_len[lane];
        const int w = w_lo + wave;
        item = static_item(w, NV, Hkv);
        const int ws0 = static_start(item, NV, Hkv), ws1 = static_start(item + 1, NV, Hkv);
        const int lo = max(ws0, w_lo), hi = min(ws1, w_lo + NW);
        Wi = ws1 - ws0;
        jg0 = lo - ws0;
        jg1 = hi - ws0;
        wa = lo - w_lo;
        we = hi - w_lo;
        nseq = N;
        plen = a.prefix_len;
        if (wave == 0) {  // the block's groups, in wave order (read after the combine barrier)
            const int wl = lane < NW ? lane : 0;
            const int it = static_item(w_lo + wl, NV, Hkv);
            const bool lead = lane < NW && (wl == 0 || static_item(w_lo + wl - 1, NV, Hkv) != it);
            const uint64_t m = __builtin_amdgcn_ballot_w64(lead);
            if (lead) {
                const int n = __builtin_popcountll(m & ((uint64_t(1) << wl) - 1));
                const int end = min(static_start(it + 1, NV, Hkv), w_lo + NW) - w_lo;
                s_grp[n][0] = wl;
                s_grp[n][1] = end;
                s_grp[n][2] = N * G;
                s_grp[n][3] = it;
            }
            if (lane == 0) s_ngrp = __builtin_popcountll(m);
        }
    } else {
        // one round trip: the suffix lengths and the units; then the scans and the placement
        bool clamped = false;
        for (int s = tid; s < N; s += NTH) {
            int L;
            if constexpr (PREFILL) {
                // instruction token t of branch b (s = b n + t) sees b's suffix up to its own position
                const int n = a.prefill_n;
                const int raw = a.suffix_len[s / n];
                const int Lb = min(max(raw, 0), max_len - n);
                clamped |= (Lb != raw);
                L = Lb + s % n + 1;
            } else {
                const int raw = a.suffix_len[s];
                L = min(max(raw, 0), max_len);
                clamped |= (L != raw);
            }
            s_len[s] = L;
            s_cs[s] = slices_of(L);
            if (vb == 0) a.lens[s] = L;  // what the merge appends at
        }
        const int32_t *ur = reinterpret_cast<const int32_t *>(a.units);
        for (int u = tid; u < a.n_units; u += NTH) {
            s_u0[u] = ur[4 * u + 0];
            s_un[u] = ur[4 * u + 1];
            s_ul[u] = ur[4 * u + 2];
            s_up[u] = ur[4 * u + 3];
        }
        if (vb == 0 && clamped) atomicOr(a.err, kErrSuffixClamped);
        if (tid < NW) s_wf[tid][0] = -1;  // waves the placement below does not reach have no item
        if constexpr (PREFILL) {
            // Cyclic placement over block sets: a set is P = prefill_groups units of one KV head
            // (its blocks split into P groups of NW / P waves, group j taking the set's j-th unit
            // over the same prefix range as the others, so they stream the same tiles side by
            // side); block vb is block k = vb / n_sets of set vb mod n_sets, each set having
            // B = blocks / n_sets blocks.  With n_sets a multiple of the 8 XCDs, every block of a
            // KV head runs on one XCD, so the blocks of one prefix range, one per unit, share its
            // tiles through that XCD's L2.
            const int P = a.prefill_groups, GW = NW / P;
            const int n_sets = (a.n_units + P - 1) / P * Hkv, B = (int)gridDim.x / n_sets;
            const int set = vb % n_sets, k = vb / n_sets;
            const int g = set % Hkv, us = set / Hkv;
            lds_barrier();  // the unit table
            if (tid < NW) {
                const int grp = tid / GW, u = us * P + grp;
                int32_t *d = s_wf[tid];
                d[0] = u < a.n_units ? u * Hkv + g : -1;
                d[1] = u;
                d[2] = B * GW;
                d[3] = k * GW;
                d[4] = (k + 1) * GW;
                d[5] = grp * GW;
                d[6] = grp * GW + GW;
            }
            if (k == 0) {  // the rows of item i read their B parts at slots i B .. i B + B - 1
                for (int grp = 0; grp < P; ++grp) {
                    const int u = us * P + grp, i = u * Hkv + g;
                    if (u >= a.n_units) break;
                    for (int r = tid; r < s_un[u] * G; r += NTH) {
                        int32_t *rr = a.rowrec + ((size_t)(s_u0[u] + r / G) * a.n_q_heads + g * G + r % G) * kRowRec;
                        rr[0] = i * B * a.slot_rows + r;
                        rr[1] = B;
                    }
                }
            }
        } else {
        lds_barrier();
            // exclusive scan of v[0..n) in place, total at v[n] (visible after the next barrier)
            auto block_scan = [&](int32_t *v, int n) {
                int carry = 0;
                for (int base = 0; base < n; base += NTH) {
                    const int i = base + tid;
                    const int x0 = i < n ? v[i] : 0;
                    int x = x0;
#pragma unroll
                    for (int off = 1; off < 64; off <<= 1) {
                        const int y = __shfl_up(x, off);
                        if (lane >= off) x += y;
                    }
                    if (lane == 63) s_wsum[wave] = x;
                    lds_barrier();
                    int pre = carry;
                    for (int w = 0; w < NW; ++w) {
                        if (w < wave) pre += s_wsum[w];
                        carry += s_wsum[w];
                    }
                    if (i < n) v[i] = pre + x - x0;
                    lds_barrier();
                }
                if (tid == 0) v[n] = carry;
            };
            block_scan(s_cs, N);
            lds_barrier();
            for (int u = tid; u < a.n_units; u += NTH)
                s_ne[u] = (slices_of(s_ul[u]) + s_cs[s_u0[u] + s_un[u]] - s_cs[s_u0[u]]) > 0 ? 1 : 0;
            lds_barrier();
            block_scan(s_ne, a.n_units);
            lds_barrier();
            const int T = __builtin_amdgcn_readfirstlane(Hkv * (a.ps_total + s_cs[N]));  // total slices
            const int NNE = __builtin_amdgcn_readfirstlane(Hkv * s_ne[a.n_units]);      // non-empty items
            const uint64_t R = T > 0 ? sched_ratio((int64_t)NV - NNE, T) : 0;
            const int n_items = a.n_units * Hkv;
            // every thread places its items' workers of this block; the block holding an item's
            // first worker writes the slot records of the item's rows (block 0 those of empty items)
            for (int i = tid; i < n_items; i += NTH) {
                const int u = i / Hkv, g = i - u * Hkv;
                const int u0 = s_u0[u], un = s_un[u];
                const int size = slices_of(s_ul[u]) + s_cs[u0 + un] - s_cs[u0];
                const int64_t C = (int64_t)Hkv * (s_up[u] + s_cs[u0]) + (int64_t)g * size;
                const int64_t K = (int64_t)Hkv * s_ne[u] + (size > 0 ? g : 0);
                int ws0 = 0, ws1 = 0;
                if (size > 0 && T > 0) {
                    ws0 = worker_start(C, K, R);
                    ws1 = worker_start(C + size, K + 1, R);
                }
                if ((ws1 > ws0 && ws0 >= w_lo && ws0 < w_lo + NW) || (ws1 == ws0 && vb == 0)) {
                    const int first = ws1 > ws0 ? ws0 / NW + i : 0, count = ws1 > ws0 ? (ws1 - 1) / NW - ws0 / NW + 1 : 0;
                    for (int r = 0; r < un * G; ++r) {
                        int32_t *rr = a.rowrec + ((size_t)(u0 + r / G) * a.n_q_heads + g * G + r % G) * kRowRec;
                        rr[0] = first * a.slot_rows + r;
                        rr[1] = count;
                    }
                }
                if (ws1 <= w_lo || ws0 >= w_lo + NW || ws1 <= ws0) continue;
                const int lo = max(ws0, w_lo), hi = min(ws1, w_lo + NW);
                for (int gw = lo; gw < hi; ++gw) {
                    int32_t *d = s_wf[gw - w_lo];
                    d[0] = i;
                    d[1] = u;
                    d[2] = ws1 - ws0;
                    d[3] = lo - ws0;
                    d[4] = hi - ws0;
                    d[5] = lo - w_lo;
                    d[6] = hi - w_lo;
                }
            }
        }
        lds_barrier();
        item = __builtin_amdgcn_readfirstlane(s_wf[wave][0]);
        if (item >= 0) {
            unit = __builtin_amdgcn_readfirstlane(s_wf[wave][1]);
            Wi = __builtin_amdgcn_readfirstlane(s_wf[wave][2]);
            jg0 = __builtin_amdgcn_readfirstlane(s_wf[wave][3]);
            jg1 = __builtin_amdgcn_readfirstlane(s_wf[wave][4]);
            wa = __builtin_amdgcn_readfirstlane(s_wf[wave][5]);
            we = __builtin_amdgcn_readfirstlane(s_wf[wave][6]);
            seq0 = __builtin_amdgcn_readfirstlane(s_u0[unit]);
            nseq = __builtin_amdgcn_readfirstlane(s_un[unit]);
            plen = __builtin_amdgcn_readfirstlane(s_ul[unit]);
        }
        if (wave == 0) {  // the block's groups, in wave order (read after the combine barrier)
            const int w = lane < NW ? lane : 0;  // lane w looks at wave w
            const bool lead = lane < NW && s_wf[w][0] >= 0 && s_wf[w][5] == w;
            const uint64_t m = __builtin_amdgcn_ballot_w64(lead);
            if (lead) {
                const int n = __builtin_popcountll(m & ((uint64_t(1) << w) - 1));
                s_grp[n][0] = w;
                s_grp[n][1] = s_wf[w][6];
                s_grp[n][2] = s_un[s_wf[w][1]] * G;
                s_grp[n][3] = s_wf[w][0];
            }
            if (lane == 0) s_ngrp = __builtin_popcountll(m);
        }
    }

    const int kvh = item >= 0 ? item % Hkv : 0;
    const int rows = nseq * G;
    const int nt_act = (rows + 15) >> 4;
    const int Ps = slices_of(plen);
    // the group's prefix slices [pa, pa + np) (known from the plan), its waves and this wave's
    // place among them: wave j of the group's gn waves takes list entries j, j + gn, ...
    const int pa = uni(pre_split(jg0, Wi, Ps)), np = uni(pre_split(jg1, Wi, Ps) - pa);
    const int gn = uni(we - wa), gw = uni(wave - wa);
    // suffix part (set once the lengths are known): lane i holds the clamped length of the
    // unit's sequence i and the inclusive scan of the sequences' slice counts
    int lenv = 0, csv = 0;
    int sa = 0, nlist = np;

    // The key sources, held in scalar registers: chosen from values, a branch between the
    // argument fields themselves becomes a load through a selected argument address, whose
    // wait drains every load in flight.
    const char *const arg_pk = reinterpret_cast<const char *>(a.prefix_k);
    const char *const arg_pv = reinterpret_cast<const char *>(a.prefix_v);
    const char *const arg_sk = reinterpret_cast<const char *>(a.suffix_k);
    const char *const arg_sv = reinterpret_cast<const char *>(a.suffix_v);
    const char *const arg_kp = reinterpret_cast<const char *>(a.k_pool);
    const char *const arg_vp = reinterpret_cast<const char *>(a.v_pool);
    const int32_t *const arg_pt = a.page_table;
    const int arg_plen = a.prefix_len, arg_cap = a.suffix_cap, arg_maxp = a.max_pages, arg_npool = a.n_pool_pages;
    asm volatile("" ::"s"(arg_pk), "s"(arg_pv), "s"(arg_sk), "s"(arg_sv), "s"(arg_kp), "s"(arg_vp), "s"(arg_pt),
                 "s"(arg_plen), "s"(arg_cap), "s"(arg_maxp), "s"(arg_npool));
    // Entry x of the group's list: prefix slice pa + x for x in [0, np), suffix slice sa + x - np
    // of the unit's suffix list for x in [np, nlist), nothing otherwise.  Written without
    // branches (the suffix lookup is always evaluated): the fields stay in scalar registers.
    auto locate = [&](int x) -> SliceSrc {
        const bool isp = x >= 0 && x < np;
        const bool iss = x >= np && x < nlist;
        const int k = sa + (x - np);  // slice of the unit's suffix list
        const uint64_t m = __builtin_amdgcn_ballot_w64(lane < nseq && csv > k);
        const int sr = uni(m ? __builtin_ctzll(m) : 0);
        const int L = __builtin_amdgcn_readlane(lenv, sr);
        const int c0 = __builtin_amdgcn_readlane(csv, sr) - slices_of(L);
        const int seq = seq0 + sr;
        SliceSrc s;
        s.tok0 = isp ? (pa + x) * kSlice : iss ? (k - c0) * kSlice : 0;
        s.tok_lim = isp ? plen : iss ? L : 0;
        s.r_lo = iss ? sr * G : 0;
        s.r_hi = isp ? rows : iss ? sr * G + G : 0;
        s.suffix = iss ? 1 : 0;
        if (PAGED) {
            s.kb = arg_kp;
            s.vb = arg_vp;
            // the prefill's virtual sequence reads its branch's page-table row
            const int prow = PREFILL ? (iss ? seq : seq0) / a.prefill_n : (iss ? seq : seq0);
            s.ptab = uni_ptr(arg_pt + (size_t)prow * arg_maxp);
            s.page_off = iss ? (plen + kPageSize - 1) / kPageSize : 0;
        } else {
            const size_t pbase = (size_t)kvh * (size_t)arg_plen * ROWB;
            const int buf = PREFILL ? seq / a.prefill_n : seq;  // prefill: branch b's buffer
            const size_t sbase = ((size_t)buf * Hkv + kvh) * (size_t)arg_cap * ROWB;
            s.kb = iss ? arg_sk + sbase : arg_pk + pbase;
            s.vb = iss ? arg_sv + sbase : arg_pv + pbase;
            s.ptab = arg_pt;
            s.page_off = 0;
        }
        return s;
    };

    // Buffer resource over the 16-row group holding positions [t, t + 16) of the slice's
    // segment (t is a multiple of 16, so a group never straddles a page).  Its size covers
    // only the rows below tok_lim, so loads of rows past the end (or of a group wholly past it,
    // or behind an out-of-range page id) return zeros.  Uniform.
    bool bad_page = false;
    auto group_rsrc = [&](const SliceSrc &s, const char *src, int t) -> __amdgpu_buffer_rsrc_t {
        int rows_ok = max(0, min(kPageSize, s.tok_lim - t));
        const char *base = src;
        if (!PAGED) {
            base = src + (size_t)t * ROWB;
        } else {
            // the table entry is read even for a group with no rows (its index is clamped into
            // the row), so that no branch depends on it
            const int32_t page = scalar_load(uni_ptr(s.ptab + uni(min(s.page_off + t / kPageSize, arg_maxp - 1))));
            const bool bad = rows_ok > 0 && (page < 0 || page >= arg_npool);
            bad_page |= bad;
            rows_ok = bad ? 0 : rows_ok;
            base = rows_ok > 0 ? src + ((size_t)page * Hkv + kvh) * (kPageSize * ROWB) : src;
        }
        return make_rsrc(base, rows_ok * ROWB);
    };

    // K slice into registers (the A operand of S^T): lane holds slice token 16u + l16,
    // bytes 16*q4 + 64c of its row, i.e. d = 32c + 8*q4 .. +7, the k-slots of q below.
    const uint32_t koff = l16 * ROWB + 16 * q4;
    auto load_k = [&](const SliceSrc &s, bf16x8 (&kr)[2][NC]) {
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            const __amdgpu_buffer_rsrc_t r = group_rsrc(s, s.kb, s.tok0 + 16 * u);
#pragma unroll
            for (int c = 0; c < NC; ++c)
                kr[u][c] = __builtin_bit_cast(bf16x8, __builtin_amdgcn_raw_buffer_load_b128(r, koff + 64 * c, 0, k_policy<PAGED, PREFILL>()));
        }
    };

    // V slice -> ring stage ST by LDS DMA.  Instruction i moves 1 KiB: slice tokens
    // T = (64i + lane) / CPR (within one 16-row group), chunk ((64i + lane) % CPR) ^ swz(T),
    // where swz(T) = 2T mod CPR spreads a column read by ds_read_b64_tr_b16 over all banks.
    // Its byte offset in the group is a per-lane base that depends only on the parity of i
    // (swz) plus 1024 * (i mod VPER), which goes into the instruction's immediate offset.  The
    // hardware adds that immediate to the LDS address as well, so the LDS pointer passed is
    // lowered by the same amount.
    static_assert(CPR == 16 || CPR == 8, "V layout");
    constexpr int VPER = CPR == 16 ? 4 : 2;  // instructions per 16 rows
    uint32_t vbase[2];
#pragma unroll
    for (int par = 0; par < 2; ++par) {
        const int p = 64 * par + lane;
        const int T = p / CPR, sl = p % CPR;
        vbase[par] = (T % kPageSize) * ROWB + 16 * (sl ^ ((2 * T) & (CPR - 1))) - 1024 * (par % VPER);
    }
    auto issue_v = [&](const SliceSrc &s, auto ST) {
        constexpr int st = decltype(ST)::value;
        lds_void *dst = (lds_void *)&vring[wave][st][0];
        const __amdgpu_buffer_rsrc_t r0 = group_rsrc(s, s.vb, s.tok0), r1 = group_rsrc(s, s.vb, s.tok0 + 16);
        static_for<VDMA>([&](auto I) {
            constexpr int i = decltype(I)::value;
            constexpr int imm = 1024 * (i % VPER);
            buffer_to_lds16<v_policy<PREFILL>(), imm>(i < VPER ? r0 : r1,
                                           (lds_void *)((__attribute__((address_space(3))) char *)dst + 1024 * i - imm),
                                           vbase[CPR == 16 ? (i & 1) : 0]);
        });
    };

    // query rows (B operand of S^T = K Q^T): lane holds row 16t + l16, d = 32c + 8*q4 .. +7
    bf16x8 qb[NT][NC];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        const int r = 16 * t + l16;
#pragma unroll
        for (int c = 0; c < NC; ++c) qb[t][c] = bf16x8{};
        if (item >= 0 && r < rows) {
            const int seq = seq0 + r / G, h = kvh * G + r % G;
            const uint16_t *qp = a.q + ((size_t)seq * a.n_q_heads + h) * HD + 8 * q4;
#pragma unroll
            for (int c = 0; c < NC; ++c) qb[t][c] = *reinterpret_cast<const bf16x8 *>(qp + 32 * c);
        }
    }

    // The first slice of this wave, issued before the lengths are waited for when it is a
    // prefix slice (always so for a static split unless the group has fewer prefix slices than
    // waves).  A wave whose first slice needs the lengths issues an empty slice here instead
    // and starts its loop one entry earlier, so the loads in flight at the loop are the same
    // on every path.
    bf16x8 kbuf[kStages][2][NC];
    const bool early = gw < np;
    SliceSrc sc = locate(early ? gw : -1);
    if (item >= 0) {
        issue_v(sc, std::integral_constant<int, 0>{});
        load_k(sc, kbuf[0]);
    }

    // ---- the suffix part of the schedule
    if (static_split) {
        const int L = min(max(lraw, 0), max_len);
        if (vb == 0 && wave == 0) {
            if (lane < N) a.lens[lane] = L;  // what the merge appends at
            if (__builtin_amdgcn_ballot_w64(lane < N && L != lraw) != 0 && lane == 0) atomicOr(a.err, kErrSuffixClamped);
        }
        lenv = lane < N ? L : 0;
    } else if (item >= 0) {
        lenv = lane < nseq ? s_len[seq0 + lane] : 0;
    }
    {
        int x = slices_of(lenv);
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const int y = __shfl_up(x, off);
            if (lane >= off) x += y;
        }
        csv = x;
    }
    if (item >= 0) {
        const int S = __builtin_amdgcn_readlane(csv, 63);
        sa = uni(suf_split(jg0, Wi, Ps, S));
        nlist = uni(np + suf_split(jg1, Wi, Ps, S) - sa);
    }
    // the query rows have arrived when only the first slice's loads are in flight (stated here,
    // so the loop does not wait for everything on its first entry)
    wait_vm<2 * KLOADS>();

    // LDS byte addresses, relative to the wave's ring, of the transposed V reads: for d-tile
    // e and token half h, lane (q4, 4j + m) reads slice token T = 16h + 4*q4 + j, d = 16e + 4m.
    // The half h = 1 is 16 rows further (4096 bytes for d = 128) with the same swizzle, so it
    // goes into the instruction's offset.
    const uint32_t ring0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char *)&vring[wave][0][0];
    uint32_t traddr[NE];
    {
        const int jt = l16 >> 2, m4 = l16 & 3;
        const int T = 4 * q4 + jt;
#pragma unroll
        for (int e = 0; e < NE; ++e) {
            const int slot = (2 * e + (m4 >> 1)) ^ ((2 * T) & (CPR - 1));
            traddr[e] = ring0 + T * CPR * 16 + slot * 16 + (m4 & 1) * 8;
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

    auto compute = [&](const SliceSrc &src, const bf16x8 (&kr)[2][NC], auto ST) {
        constexpr int st = decltype(ST)::value;
        const int valid = src.tok_lim - src.tok0;  // keys of this slice in range (may exceed 32)
        const bool full = valid >= kSlice;
        const bool suf = src.suffix != 0;
        // a suffix slice: its rows' tiles only, and within them its rows only
        const int t_lo = src.r_lo >> 4, t_hi = suf ? ((src.r_hi - 1) >> 4) : NT - 1;
        // whether this lane's row of tile t reads the slice
        auto row_ok = [&](int t) { return (uint32_t)(16 * t + l16 - src.r_lo) < (uint32_t)(src.r_hi - src.r_lo); };
        bf16x8 ph[NT], pl[NT];
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            ph[t] = bf16x8{};
            pl[t] = bf16x8{};
            if (t >= nt_act || t < t_lo || t > t_hi) continue;
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
                // keys left from this lane's first token (the lane's offset recomputed here: a
                // value kept for this rare path would be spilled)
                const int v4 = valid - 4 * (opaque_lane_id() >> 4);
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    x[j] = (j < v4) ? x[j] : -INFINITY;
                    x[4 + j] = (16 + j < v4) ? x[4 + j] : -INFINITY;
                }
            }
            if (suf) {
                const bool ok = row_ok(t);
#pragma unroll
                for (int j = 0; j < 8; ++j) x[j] = ok ? x[j] : -INFINITY;
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
        // V^T operands, read after the softmax so that they are not live with its temporaries:
        // the transposed read hands lane l16 column d = 16e + l16 of four slice tokens
        vtr_t vr[NE][2];
#pragma unroll
        for (int e = 0; e < NE; ++e) {
            vr[e][0] = ds_read_tr16<st * SLICE_CHUNKS * 16>(traddr[e]);
            vr[e][1] = ds_read_tr16<st * SLICE_CHUNKS * 16 + 16 * CPR * 16>(traddr[e]);
        }
        lds_wait_all(vr);
        if (suf) {
            // The other rows of the tiles multiply this slice's values by p = 0, and 0 times a
            // non-finite value is NaN.  So a non-finite value of this sequence's suffix is
            // replaced by 0 for the product and this sequence's rows are made NaN instead
            // (through their running sums).  A bf16 half is non-finite when its exponent bits
            // are all ones: adding 0x80 to them then carries into the half's top bit.
            uint32_t bits = 0;
#pragma unroll
            for (int e = 0; e < NE; ++e)
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const uint64_t w = (uint64_t)vr[e][h];
                    bits |= (((uint32_t)w & 0x7f807f80u) + 0x00800080u) | ((((uint32_t)(w >> 32)) & 0x7f807f80u) + 0x00800080u);
                }
            if (__builtin_expect(__builtin_amdgcn_ballot_w64((bits & 0x80008000u) != 0) != 0, 0)) {
#pragma unroll
                for (int e = 0; e < NE; ++e)
#pragma unroll
                    for (int h = 0; h < 2; ++h) {
                        uint64_t w = (uint64_t)vr[e][h];
                        uint32_t lo32 = (uint32_t)w, hi32 = (uint32_t)(w >> 32);
                        const uint32_t ml = ((lo32 & 0x7f807f80u) + 0x00800080u) & 0x80008000u;
                        const uint32_t mh = ((hi32 & 0x7f807f80u) + 0x00800080u) & 0x80008000u;
                        lo32 &= ~((ml >> 15) * 0xffffu);
                        hi32 &= ~((mh >> 15) * 0xffffu);
                        vr[e][h] = (vtr_t)(((uint64_t)hi32 << 32) | lo32);
                    }
#pragma unroll
                for (int t = 0; t < NT; ++t)
                    if (t < nt_act && t >= t_lo && t <= t_hi) l_run[t] = row_ok(t) ? __builtin_nanf("") : l_run[t];
            }
        }
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            if (t >= nt_act) break;
            if (t < t_lo || t > t_hi) continue;
#pragma unroll
            for (int e = 0; e < NE; ++e) {
                const bf16x8 va = join_tr16(vr[e][0], vr[e][1]);
                acc[t][e] = mfma16(va, ph[t], acc[t][e]);
                acc[t][e] = mfma16(va, pl[t], acc[t][e]);
            }
        }
    };

    // Pipeline, one slice ahead: slice xc sits in V ring stage 0 / K registers 0 while the
    // next one loads into stage 1, then the roles swap.  Loads are issued at every step
    // (entries past the list's end have empty buffer resources and move no data), so the
    // wait count is fixed: V(x), K(x) precede the two loads of the slice behind them.  The
    // loop is tested at the top (a test in the middle costs the allocator registers).
    if (item >= 0) {
        int xc = uni(early ? gw : gw - gn);
        while (xc < nlist) {
            const int xn = uni(xc + gn);
            const SliceSrc sn = locate(xn);
            issue_v(sn, std::integral_constant<int, 1>{});
            load_k(sn, kbuf[1]);
            wait_vm<2 * KLOADS>();
            compute(sc, kbuf[0], std::integral_constant<int, 0>{});
            xc = uni(xn + gn);
            sc = locate(xc);
            issue_v(sc, std::integral_constant<int, 0>{});
            load_k(sc, kbuf[0]);
            wait_vm<2 * KLOADS>();
            if (xn < nlist)
                compute(sn, kbuf[1], std::integral_constant<int, 1>{});
            else
                xc = nlist;
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
    // Staging: wave w writes [tile][row][d] of its own accumulator (the 16-byte chunks of row r
    // XOR-permuted by r mod 16, so that one chunk of 16 consecutive rows lies in 16 different
    // bank groups: a staging store covers 16 rows at one chunk, and so does a combine load, whose
    // consecutive lanes take consecutive rows): tiles 0 and 1 into its ring, further tiles
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
        return r * HD + 4 * (c4 ^ (r & 15));
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
            // the group's slot: vb + it, or under the cyclic placement it B + (vb / n_sets)
            const int n_sets_c = (a.n_units + a.prefill_groups - 1) / a.prefill_groups * Hkv;
            const int slot_c = PREFILL ? it * ((int)gridDim.x / n_sets_c) + vb / n_sets_c : vb + it;
            if (slot_c >= a.n_slots || it < 0) continue;  // never store outside the workspace
            const int r0 = 16 * TPP * pass, r1 = min(gi.z, r0 + 16 * TPP);
            const bool whole = lw == 0 && ge == NW;  // the usual case: one group, all waves
            for (int u = tid_c; u < (r1 - r0) * CHU; u += NTH) {
                const int row = r0 + u % (r1 - r0), cu = u / (r1 - r0);
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
                const size_t so = (size_t)slot_c * a.slot_rows + row;
                float *dst = a.part_o + so * HD + 4 * UQ * cu;
#pragma unroll
                for (int q = 0; q < UQ; ++q) *reinterpret_cast<f32x4 *>(dst + 4 * q) = o[q] * inv;
                if (cu == 0) a.part_lse[so] = (L == 0.f) ? -INFINITY : (((M == -INFINITY) ? 0.f : M) + log2f(L)) * kLn2;
            }
        }
    }
    if (bad_page) atomicOr(a.err, kErrBadPage);
}

template <int HD, bool PAGED, bool PREFILL>
int blocks_per_cu_hd(int row_tiles)
{
    const void *f = nullptr;
    int threads = 0;
    switch (row_tiles) {
    case 1: f = reinterpret_cast<const void *>(&partials_kernel<HD, 1, PAGED, PREFILL>); threads = 256 * waves_per_simd<HD, 1, PAGED, PREFILL>(); break;
    case 2: f = reinterpret_cast<const void *>(&partials_kernel<HD, 2, PAGED, PREFILL>); threads = 256 * waves_per_simd<HD, 2, PAGED, PREFILL>(); break;
    case 3: f = reinterpret_cast<const void *>(&partials_kernel<HD, 3, PAGED, PREFILL>); threads = 256 * waves_per_simd<HD, 3, PAGED, PREFILL>(); break;
    case 4: f = reinterpret_cast<const void *>(&partials_kernel<HD, 4, PAGED, PREFILL>); threads = 256 * waves_per_simd<HD, 4, PAGED, PREFILL>(); break;
    default: return 0;
    }
    int n = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, f, threads, 0) != hipSuccess) return 0;
    return n;
}

template <int HD, bool PAGED, bool PREFILL>
hipError_t launch_hd(const AttnArgs &a, int n_blocks, int row_tiles, hipStream_t s)
{
    const dim3 grid(n_blocks);
    switch (row_tiles) {
    case 1: partials_kernel<HD, 1, PAGED, PREFILL><<<grid, 256 * waves_per_simd<HD, 1, PAGED, PREFILL>(), 0, s>>>(a); break;
    case 2: partials_kernel<HD, 2, PAGED, PREFILL><<<grid, 256 * waves_per_simd<HD, 2, PAGED, PREFILL>(), 0, s>>>(a); break;
    case 3: partials_kernel<HD, 3, PAGED, PREFILL><<<grid, 256 * waves_per_simd<HD, 3, PAGED, PREFILL>(), 0, s>>>(a); break;
    case 4: partials_kernel<HD, 4, PAGED, PREFILL><<<grid, 256 * waves_per_simd<HD, 4, PAGED, PREFILL>(), 0, s>>>(a); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace

int partials_blocks_per_cu(int head_dim, int row_tiles, bool paged)
{
    if (head_dim == 128)
        return paged ? blocks_per_cu_hd<128, true, false>(row_tiles) : blocks_per_cu_hd<128, false, false>(row_tiles);
    if (head_dim == 64)
        return paged ? blocks_per_cu_hd<64, true, false>(row_tiles) : blocks_per_cu_hd<64, false, false>(row_tiles);
    return 0;
}

template <bool PAGED, bool PREFILL>
int waves_per_block_hd128(int row_tiles)
{
    switch (row_tiles) {
    case 1: return 4 * waves_per_simd<128, 1, PAGED, PREFILL>();
    case 2: return 4 * waves_per_simd<128, 2, PAGED, PREFILL>();
    case 3: return 4 * waves_per_simd<128, 3, PAGED, PREFILL>();
    case 4: return 4 * waves_per_simd<128, 4, PAGED, PREFILL>();
    default: return 0;
    }
}

int partials_waves_per_block(int head_dim, int row_tiles, bool paged)
{
    if (head_dim == 64) return 4 * waves_per_simd<64, 1, false, false>();
    return paged ? waves_per_block_hd128<true, false>(row_tiles) : waves_per_block_hd128<false, false>(row_tiles);
}

int prefill_max_rows(int head_dim, int group)
{
    // two 16-row tiles per wave where a unit of them holds at least one token (two waves per SIMD)
    return (head_dim == 128 && group <= 32) ? 32 : kMaxRows;
}

int prefill_waves_per_block(int head_dim, int row_tiles, bool paged)
{
    if (head_dim == 64) return 4 * waves_per_simd<64, 1, false, true>();
    return paged ? waves_per_block_hd128<true, true>(row_tiles) : waves_per_block_hd128<false, true>(row_tiles);
}

hipError_t launch_partials(const AttnArgs &a, int n_blocks, int head_dim, int row_tiles, hipStream_t s)
{
    if (n_blocks <= 0) return hipSuccess;
    if (head_dim == 128) return a.paged ? launch_hd<128, true, false>(a, n_blocks, row_tiles, s)
                                        : launch_hd<128, false, false>(a, n_blocks, row_tiles, s);
    if (head_dim == 64) return a.paged ? launch_hd<64, true, false>(a, n_blocks, row_tiles, s)
                                       : launch_hd<64, false, false>(a, n_blocks, row_tiles, s);
    return hipErrorInvalidValue;
}

int prefill_blocks_per_cu(int head_dim, int row_tiles, bool paged)
{
    if (head_dim == 128)
        return paged ? blocks_per_cu_hd<128, true, true>(row_tiles) : blocks_per_cu_hd<128, false, true>(row_tiles);
    if (head_dim == 64)
        return paged ? blocks_per_cu_hd<64, true, true>(row_tiles) : blocks_per_cu_hd<64, false, true>(row_tiles);
    return 0;
}

hipError_t launch_prefill(const AttnArgs &a, int n_blocks, int head_dim, int row_tiles, hipStream_t s)
{
    if (n_blocks <= 0) return hipSuccess;
    if (head_dim == 128) return a.paged ? launch_hd<128, true, true>(a, n_blocks, row_tiles, s)
                                        : launch_hd<128, false, true>(a, n_blocks, row_tiles, s);
    if (head_dim == 64) return a.paged ? launch_hd<64, true, true>(a, n_blocks, row_tiles, s)
                                       : launch_hd<64, false, true>(a, n_blocks, row_tiles, s);
    return hipErrorInvalidValue;
}

}  // namespace fka
