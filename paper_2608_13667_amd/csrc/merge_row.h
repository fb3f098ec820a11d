// Log-sum-exp merge of one output row from its partial results: the second stage of fork-aware
// decode attention (the merge kernel runs one block per output row).
//
// A part p of row (s, h) holds the row's attention over a disjoint set of its keys: the
// normalised output o_p and lse_p = ln(sum of exp(score)) over that set.  Their union is
//   M = max_p lse_p,  w_p = exp(lse_p - M),  o = sum_p w_p o_p / sum_p w_p,  lse = M + ln sum_p w_p.
// A part with lse = -inf holds no keys and has weight 0; if every part is empty the row has no
// keys at all and gets o = 0, lse = -inf.  A NaN part propagates.  In a fused step the token
// being appended is one more part, o = v_new, lse = scale * q . k_new, read from k_new / v_new
// (it is stored into the cache after every block of the step has read the lengths).
#pragma once

#include "internal.h"

namespace fka {

typedef float merge_f32x4 __attribute__((ext_vector_type(4)));

struct RowMerge {
    const float *part_o;    // part j of the row at part_o[(p_first + j * p_step) * HD]
    const float *part_lse;  // ... and part_lse[p_first + j * p_step]
    int64_t p_first, p_step;
    int n;                  // parts
    // fused step (the token appended this step joins as one more part): q . k_new and v_new are
    // read whenever `step` is set; the token joins the row when its sequence has room
    // (L < max_len), decided only after the parts are in, so that a length still in flight does
    // not hold them up
    int step;
    int L, max_len;
    const uint16_t *q_row;  // bf16 [HD]
    const uint16_t *k_row;  // bf16 [HD] k_new of the row's (sequence, KV head)
    const uint16_t *v_row;  // bf16 [HD]
    float scale;            // softmax scale (natural-log units)
    float *out_row;         // fp32 [HD]
    float *out_lse;         // fp32, nullable
};

// LDS the routine uses.
template <int HD>
struct MergeLds {
    static constexpr int CH = HD / 4;    // float4 chunks per row
    static constexpr int SL = 256 / CH;  // part slices: slice k takes parts k, k + SL, ...
    merge_f32x4 acc[SL][CH];
    float m[SL], w[SL];
    float lse_new;
};

// Merges row m with a block of 256 threads (every thread must call it).  Ends with a barrier, so
// the LDS can be reused at once.
template <int HD>
__device__ inline void merge_row(const RowMerge &m, MergeLds<HD> &lds)
{
    constexpr int CH = MergeLds<HD>::CH, SL = MergeLds<HD>::SL;
    constexpr float kLog2eM = 1.442695040888963407f;
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int chunk = tid % CH, slice = tid / CH;
    const __amdgpu_buffer_rsrc_t ro = __builtin_amdgcn_make_buffer_rsrc((void *)m.part_o, 0, 0x7fffffff, 0x00020000);
    const __amdgpu_buffer_rsrc_t rl = __builtin_amdgcn_make_buffer_rsrc((void *)m.part_lse, 0, 0x7fffffff, 0x00020000);

    float dot = 0.f;
    uint2 new_v = {0, 0};
    if (m.step) {
        if (slice == 0) new_v = *reinterpret_cast<const uint2 *>(m.v_row + 4 * chunk);
        if (wave == 0)
            for (int c = lane; c < HD; c += 64)
                dot += __uint_as_float((uint32_t)m.q_row[c] << 16) * __uint_as_float((uint32_t)m.k_row[c] << 16);
    }
    // online merge of this slice's parts (each part's lse and o loaded together)
    float mx = -INFINITY, w = 0.f;
    merge_f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    constexpr int U = 4;  // parts loaded ahead of their use
    {
        for (int j0 = slice; j0 < m.n; j0 += U * SL) {
            float l[U];
            merge_f32x4 o[U];
#pragma unroll
            for (int u = 0; u < U; ++u) {
                const int j = j0 + u * SL;
                l[u] = -INFINITY;
                o[u] = merge_f32x4{0.f, 0.f, 0.f, 0.f};
                if (j < m.n) {
                    const int64_t off = m.p_first + (int64_t)j * m.p_step;
                    l[u] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(rl, (uint32_t)(off * 4), 0, 0));
                    o[u] = __builtin_bit_cast(merge_f32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                                                ro, (uint32_t)((off * HD + 4 * chunk) * 4), 0, 0));
                }
            }
#pragma unroll
            for (int u = 0; u < U; ++u) {
                if (l[u] == -INFINITY) continue;
                const float mn = fmaxf(mx, l[u]);
                const float sc = (mx == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f((mx - mn) * kLog2eM);
                const float e = __builtin_amdgcn_exp2f((l[u] - mn) * kLog2eM);
                w = w * sc + e;
                acc = acc * sc + e * o[u];
                mx = mn;
            }
        }
        if (chunk == 0) {
            lds.m[slice] = mx;
            lds.w[slice] = w;
        }
        lds.acc[slice][chunk] = acc;
        if (m.step && wave == 0) {
#pragma unroll
            for (int off = 32; off >= 1; off >>= 1) dot += __shfl_xor(dot, off);
            if (lane == 0) lds.lse_new = dot * m.scale;
        }
    }
    __syncthreads();
    const bool with_new = m.step && m.L < m.max_len;
    if (slice == 0) {
        const float lse_new = with_new ? lds.lse_new : -INFINITY;
        float M = lse_new;
#pragma unroll
        for (int k = 0; k < SL; ++k) M = fmaxf(M, lds.m[k]);
        merge_f32x4 t = {0.f, 0.f, 0.f, 0.f};
        float W = 0.f;
        if (M != -INFINITY) {
#pragma unroll
            for (int k = 0; k < SL; ++k) {
                const float sc = (lds.m[k] == -INFINITY) ? 0.f : __builtin_amdgcn_exp2f((lds.m[k] - M) * kLog2eM);
                t += sc * lds.acc[k][chunk];
                W += sc * lds.w[k];
            }
            if (with_new) {
                const float e = __builtin_amdgcn_exp2f((lse_new - M) * kLog2eM);
                W += e;
                t += e * merge_f32x4{__uint_as_float(new_v.x << 16), __uint_as_float(new_v.x & 0xffff0000u),
                                     __uint_as_float(new_v.y << 16), __uint_as_float(new_v.y & 0xffff0000u)};
            }
        }
        const merge_f32x4 r = (W == 0.f) ? merge_f32x4{0.f, 0.f, 0.f, 0.f} : t * __builtin_amdgcn_rcpf(W);
        *reinterpret_cast<merge_f32x4 *>(m.out_row + 4 * chunk) = r;
        if (m.out_lse && chunk == 0) *m.out_lse = (W == 0.f) ? -INFINITY : M + logf(W);
    }
    __syncthreads();
}

}  // namespace fka
