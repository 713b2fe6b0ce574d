// Attention of one query head over a list of selected keys, for a block of
// 1024 threads (Eqs. approx_weight, approx_output):
//   o = sum_{i in list} softmax_i(scale <k_i, q>) v_i,  float16 in, float32 math.
// Shared by the stand-alone attention kernel and the fused top-k + attention
// kernel, so both produce the same bits.
//
// 64 key slots of 16 lanes: lane l16 owns dims [8 l16, 8 l16 + 8), so a K or
// V row is one 256-byte contiguous read by 16 lanes.  Slot s takes list
// entries s, s + 64, ...; every lane keeps 8 K and 8 V row segments in flight.
// Each slot keeps an online-softmax state (running max, sum, 8 accumulators
// per lane).  At the end the 4 slots of a wave merge by two butterfly steps
// across its rows of 16 lanes (partners lane ^ 16, then lane ^ 32), and the 16
// wave states merge through LDS, 8 threads per dimension.
//
// Rows come from one of two caches: a list entry with kWinRow set names row
// (entry - kWinRow) of the window cache (Kw, Vw, win_capacity: Sink and Local /
// Update Buffer kept on the GPU), any other entry >= 0 a row of the main cache
// (K, V, kv_capacity: the retrieval rows, in HBM or in host memory).  Entries
// past their cache's capacity, and negative entries (-1 padding), are skipped.
//
// A caller that already holds some rows in LDS passes prow (LDS rows of 32
// uint4: K then V) and lists such a row as entry -2 - (LDS row); it is read from
// LDS, the same bytes in the same order, so the result does not depend on which
// rows were held.  Without prow every negative entry is skipped.
#pragma once

#include <hip/hip_fp16.h>

#include "internal.hpp"

namespace pariskv {

constexpr int kAtThreads = 1024;
constexpr int kAtGroups = kAtThreads / 16;  // concurrent key slots per block
constexpr int kAtWaves = kAtThreads / 64;   // slot states left after the in-wave merge
constexpr int kAtUnroll = 8;                // K/V rows in flight per lane

// LDS the row needs beyond the key list: running max, sum and accumulators per wave.
struct AttendScratch {
    float m[kAtWaves];
    float l[kAtWaves];
    float acc[kAtWaves][kD];
};

__device__ __forceinline__ void unpack8_half(const uint4 v, float* f) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int h = 0; h < 4; ++h) {
        f[2 * h] = __half2float(__ushort_as_half((unsigned short)(w[h] & 0xffffu)));
        f[2 * h + 1] = __half2float(__ushort_as_half((unsigned short)(w[h] >> 16)));
    }
}

// Sum of x over the 16 lanes of each row of the wave, in every lane, through
// DPP adds (no LDS): partners lane ^ 1 and lane ^ 2 (quad_perm), then the
// mirrored lane in the half row and in the row.  After the quad steps the lanes
// of a quad hold equal values, so the mirror partners add the same values as
// partners lane ^ 4 and lane ^ 8 would: the xor butterfly's result, bit for bit.
__device__ __forceinline__ float sum16(float x) {
    x += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0xB1, 0xF, 0xF, false));   // quad_perm 1,0,3,2
    x += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x4E, 0xF, 0xF, false));   // quad_perm 2,3,0,1
    x += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x141, 0xF, 0xF, false));  // row_half_mirror
    x += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x140, 0xF, 0xF, false));  // row_mirror
    return x;
}

// The 16 bytes of the head's float16 query that thread `tid` uses: dims
// [8 (tid & 15), 8 (tid & 15) + 8).  Callers load it first, so its latency
// overlaps their own work.
__device__ __forceinline__ uint4 attend_query_part(const __half* q_row) {
    return reinterpret_cast<const uint4*>(q_row)[threadIdx.x & 15];
}

// qv: this thread's query part (attend_query_part); K, V: the KV head's rows
// [kv_capacity][D]; Kw, Vw: its window-cache rows [win_capacity][D] (entries
// with kWinRow); list: k entries in LDS (already synchronised); out: D floats.
// Every thread of the block must call it; it ends with the block synchronised.
__device__ __forceinline__ void attend_row(uint4 qv, const __half* __restrict__ K,
                                           const __half* __restrict__ V, int64_t kv_capacity,
                                           const __half* __restrict__ Kw, const __half* __restrict__ Vw,
                                           int64_t win_capacity, const int32_t* list, int32_t k,
                                           float scale, float* __restrict__ out, AttendScratch& sm,
                                           const uint4* prow = nullptr) {
    const int tid = threadIdx.x;
    const int grp16 = tid >> 4;  // key slot 0 .. kAtGroups-1
    const int l16 = tid & 15;

    float qf[8];
    unpack8_half(qv, qf);
#pragma unroll
    for (int d = 0; d < 8; ++d) qf[d] *= scale;

    float m = -__builtin_huge_valf(), lsum = 0.f;
    float acc[8];
#pragma unroll
    for (int d = 0; d < 8; ++d) acc[d] = 0.f;

    for (int base = 0; base < k; base += kAtGroups * kAtUnroll) {
        int32_t key[kAtUnroll];
        uint4 kc[kAtUnroll], vc[kAtUnroll];
#pragma unroll
        for (int u = 0; u < kAtUnroll; ++u) {
            const int r = base + grp16 + kAtGroups * u;
            key[u] = r < k ? list[r] : -1;
            const bool win = key[u] >= kWinRow;
            const int64_t rowi = win ? key[u] - kWinRow : key[u];
            if (rowi >= (win ? win_capacity : kv_capacity)) key[u] = -1;
            kc[u] = make_uint4(0, 0, 0, 0);
            vc[u] = make_uint4(0, 0, 0, 0);
            // A held row (entry <= -2 with prow) is read from LDS where it is used.
            if (prow == nullptr && key[u] < 0) key[u] = -1;
            if (key[u] >= 0) {
                const int64_t off = rowi * kD;
                kc[u] = reinterpret_cast<const uint4*>((win ? Kw : K) + off)[l16];
                vc[u] = reinterpret_cast<const uint4*>((win ? Vw : V) + off)[l16];
            }
        }
        float dot[kAtUnroll];
#pragma unroll
        for (int u = 0; u < kAtUnroll; ++u) {
            if (prow != nullptr && key[u] <= -2) {
                kc[u] = prow[32 * (-2 - key[u]) + l16];
                vc[u] = prow[32 * (-2 - key[u]) + 16 + l16];
            }
            float kf[8];
            unpack8_half(kc[u], kf);
            float d0 = 0.f;
#pragma unroll
            for (int d = 0; d < 8; ++d) d0 += qf[d] * kf[d];
            dot[u] = d0;
        }
#pragma unroll
        for (int u = 0; u < kAtUnroll; ++u) dot[u] = sum16(dot[u]);
        float mn = m;
#pragma unroll
        for (int u = 0; u < kAtUnroll; ++u)
            if (key[u] != -1) mn = fmaxf(mn, dot[u]);
        if (mn > -__builtin_huge_valf()) {
            const float corr = __expf(m - mn);
            lsum *= corr;
#pragma unroll
            for (int d = 0; d < 8; ++d) acc[d] *= corr;
#pragma unroll
            for (int u = 0; u < kAtUnroll; ++u) {
                if (key[u] != -1) {
                    const float p = __expf(dot[u] - mn);
                    float vf[8];
                    unpack8_half(vc[u], vf);
                    lsum += p;
#pragma unroll
                    for (int d = 0; d < 8; ++d) acc[d] += p * vf[d];
                }
            }
            m = mn;
        }
    }

    // The wave's 4 slot states (rows of 16 lanes holding the same dims) into one.
    const int lane = tid & 63;
#pragma unroll
    for (int step = 16; step <= 32; step <<= 1) {
        const float mp = __uint_as_float(lane_xor(__float_as_uint(m), step, lane));
        const float lp = __uint_as_float(lane_xor(__float_as_uint(lsum), step, lane));
        float ap[8];
#pragma unroll
        for (int d = 0; d < 8; ++d) ap[d] = __uint_as_float(lane_xor(__float_as_uint(acc[d]), step, lane));
        const float mn = fmaxf(m, mp);
        if (mn > -__builtin_huge_valf()) {
            const float c0 = __expf(m - mn), c1 = __expf(mp - mn);
            lsum = lsum * c0 + lp * c1;
#pragma unroll
            for (int d = 0; d < 8; ++d) acc[d] = acc[d] * c0 + ap[d] * c1;
        }
        m = mn;
    }
    const int wave = tid >> 6;
    if (lane < 16) {
        if (l16 == 0) {
            sm.m[wave] = m;
            sm.l[wave] = lsum;
        }
#pragma unroll
        for (int d = 0; d < 8; ++d) sm.acc[wave][8 * l16 + d] = acc[d];
    }
    __syncthreads();
    {
        // Every thread: dim d of 2 of the 16 wave states, then a sum over the 8 threads
        // of the dim (lanes 8 d' + part) by lane exchanges.  An empty state (m = -inf,
        // l = 0, acc = 0) is scaled by exp(-inf) = 0, so it needs no test.
        static_assert(kAtThreads == 8 * kD && kAtWaves == 16, "8 threads per dim, 2 states each");
        const int d = tid >> 3, part = tid & 7;
        float M = -__builtin_huge_valf();
#pragma unroll
        for (int j = 0; j < kAtWaves; ++j) M = fmaxf(M, sm.m[j]);
        float L = 0.f, O = 0.f;
        if (M > -__builtin_huge_valf()) {
#pragma unroll
            for (int r = 0; r < 2; ++r) {
                const int j = 2 * part + r;
                const float c = __expf(sm.m[j] - M);
                L += sm.l[j] * c;
                O += sm.acc[j][d] * c;
            }
        }
#pragma unroll
        for (int x = 1; x < 8; x <<= 1) {
            L += __uint_as_float(lane_xor(__float_as_uint(L), x, lane));
            O += __uint_as_float(lane_xor(__float_as_uint(O), x, lane));
        }
        if (part == 0) out[d] = L > 0.f ? O / L : 0.f;
    }
    __syncthreads();
}

}  // namespace pariskv
