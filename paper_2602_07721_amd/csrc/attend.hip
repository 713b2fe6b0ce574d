// Attention over the selected keys only (Sec. "Background and Problem
// Formulation", Eqs. approx_weight and approx_output; Sec. "On-Demand UVA
// Fetch": only the top-k K/V rows are read, from HBM or, through a device
// pointer to pinned host memory, straight over the host link).
//
//   o = sum_{i in idx} softmax_i(scale <k_i, q>) v_i,  fp16 in, fp32 math.
//
// One block per query head, 16 waves.  A wave works on 4 keys at a time, 16
// lanes per key: lane l16 owns dims [8 l16, 8 l16 + 8), so each K or V row is
// one 256-byte contiguous read by 16 lanes.  Indices outside
// [0, kv_capacity) are skipped like -1.  Every one of the 64 key slots keeps
// an online-softmax state (running max, sum, 8 accumulators per lane); the
// states are merged in LDS at the end.  The row's indices are staged in LDS
// first and every lane keeps 8 K and 8 V row segments in flight.

#include <hip/hip_fp16.h>

#include "internal.hpp"

namespace pariskv {

namespace {

constexpr int kAtThreads = 1024;
constexpr int kAtGroups = kAtThreads / 16;  // concurrent key slots per block
constexpr int kAtUnroll = 8;                // K/V rows in flight per lane
constexpr int kAtMaxK = 4096;               // largest k a block stages in LDS

__device__ __forceinline__ void unpack8(const uint4 v, float* f) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int h = 0; h < 4; ++h) {
        f[2 * h] = __half2float(__ushort_as_half((unsigned short)(w[h] & 0xffffu)));
        f[2 * h + 1] = __half2float(__ushort_as_half((unsigned short)(w[h] >> 16)));
    }
}

__global__ __launch_bounds__(kAtThreads) void attend_kernel(const __half* __restrict__ q,
                                                            const __half* __restrict__ K,
                                                            const __half* __restrict__ V,
                                                            int64_t kv_capacity,
                                                            const int32_t* __restrict__ idx,
                                                            int32_t k, int32_t hkv, int32_t g,
                                                            int32_t hq, float scale,
                                                            float* __restrict__ out) {
    __shared__ float s_m[kAtGroups], s_l[kAtGroups];
    __shared__ float s_acc[kAtGroups][kD];
    __shared__ int32_t s_idx[kAtMaxK];

    const int tid = threadIdx.x;
    const int grp16 = tid >> 4;      // key slot 0 .. kAtGroups-1
    const int l16 = tid & 15;
    const int64_t row = blockIdx.x;  // seq * hq + head
    const int seq = (int)(row / hq);
    const int h = (int)(row % hq);
    const int64_t kvrow0 = ((int64_t)seq * hkv + h / g) * kv_capacity;

    // Stage the row's indices (invalid ones as -1) so the row loads never wait on them.
    const int32_t* ir = idx + row * k;
    for (int r = tid; r < k; r += kAtThreads) {
        const int32_t key = ir[r];
        s_idx[r] = (key >= 0 && key < kv_capacity) ? key : -1;
    }

    float qf[8];
    unpack8(reinterpret_cast<const uint4*>(q + row * kD)[l16], qf);
#pragma unroll
    for (int d = 0; d < 8; ++d) qf[d] *= scale;
    __syncthreads();

    float m = -__builtin_huge_valf(), lsum = 0.f;
    float acc[8];
#pragma unroll
    for (int d = 0; d < 8; ++d) acc[d] = 0.f;

    // Slot grp16 takes keys grp16, grp16 + kAtGroups, ...; kAtUnroll rows in flight per lane.
    for (int base = 0; base < k; base += kAtGroups * kAtUnroll) {
        int32_t key[kAtUnroll];
        uint4 kc[kAtUnroll], vc[kAtUnroll];
#pragma unroll
        for (int u = 0; u < kAtUnroll; ++u) {
            const int r = base + grp16 + kAtGroups * u;
            key[u] = r < k ? s_idx[r] : -1;
            kc[u] = make_uint4(0, 0, 0, 0);
            vc[u] = make_uint4(0, 0, 0, 0);
            if (key[u] >= 0) {
                const int64_t off = (kvrow0 + key[u]) * kD;
                kc[u] = reinterpret_cast<const uint4*>(K + off)[l16];
                vc[u] = reinterpret_cast<const uint4*>(V + off)[l16];
            }
        }
        float dot[kAtUnroll];
#pragma unroll
        for (int u = 0; u < kAtUnroll; ++u) {
            float kf[8];
            unpack8(kc[u], kf);
            float d0 = 0.f;
#pragma unroll
            for (int d = 0; d < 8; ++d) d0 += qf[d] * kf[d];
            dot[u] = d0;
        }
#pragma unroll
        for (int st = 1; st < 16; st <<= 1) {
#pragma unroll
            for (int u = 0; u < kAtUnroll; ++u) dot[u] += __shfl_xor(dot[u], st, 64);
        }
        float mn = m;
#pragma unroll
        for (int u = 0; u < kAtUnroll; ++u)
            if (key[u] >= 0) mn = fmaxf(mn, dot[u]);
        if (mn > -__builtin_huge_valf()) {
            const float corr = __expf(m - mn);
            lsum *= corr;
#pragma unroll
            for (int d = 0; d < 8; ++d) acc[d] *= corr;
#pragma unroll
            for (int u = 0; u < kAtUnroll; ++u) {
                if (key[u] >= 0) {
                    const float p = __expf(dot[u] - mn);
                    float vf[8];
                    unpack8(vc[u], vf);
                    lsum += p;
#pragma unroll
                    for (int d = 0; d < 8; ++d) acc[d] += p * vf[d];
                }
            }
            m = mn;
        }
    }

    if (l16 == 0) {
        s_m[grp16] = m;
        s_l[grp16] = lsum;
    }
#pragma unroll
    for (int d = 0; d < 8; ++d) s_acc[grp16][8 * l16 + d] = acc[d];
    __syncthreads();
    if (tid < kD) {
        float M = -__builtin_huge_valf();
#pragma unroll
        for (int j = 0; j < kAtGroups; ++j) M = fmaxf(M, s_m[j]);
        float L = 0.f, O = 0.f;
        if (M > -__builtin_huge_valf()) {
#pragma unroll
            for (int j = 0; j < kAtGroups; ++j) {
                if (s_l[j] > 0.f) {
                    const float c = __expf(s_m[j] - M);
                    L += s_l[j] * c;
                    O += s_acc[j][tid] * c;
                }
            }
        }
        out[row * kD + tid] = L > 0.f ? O / L : 0.f;
    }
}

}  // namespace

hipError_t launch_attend(const void* q, const void* K, const void* V, int64_t kv_capacity,
                         const int32_t* idx, int32_t k, int32_t batch, int32_t hkv, int32_t g,
                         float scale, float* out, hipStream_t s) {
    const int32_t hq = hkv * g;
    const ProfEvents pe = prof_begin("attend");
    hipExtLaunchKernelGGL(attend_kernel, dim3((unsigned)(batch * hq)), dim3(kAtThreads), 0, s, pe.start, pe.stop, 0,
                       static_cast<const __half*>(q), static_cast<const __half*>(K),
                       static_cast<const __half*>(V), kv_capacity, idx, k, hkv, g, hq, scale, out);
    return hipGetLastError();
}

}  // namespace pariskv
