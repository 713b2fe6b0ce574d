// Attention over the selected keys only (Sec. "Background and Problem
// Formulation", Eqs. approx_weight and approx_output; Sec. "On-Demand UVA
// Fetch": only the top-k K/V rows are read, from HBM or, through a device
// pointer to pinned host memory, straight over the host link).
//
//   o = sum_{i in idx} softmax_i(scale <k_i, q>) v_i,  fp16 in, fp32 math.
//
// One block per query head, 4 waves.  A wave works on 4 keys at a time, 16
// lanes per key: lane l16 owns dims [8 l16, 8 l16 + 8), so each K or V row is
// one 256-byte contiguous read by 16 lanes.  Indices outside
// [0, kv_capacity) are skipped like -1.  Every (wave, key slot) keeps an
// online-softmax state (running max, sum, 8 accumulators per lane); the 16
// states are merged in LDS at the end.

#include <hip/hip_fp16.h>

#include "internal.hpp"

namespace pariskv {

namespace {

constexpr int kAtThreads = 256;
constexpr int kAtGroups = kAtThreads / 16;  // concurrent key slots per block

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

    const int tid = threadIdx.x;
    const int grp16 = tid >> 4;      // key slot 0..15
    const int l16 = tid & 15;
    const int64_t row = blockIdx.x;  // seq * hq + head
    const int seq = (int)(row / hq);
    const int h = (int)(row % hq);
    const int64_t kvrow0 = ((int64_t)seq * hkv + h / g) * kv_capacity;

    float qf[8];
    unpack8(reinterpret_cast<const uint4*>(q + row * kD)[l16], qf);
#pragma unroll
    for (int d = 0; d < 8; ++d) qf[d] *= scale;

    float m = -__builtin_huge_valf(), lsum = 0.f;
    float acc[8];
#pragma unroll
    for (int d = 0; d < 8; ++d) acc[d] = 0.f;

    const int32_t* ir = idx + row * k;
    for (int base = 0; base < k; base += kAtGroups) {
        const int r = base + grp16;
        int32_t key = r < k ? ir[r] : -1;
        if (key >= kv_capacity) key = -1;  // never read outside the K/V rows
        uint4 kc = make_uint4(0, 0, 0, 0), vc = make_uint4(0, 0, 0, 0);
        if (key >= 0) {
            const int64_t off = (kvrow0 + key) * kD;
            kc = reinterpret_cast<const uint4*>(K + off)[l16];
            vc = reinterpret_cast<const uint4*>(V + off)[l16];
        }
        float kf[8], vf[8];
        unpack8(kc, kf);
        unpack8(vc, vf);
        float dot = 0.f;
#pragma unroll
        for (int d = 0; d < 8; ++d) dot += qf[d] * kf[d];
        dot += __shfl_xor(dot, 1, 64);
        dot += __shfl_xor(dot, 2, 64);
        dot += __shfl_xor(dot, 4, 64);
        dot += __shfl_xor(dot, 8, 64);
        if (key >= 0) {
            const float mn = fmaxf(m, dot);
            const float corr = __expf(m - mn);
            const float p = __expf(dot - mn);
            lsum = lsum * corr + p;
#pragma unroll
            for (int d = 0; d < 8; ++d) acc[d] = acc[d] * corr + p * vf[d];
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
    prof_begin("attend", s);
    hipLaunchKernelGGL(attend_kernel, dim3((unsigned)(batch * hq)), dim3(kAtThreads), 0, s,
                       static_cast<const __half*>(q), static_cast<const __half*>(K),
                       static_cast<const __half*>(V), kv_capacity, idx, k, hkv, g, hq, scale, out);
    prof_end(s);
    return hipGetLastError();
}

}  // namespace pariskv
