// Attention over the selected keys only (Sec. "Background and Problem
// Formulation", Eqs. approx_weight and approx_output; Sec. "On-Demand UVA
// Fetch": only the top-k K/V rows are read, from HBM or, through a device
// pointer to pinned host memory, straight over the host link).
//
//   o = sum_{i in idx} softmax_i(scale <k_i, q>) v_i,  fp16 in, fp32 math.
//
// One block of 1024 threads per query head: the row's list is staged in LDS
// -- Sink rows, then Local + Update Buffer rows, then the retrieved keys at
// their cache rows (Sec. "Buffer Update"; with an all-zero window just the
// retrieved keys) -- and the shared attention body of attend_row.hpp (64 key
// slots of 16 lanes, 8 K and 8 V row segments in flight per lane, online
// softmax merged in LDS) runs over it.  Retrieved entries that are negative or
// land outside [0, kv_capacity) are empty slots.

#include "attend_row.hpp"

namespace pariskv {

namespace {

__global__ __launch_bounds__(kAtThreads) void attend_kernel(const __half* __restrict__ q,
                                                            const __half* __restrict__ K,
                                                            const __half* __restrict__ V,
                                                            int64_t kv_capacity,
                                                            const int32_t* __restrict__ idx,
                                                            int32_t k, int32_t hkv, int32_t g,
                                                            int32_t hq, float scale,
                                                            float* __restrict__ out, AttendWindow win,
                                                            const __half* __restrict__ Kw,
                                                            const __half* __restrict__ Vw) {
    __shared__ AttendScratch s_sm;
    __shared__ int32_t s_idx[kMaxAttendRows];
    const int64_t row = blockIdx.x;  // seq * hq + head
    const int seq = (int)(row / hq);
    const int h = (int)(row % hq);
    const int64_t kvrow0 = ((int64_t)seq * hkv + h / g) * kv_capacity;
    const uint4 qv = attend_query_part(q + row * kD);
    // Stage the row's list so the row loads never wait on it (the host checked
    // that dense rows + k fit kMaxAttendRows).
    const int32_t* ir = idx + row * k;
    const int nd = (int)win.dense_rows();
    for (int r = threadIdx.x; r < nd + k; r += kAtThreads) {
        int32_t v;
        if (r < nd) {
            v = win.dense_entry(r);
        } else {
            const int32_t j = ir[r - nd];
            const int64_t cr = win.retr_begin + (int64_t)j;
            v = (j >= 0 && cr < kv_capacity) ? (int32_t)cr : -1;
        }
        s_idx[r] = v;
    }
    __syncthreads();
    const int64_t wrow0 = win.win_capacity > 0 ? ((int64_t)seq * hkv + h / g) * win.win_capacity : 0;
    attend_row(qv, K + kvrow0 * kD, V + kvrow0 * kD, kv_capacity, Kw + wrow0 * kD,
               Vw + wrow0 * kD, win.win_capacity, s_idx, nd + k, scale, out + row * kD, s_sm);
}

}  // namespace

hipError_t launch_attend(const void* q, const void* K, const void* V, int64_t kv_capacity,
                         const void* Kw, const void* Vw, const int32_t* idx, int32_t k, int32_t batch,
                         int32_t hkv, int32_t g, float scale, float* out, const AttendWindow& win,
                         hipStream_t s) {
    const int32_t hq = hkv * g;
    const ProfEvents pe = prof_begin(win.dense_rows() > 0 ? "window_attend" : "attend");
    hipExtLaunchKernelGGL(attend_kernel, dim3((unsigned)(batch * hq)), dim3(kAtThreads), 0, s, pe.start, pe.stop, 0,
                       static_cast<const __half*>(q), static_cast<const __half*>(K),
                       static_cast<const __half*>(V), kv_capacity, idx, k, hkv, g, hq, scale, out, win,
                       static_cast<const __half*>(win.win_capacity > 0 ? Kw : K),
                       static_cast<const __half*>(win.win_capacity > 0 ? Vw : V));
    return hipGetLastError();
}

}  // namespace pariskv
