// Key summarisation kernel: centroid ids, 4-bit direction codes, weights W
// and cluster counts (Sec. "Prefill Phase" steps (1)-(3), Eqs. dir_assign,
// rsqip_sign_mag_code, alpha_def, scaling_factor; Alg. 1 encode loop).
//
// Arithmetic (bit-exact by construction):
//   y = H (s (.) k) in float64.  float16 inputs are integer multiples of 2^-24
//   below 2^16, so every partial sum of at most 128 of them is an integer
//   multiple of 2^-24 below 2^47 and is exact in float64 in any order.  y is
//   sqrt(D) ||k|| times the rotated, normalised key, a positive factor that
//   every decision below is invariant to.
//   id bit j    = [y_j < 0]                      (argmax over {+-1/sqrt m}^m),
//                 stored as id_slot(id); counts are kept by the id itself
//   Y_j         = fl(y_j * y_j)
//   S_b         = ((Y0+Y1)+(Y2+Y3))+((Y4+Y5)+(Y6+Y7))
//   t_j         = #{t : Y_j >= fl(tau_t^2 * S_b)}   (|u_j| >= tau_t), 0 if S_b = 0
//   A_b         = same tree over fl(a[t_j] * |y_j|) (= sqrt(S_b) alpha_b)
//   W_b         = float(fl(S_b / A_b))              (= sqrt(D) w_b), 0 if S_b = 0
// Every float64 operation is an explicit round-to-nearest multiply or add
// (no contraction), so the results do not depend on the compiler.
//
// Mapping: 4 lanes per key; lane q holds coordinates [32q, 32q+32), i.e.
// subspaces 4q..4q+3.  Butterfly strides 1..16 are in registers, 32 and 64
// cross lanes (partners q^1, q^2).  Each lane then writes its 4 id bytes and
// the two 16-byte record chunks 2q and 2q+1.  Cluster counts are gathered in
// an LDS histogram per block and added to global memory once per block.

#include <hip/hip_fp16.h>

#include "internal.hpp"

// The decision path is specified operation by operation; never fuse.
#pragma clang fp contract(off)

namespace pariskv {

namespace {

constexpr int kThreads = 256;
constexpr int kKeysPerIter = kThreads / 4;

__device__ __forceinline__ double tree8_sum(const double* v) {
    double s01 = __dadd_rn(v[0], v[1]);
    double s23 = __dadd_rn(v[2], v[3]);
    double s45 = __dadd_rn(v[4], v[5]);
    double s67 = __dadd_rn(v[6], v[7]);
    return __dadd_rn(__dadd_rn(s01, s23), __dadd_rn(s45, s67));
}

template <bool kLdsCounts>
__global__ __launch_bounds__(kThreads) void encode_kernel(
    const __half* __restrict__ keys, int64_t n_src, int64_t src_stride, int64_t keys_per_block, int64_t row0,
    int64_t capacity, uint8_t* __restrict__ ids, uint8_t* __restrict__ rec,
    uint32_t* __restrict__ counts, SignBits sb, QuantConsts qc, uint32_t flags) {
    __shared__ double s_a[8];
    __shared__ uint32_t s_cnt[kLdsCounts ? kB * kCentroids : 1];

    const int tid = threadIdx.x;
    const int q = tid & 3;
    const int slot = tid >> 2;
    const int64_t grp = blockIdx.y;
    const int64_t k_begin = (int64_t)blockIdx.x * keys_per_block;
    const int64_t k_end = min(k_begin + keys_per_block, n_src);

    if (tid < 8) s_a[tid] = qc.a[tid];
    if (kLdsCounts) {
        for (int i = tid; i < kB * kCentroids; i += kThreads) s_cnt[i] = 0;
    }
    __syncthreads();

    const uint32_t smask = sb.w[q];
    double tau2[7];
#pragma unroll
    for (int t = 0; t < 7; ++t) tau2[t] = qc.tau2[t];

    for (int64_t base = k_begin; base < k_end; base += kKeysPerIter) {
        const int64_t i = base + slot;
        const bool live = i < k_end;
        // Out-of-range lanes still join the shuffles (with zeros) and store nothing.
        double x[32];
        if (live) {
            const uint4* src = reinterpret_cast<const uint4*>(keys + ((grp * src_stride + i) * kD + 32 * q));
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                uint4 v = src[c];
                uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
                for (int h = 0; h < 4; ++h) {
                    __half lo = __ushort_as_half((unsigned short)(w[h] & 0xffffu));
                    __half hi = __ushort_as_half((unsigned short)(w[h] >> 16));
                    x[8 * c + 2 * h] = (double)__half2float(lo);
                    x[8 * c + 2 * h + 1] = (double)__half2float(hi);
                }
            }
        } else {
#pragma unroll
            for (int j = 0; j < 32; ++j) x[j] = 0.0;
        }
        if (!(flags & kFlagNoRotation)) {
#pragma unroll
            for (int j = 0; j < 32; ++j)
                if ((smask >> j) & 1u) x[j] = -x[j];

            // In-register butterflies, strides 1..16 (exact).
#pragma unroll
            for (int h = 1; h < 32; h <<= 1) {
#pragma unroll
                for (int j = 0; j < 32; ++j) {
                    if ((j & h) == 0) {
                        double a0 = x[j], a1 = x[j + h];
                        x[j] = __dadd_rn(a0, a1);
                        x[j + h] = __dsub_rn(a0, a1);
                    }
                }
            }
            // Cross-lane butterflies, strides 32 (lane q^1) and 64 (lane q^2).
#pragma unroll
            for (int m = 1; m <= 2; m <<= 1) {
                const bool upper = (q & m) != 0;
#pragma unroll
                for (int j = 0; j < 32; ++j) {
                    double p = __shfl_xor(x[j], m, 64);
                    x[j] = upper ? __dsub_rn(p, x[j]) : __dadd_rn(x[j], p);
                }
            }
        }

        uint32_t id_word = 0, slot_word = 0;  // true ids (for counts), stored slots
        uint32_t code[4];
        float wgt[4];
#pragma unroll
        for (int sbi = 0; sbi < 4; ++sbi) {
            const double* y = x + 8 * sbi;
            double Y[8], P[8];
            uint32_t idb = 0, cw = 0;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                Y[j] = __dmul_rn(y[j], y[j]);
                idb |= (y[j] < 0.0 ? 1u : 0u) << j;
            }
            const double S = tree8_sum(Y);
            double TS[7];
#pragma unroll
            for (int t = 0; t < 7; ++t) TS[t] = __dmul_rn(tau2[t], S);
            const bool nz = S > 0.0;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                uint32_t t = 0;
#pragma unroll
                for (int u = 0; u < 7; ++u) t += (Y[j] >= TS[u]) ? 1u : 0u;
                t = nz ? t : 0u;
                P[j] = __dmul_rn(s_a[t], fabs(y[j]));
                cw |= ((((idb >> j) & 1u) << 3) | t) << (4 * j);
            }
            const double A = tree8_sum(P);
            // Without the alpha-correction the weight is ||y_b|| = sqrt(S_b).
            wgt[sbi] = !nz ? 0.0f : (flags & kFlagNoAlpha) ? (float)__dsqrt_rn(S) : (float)(S / A);
            code[sbi] = cw;
            id_word |= idb << (8 * sbi);
            slot_word |= id_slot(idb) << (8 * sbi);
        }

        if (live) {
            const int64_t row = grp * capacity + row0 + i;
            *reinterpret_cast<uint32_t*>(ids + row * kB + 4 * q) = slot_word;
            uint4* dst = reinterpret_cast<uint4*>(rec + row * kRec + 32 * q);
            dst[0] = make_uint4(code[0], code[1], __float_as_uint(wgt[0]), __float_as_uint(wgt[1]));
            dst[1] = make_uint4(code[2], code[3], __float_as_uint(wgt[2]), __float_as_uint(wgt[3]));
#pragma unroll
            for (int sbi = 0; sbi < 4; ++sbi) {
                const int b = 4 * q + sbi;
                const uint32_t c = (id_word >> (8 * sbi)) & 0xffu;
                if (kLdsCounts)
                    atomicAdd(&s_cnt[b * kCentroids + c], 1u);
                else
                    atomicAdd(&counts[grp * (kB * kCentroids) + b * kCentroids + c], 1u);
            }
        }
    }

    if (kLdsCounts) {
        __syncthreads();
        for (int i = tid; i < kB * kCentroids; i += kThreads) {
            const uint32_t v = s_cnt[i];
            if (v) atomicAdd(&counts[grp * (kB * kCentroids) + i], v);
        }
    }
}

__global__ void zero_u32_kernel(uint32_t* p, int64_t count) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < count) p[i] = 0u;
}

}  // namespace

hipError_t launch_zero_u32(uint32_t* p, int64_t count, hipStream_t s) {
    if (count <= 0) return hipSuccess;
    const int64_t blocks = (count + 255) / 256;
    const ProfEvents pe = prof_begin("zero_counts");
    hipExtLaunchKernelGGL(zero_u32_kernel, dim3((unsigned)blocks), dim3(256), 0, s, pe.start, pe.stop, 0, p, count);
    return hipGetLastError();
}

hipError_t launch_encode(const void* keys, int64_t n_src, int64_t src_stride, int64_t groups,
                         int64_t row0, int64_t capacity, uint8_t* ids, uint8_t* rec,
                         uint32_t* counts, const SignBits& sb, const QuantConsts& qc, uint32_t flags,
                         hipStream_t s) {
    if (n_src <= 0 || groups <= 0) return hipSuccess;
    const __half* k = static_cast<const __half*>(keys);
    if (n_src >= 1024) {
        // Bulk: blocks of 2048 keys share one LDS histogram flush.
        const int64_t per = 2048;
        const int64_t bx = (n_src + per - 1) / per;
        const ProfEvents pe = prof_begin("encode");
        hipExtLaunchKernelGGL(encode_kernel<true>, dim3((unsigned)bx, (unsigned)groups), dim3(kThreads),
                           0, s, pe.start, pe.stop, 0, k, n_src, src_stride, per, row0, capacity, ids, rec, counts, sb, qc, flags);
    } else {
        // Streaming append: few keys per group, count straight into global memory.
        const int64_t per = kKeysPerIter;
        const int64_t bx = (n_src + per - 1) / per;
        const ProfEvents pe = prof_begin("append");
        hipExtLaunchKernelGGL(encode_kernel<false>, dim3((unsigned)bx, (unsigned)groups), dim3(kThreads),
                           0, s, pe.start, pe.stop, 0, k, n_src, src_stride, per, row0, capacity, ids, rec, counts, sb, qc, flags);
    }
    return hipGetLastError();
}

}  // namespace pariskv
