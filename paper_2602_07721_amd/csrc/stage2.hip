// Stage II of the decode-time retrieval: RSQ-IP reranking of the candidates
// and the final top-k (Sec. "Retrieval" (2); Appendix "RSQ-IP Reranking from
// 4-Bit Key Summaries", Eqs. rsqip_raw and rsqip_raw_weighted; Alg. 1 Stage II).
//
// With z = H(s q) (so ||q|| q_tilde_b = z_b / sqrt(D)) and the stored
// W_b = sqrt(D) w_b, the estimator of <k_i, q> is
//     s_hat_i = ||q|| sum_b w_b <v_b, q_tilde_b> = sum_b W_b <v_b, z_b / D>,
// where v_b has coordinates sign * a[t] decoded from the 4-bit codes.  The
// query side z/D arrives as float from the query kernel.
//
// rerank_kernel: 8 lanes per candidate; lane l reads the 16-byte chunk l of
// the 128-byte record (codes of subspaces 2l, 2l+1 and their W), so one
// candidate is one fully used 128-byte line and a wave reads 8 lines per
// load instruction.  Lane l keeps the 16 query coordinates of its two
// subspaces in registers; the signed level table (16 floats) lives in LDS
// and is read with at most 16 distinct addresses per instruction.
//
// topk_kernel: one block per query head.  Exact radix select (8-bit digits,
// taken from the top of the occupied [min, max] key range so the histograms
// spread) of the k-th largest estimate on order-preserving uint32 keys, ties
// at the threshold taken in candidate order, then an ordered compaction: the
// winners come out in ascending key index (candidate order), no sort.

#include "internal.hpp"

namespace pariskv {

namespace {

constexpr int kRrThreads = 256;
constexpr int kRrSlots = kRrThreads / 8;    // candidates per block iteration
constexpr int kRrTile = 8 * kRrSlots;       // candidates per block

__global__ __launch_bounds__(kRrThreads) void rerank_kernel(RetrieveArgs a) {
    __shared__ float s_tab[16];
    const int tid = threadIdx.x;
    const int l = tid & 7;
    const int slot = tid >> 3;
    const int64_t row = blockIdx.y;                 // seq * hq + hq
    const int seq = (int)(row / a.hq);
    const int hq = (int)(row % a.hq);
    const int64_t grp = (int64_t)seq * a.hkv + hq / a.g;

    if (tid < 16) s_tab[tid] = (tid & 8) ? -a.qc.a32[tid & 7] : a.qc.a32[tid & 7];
    float z[16];
    {
        const float4* zp = reinterpret_cast<const float4*>(a.zq + row * kD + 16 * l);
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const float4 t = zp[v];
            z[4 * v] = t.x; z[4 * v + 1] = t.y; z[4 * v + 2] = t.z; z[4 * v + 3] = t.w;
        }
    }
    __syncthreads();

    const int32_t* cand = a.cand + row * a.n_cand;
    float* out = a.cand_score + row * a.n_cand;
    const uint8_t* rec = a.rec + grp * a.capacity * kRec;
    const int64_t t0 = (int64_t)blockIdx.x * kRrTile;

    constexpr int kUnroll = 4;
#pragma unroll 1
    for (int it = 0; it < kRrTile / kRrSlots; it += kUnroll) {
        uint4 chunk[kUnroll];
        int64_t ci[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            ci[u] = t0 + (int64_t)(it + u) * kRrSlots + slot;
            chunk[u] = make_uint4(0, 0, 0, 0);
            if (ci[u] < a.c_eff) {
                const int64_t key = cand[ci[u]];
                if (key >= 0 && key < a.n) chunk[u] = reinterpret_cast<const uint4*>(rec + key * kRec)[l];
            }
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
            const uint32_t c0 = chunk[u].x, c1 = chunk[u].y;
            float d0 = 0.f, d1 = 0.f;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                d0 += s_tab[(c0 >> (4 * j)) & 15u] * z[j];
                d1 += s_tab[(c1 >> (4 * j)) & 15u] * z[8 + j];
            }
            float part = __uint_as_float(chunk[u].z) * d0 + __uint_as_float(chunk[u].w) * d1;
            part += __shfl_xor(part, 1, 64);
            part += __shfl_xor(part, 2, 64);
            part += __shfl_xor(part, 4, 64);
            // + 0.0f turns -0 into +0, so equal estimates compare equal in the top-k keys.
            if (l == 0 && ci[u] < a.c_eff) out[ci[u]] = part + 0.0f;
        }
    }
}

// ---------------------------------------------------------------- top-k

constexpr int kTkThreads = 1024;
constexpr int kTkWaves = kTkThreads / 64;

__device__ __forceinline__ uint32_t order_key(float f) {
    const uint32_t u = __float_as_uint(f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float key_float(uint32_t k) {
    const uint32_t u = (k & 0x80000000u) ? (k & 0x7fffffffu) : ~k;
    return __uint_as_float(u);
}

__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t v, int lane) {
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        uint32_t o = __shfl_up(v, d, 64);
        if (lane >= d) v += o;
    }
    return v;
}

// Exclusive block-wide prefix of v (all threads must call).
__device__ __forceinline__ uint32_t block_excl_scan(uint32_t v, uint32_t* s_w, uint32_t* total) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const uint32_t incl = wave_incl_scan(v, lane);
    if (lane == 63) s_w[wave] = incl;
    __syncthreads();
    uint32_t pre = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < kTkWaves; ++w) {
        const uint32_t x = s_w[w];
        if (w < wave) pre += x;
        tot += x;
    }
    __syncthreads();
    *total = tot;
    return pre + incl - v;
}

template <int EPT>
__global__ __launch_bounds__(kTkThreads) void topk_kernel(RetrieveArgs a) {
    __shared__ uint32_t s_hist[256];
    __shared__ uint32_t s_w[kTkWaves];
    __shared__ uint32_t s_mm[2][kTkWaves];
    __shared__ uint32_t s_digit, s_need;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t row = blockIdx.x;
    const int C = (int)a.c_eff;
    const int kk = min(a.top_k, C);
    const float* sc = a.cand_score + row * a.n_cand;
    const int32_t* cand = a.cand + row * a.n_cand;

    // Order-preserving keys of this thread's contiguous run of candidates.
    uint32_t key[EPT];
    uint32_t kmin = 0xffffffffu, kmax = 0u;
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
        const int p = tid * EPT + e;
        key[e] = p < C ? order_key(sc[p]) : 0u;  // valid keys are all > 0
        if (p < C) {
            kmin = min(kmin, key[e]);
            kmax = max(kmax, key[e]);
        }
    }
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        kmin = min(kmin, (uint32_t)__shfl_xor(kmin, d, 64));
        kmax = max(kmax, (uint32_t)__shfl_xor(kmax, d, 64));
    }
    if (lane == 0) { s_mm[0][wave] = kmin; s_mm[1][wave] = kmax; }
    __syncthreads();
#pragma unroll
    for (int w = 0; w < kTkWaves; ++w) {
        kmin = min(kmin, s_mm[0][w]);
        kmax = max(kmax, s_mm[1][w]);
    }

    // Radix select of the kk-th largest u = key - kmin, 8-bit digits from the top
    // of the occupied range (so the first histogram is spread over the data).
    const uint32_t range = kmax - kmin;
    const int nbits = range ? 32 - __clz(range) : 0;
    uint32_t prefix = 0, mask = 0, need = (uint32_t)kk;
    int shift = nbits > 8 ? nbits - 8 : 0;
#pragma unroll 1
    for (int pass = 0; pass < 4 && nbits > 0; ++pass) {
        if (tid < 256) s_hist[tid] = 0;
        __syncthreads();
#pragma unroll
        for (int e = 0; e < EPT; ++e) {
            const uint32_t u = key[e] - kmin;
            if (key[e] != 0u && (u & mask) == prefix) atomicAdd(&s_hist[(u >> shift) & 255u], 1u);
        }
        __syncthreads();
        if (wave == 0) {
            // Suffix sums over digits 255..0: lane L owns digits 255-4L..252-4L.
            uint32_t h[4];
            uint32_t tot = 0;
#pragma unroll
            for (int r = 0; r < 4; ++r) { h[r] = s_hist[255 - 4 * lane - r]; tot += h[r]; }
            const uint32_t incl = wave_incl_scan(tot, lane);
            uint32_t above = incl - tot;  // keys with a larger digit
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                if (above < need && above + h[r] >= need) {
                    s_digit = 255u - 4u * lane - r;
                    s_need = need - above;
                }
                above += h[r];
            }
        }
        __syncthreads();
        prefix |= s_digit << shift;
        mask |= 255u << shift;
        need = s_need;
        __syncthreads();
        if (shift == 0) break;
        shift = shift > 8 ? shift - 8 : 0;
    }
    const uint32_t T = kmin + prefix;  // the kk-th largest key value
    const uint32_t quota = need;       // how many keys equal to T are taken

    uint32_t n_eq = 0;
#pragma unroll
    for (int e = 0; e < EPT; ++e) n_eq += (key[e] == T && key[e] != 0u) ? 1u : 0u;
    uint32_t tot;
    uint32_t eq_before = block_excl_scan(n_eq, s_w, &tot);
    uint32_t n_sel = 0;
    uint64_t selmask = 0;
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
        bool s = false;
        if (key[e] != 0u) {
            if (key[e] > T) s = true;
            else if (key[e] == T) { s = eq_before < quota; ++eq_before; }
        }
        selmask |= (s ? 1ull : 0ull) << e;
        n_sel += s ? 1u : 0u;
    }
    uint32_t pos = block_excl_scan(n_sel, s_w, &tot);
    // Winners in candidate order, i.e. ascending key index.
    int32_t* oi = a.out_idx + row * a.top_k;
    float* os = a.out_score ? a.out_score + row * a.top_k : nullptr;
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
        if ((selmask >> e) & 1ull) {
            const int p = tid * EPT + e;
            if (pos < (uint32_t)kk) {
                oi[pos] = cand[p];
                if (os) os[pos] = key_float(key[e]);
            }
            ++pos;
        }
    }
    for (int r = kk + tid; r < a.top_k; r += kTkThreads) {
        oi[r] = -1;
        if (os) os[r] = -__builtin_huge_valf();
    }
}

__global__ void pad_outputs_kernel(int32_t* out_idx, float* out_score, int64_t count) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < count) {
        out_idx[i] = -1;
        if (out_score) out_score[i] = -__builtin_huge_valf();
    }
}

}  // namespace

hipError_t launch_rerank(const RetrieveArgs& a, hipStream_t s) {
    const int64_t tiles = (a.c_eff + kRrTile - 1) / kRrTile;
    prof_begin("rerank", s);
    hipLaunchKernelGGL(rerank_kernel, dim3((unsigned)tiles, (unsigned)(a.batch * a.hq)), dim3(kRrThreads),
                       0, s, a);
    prof_end(s);
    return hipGetLastError();
}

hipError_t launch_topk(const RetrieveArgs& a, hipStream_t s) {
    const int64_t ept = (a.c_eff + kTkThreads - 1) / kTkThreads;
    const dim3 grid((unsigned)(a.batch * a.hq));
    prof_begin("topk", s);
    if (ept <= 1)
        hipLaunchKernelGGL(topk_kernel<1>, grid, dim3(kTkThreads), 0, s, a);
    else if (ept <= 2)
        hipLaunchKernelGGL(topk_kernel<2>, grid, dim3(kTkThreads), 0, s, a);
    else if (ept <= 4)
        hipLaunchKernelGGL(topk_kernel<4>, grid, dim3(kTkThreads), 0, s, a);
    else if (ept <= 8)
        hipLaunchKernelGGL(topk_kernel<8>, grid, dim3(kTkThreads), 0, s, a);
    else if (ept <= 16)
        hipLaunchKernelGGL(topk_kernel<16>, grid, dim3(kTkThreads), 0, s, a);
    else if (ept <= 32)
        hipLaunchKernelGGL(topk_kernel<32>, grid, dim3(kTkThreads), 0, s, a);
    else
        hipLaunchKernelGGL(topk_kernel<64>, grid, dim3(kTkThreads), 0, s, a);
    prof_end(s);
    return hipGetLastError();
}

hipError_t launch_pad_outputs(const RetrieveArgs& a, hipStream_t s) {
    const int64_t count = (int64_t)a.batch * a.hq * a.top_k;
    prof_begin("pad_outputs", s);
    hipLaunchKernelGGL(pad_outputs_kernel, dim3((unsigned)((count + 255) / 256)), dim3(256), 0, s,
                       a.out_idx, a.out_score, count);
    prof_end(s);
    return hipGetLastError();
}

}  // namespace pariskv
