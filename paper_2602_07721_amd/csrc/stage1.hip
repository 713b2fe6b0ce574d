// Stage I of the decode-time retrieval: query transform, per-subspace
// cluster ranking -> tier-bonus table, collision scan over every key, and the
// bucket top-beta selection (Sec. "Retrieval" (1); Appendix "Coarse Candidate
// Generation (Collision Ratio and Multi-Tier Weights)", Eq. collision_score,
// "Top-beta selection with small-range integer scores"; Alg. 1 Stage I).
//
// Kernels, in launch order:
//   query_lut_kernel   one block per (sequence, KV head, quad, slot): z = H(s q)
//                      in exact float64, writes z/D as float for the rerank,
//                      ranks the 256 centroids of every subspace by the exact
//                      proxy sum_j +-z_j (ties: lower id), prefix-sums the
//                      cluster counts in that order and writes the tier bonus
//                      of each cluster into byte `slot` of a packed table
//                      (4 query heads of a KV head share one uint32 entry).
//   collide_kernel     streams the 16 id bytes of every key once per quad of
//                      query heads, sums 16 packed LDS lookups (the 4 head
//                      scores ride in the 4 bytes of one uint32; each is at
//                      most 96, so no carries), writes S as bytes per head and
//                      a 97-bin histogram per head and chunk (no atomics in
//                      global memory).
//   threshold_kernel   one block per query head: theta = largest v with
//                      #{S >= v} >= C_eff, quota of S == theta keys, and for
//                      every chunk the number of S > theta / S == theta keys in
//                      earlier chunks.
//   compact_kernel     writes candidate indices in ascending key order: all
//                      S > theta and the first `quota` S == theta keys.

#include <hip/hip_fp16.h>

#include "internal.hpp"

#pragma clang fp contract(off)

namespace pariskv {

namespace {

// ---------------------------------------------------------------- helpers

__device__ __forceinline__ uint32_t wave_incl_scan_u32(uint32_t v, int lane) {
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        uint32_t o = __shfl_up(v, d, 64);
        if (lane >= d) v += o;
    }
    return v;
}

// ---------------------------------------------------------------- query + LUT

constexpr int kLutThreads = 256;

__global__ __launch_bounds__(kLutThreads) void query_lut_kernel(RetrieveArgs a) {
    __shared__ double s_z[kD];
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;

    // blockIdx.x = ((seq * hkv + kvh) * quads + quad) * 4 + slot
    const int slot = blockIdx.x & 3;
    const int quad = (blockIdx.x >> 2) % a.quads;
    const int64_t grp = (blockIdx.x >> 2) / a.quads;  // seq * hkv + kvh
    const int seq = (int)(grp / a.hkv);
    const int kvh = (int)(grp % a.hkv);
    const int hg = quad * 4 + slot;  // head within the KV group
    uint8_t* lut_bytes = reinterpret_cast<uint8_t*>(a.lut + (grp * a.quads + quad) * (kB * kCentroids));

    if (hg >= a.g) {
        // Unused slot of the last quad: zero bonus everywhere.
        for (int i = tid; i < kB * kCentroids; i += kLutThreads) lut_bytes[4 * i + slot] = 0;
        return;
    }
    const int hq = kvh * a.g + hg;
    const int64_t row = (int64_t)seq * a.hq + hq;

    // z = H (s (.) q), exact in float64 (butterflies in LDS).
    if (tid < kD) {
        const __half* qp = static_cast<const __half*>(a.q) + row * kD;
        double v = (double)__half2float(qp[tid]);
        if ((a.sb.w[tid >> 5] >> (tid & 31)) & 1u) v = -v;
        s_z[tid] = v;
    }
    __syncthreads();
    for (int h = 1; h < kD; h <<= 1) {
        if (tid < kD / 2) {
            const int i = ((tid / h) * 2 * h) + (tid % h);
            const double x0 = s_z[i], x1 = s_z[i + h];
            s_z[i] = __dadd_rn(x0, x1);
            s_z[i + h] = __dsub_rn(x0, x1);
        }
        __syncthreads();
    }
    if (tid < kD) a.zq[row * kD + tid] = (float)(s_z[tid] * (1.0 / kD));

    const uint32_t* cnt = a.counts + grp * (kB * kCentroids);
    // One wave per subspace; lane L holds ranks 4L..4L+3 after the sort.
    for (int b = wave; b < kB; b += kLutThreads / 64) {
        double zb[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) zb[j] = s_z[8 * b + j];
        int64_t key[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int c = 4 * lane + r;
            double p = 0.0;
#pragma unroll
            for (int j = 0; j < 8; ++j) p = ((c >> j) & 1) ? __dsub_rn(p, zb[j]) : __dadd_rn(p, zb[j]);
            // p is an exact multiple of 2^-24 with |p| < 2^26: exact as an integer.
            const int64_t pi = (int64_t)(p * 16777216.0);
            key[r] = pi * 256 + (255 - c);  // descending key: proxy desc, then id asc
        }
        // Bitonic sort, descending, element e = 4*lane + r.
#pragma unroll
        for (int k = 2; k <= kCentroids; k <<= 1) {
#pragma unroll
            for (int j = k >> 1; j > 0; j >>= 1) {
                if (j >= 4) {
                    const int lm = j >> 2;
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int e = 4 * lane + r;
                        const int64_t other = __shfl_xor(key[r], lm, 64);
                        const bool lower = (e & j) == 0;
                        const bool desc = (e & k) == 0;
                        const int64_t mx = key[r] > other ? key[r] : other;
                        const int64_t mn = key[r] > other ? other : key[r];
                        key[r] = (lower == desc) ? mx : mn;
                    }
                } else {
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int r2 = r ^ j;
                        if (r2 > r) {
                            const int e = 4 * lane + r;
                            const bool desc = (e & k) == 0;
                            const int64_t x0 = key[r], x1 = key[r2];
                            const bool swap = desc ? (x0 < x1) : (x0 > x1);
                            key[r] = swap ? x1 : x0;
                            key[r2] = swap ? x0 : x1;
                        }
                    }
                }
            }
        }
        // Exclusive prefix of cluster counts in rank order -> start rank P(c).
        uint32_t cc[4];
        int cid[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            cid[r] = 255 - (int)(key[r] & 255);
            cc[r] = cnt[b * kCentroids + cid[r]];
        }
        const uint32_t tot = cc[0] + cc[1] + cc[2] + cc[3];
        const uint32_t incl = wave_incl_scan_u32(tot, lane);
        uint32_t start = incl - tot;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            uint32_t bonus = 0;
#pragma unroll
            for (int l = kTierCount - 1; l >= 0; --l)
                if (start < a.cuts[l]) bonus = (uint32_t)(kTierCount - l);
            lut_bytes[4 * (b * kCentroids + cid[r]) + slot] = (uint8_t)bonus;
            start += cc[r];
        }
    }
}

// ---------------------------------------------------------------- collision scan

constexpr int kColThreads = 256;
constexpr int kColWaves = kColThreads / 64;

__global__ __launch_bounds__(kColThreads) void collide_kernel(RetrieveArgs a) {
    __shared__ uint32_t s_lut[kB * kCentroids];
    __shared__ uint32_t s_hist[kColWaves][4][kBins];

    const int tid = threadIdx.x;
    const int wave = tid >> 6;
    const int64_t chunk = blockIdx.x;
    const int quad = blockIdx.y % a.quads;
    const int64_t grp = blockIdx.y / a.quads;  // seq * hkv + kvh
    const int seq = (int)(grp / a.hkv);
    const int kvh = (int)(grp % a.hkv);
    const int nh = min(4, a.g - 4 * quad);     // heads in this quad

    const uint4* lsrc = reinterpret_cast<const uint4*>(a.lut + (grp * a.quads + quad) * (kB * kCentroids));
    for (int i = tid; i < kB * kCentroids / 4; i += kColThreads)
        reinterpret_cast<uint4*>(s_lut)[i] = lsrc[i];
    for (int i = tid; i < kColWaves * 4 * kBins; i += kColThreads) (&s_hist[0][0][0])[i] = 0;
    __syncthreads();

    const uint8_t* ids = a.ids + grp * a.capacity * kB;
    const int64_t c0 = chunk * kChunk;
    const int64_t c1 = min(c0 + kChunk, a.n);
    uint8_t* srow[4];
#pragma unroll
    for (int h = 0; h < 4; ++h) {
        const int hq = kvh * a.g + 4 * quad + min(h, nh - 1);
        srow[h] = a.score8 + ((int64_t)seq * a.hq + hq) * a.n_pad;
    }

    for (int64_t base = c0 + 4 * tid; base < c1; base += 4 * kColThreads) {
        uint32_t s[4];
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
            const int64_t i = base + kk;
            uint32_t acc = 0;
            if (i < c1) {
                const uint4 w = *reinterpret_cast<const uint4*>(ids + i * kB);
                const uint32_t ww[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
                for (int b = 0; b < kB; ++b)
                    acc += s_lut[b * kCentroids + ((ww[b >> 2] >> (8 * (b & 3))) & 0xffu)];
#pragma unroll
                for (int h = 0; h < 4; ++h)
                    if (h < nh) atomicAdd(&s_hist[wave][h][(acc >> (8 * h)) & 0xffu], 1u);
            }
            s[kk] = acc;
        }
        // Transpose 4 keys x 4 heads of bytes into one word per head.
        const uint32_t lo01 = __builtin_amdgcn_perm(s[1], s[0], 0x05010400u);
        const uint32_t hi01 = __builtin_amdgcn_perm(s[1], s[0], 0x07030602u);
        const uint32_t lo23 = __builtin_amdgcn_perm(s[3], s[2], 0x05010400u);
        const uint32_t hi23 = __builtin_amdgcn_perm(s[3], s[2], 0x07030602u);
        uint32_t o[4];
        o[0] = __builtin_amdgcn_perm(lo23, lo01, 0x05040100u);
        o[1] = __builtin_amdgcn_perm(lo23, lo01, 0x07060302u);
        o[2] = __builtin_amdgcn_perm(hi23, hi01, 0x05040100u);
        o[3] = __builtin_amdgcn_perm(hi23, hi01, 0x07060302u);
#pragma unroll
        for (int h = 0; h < 4; ++h)
            if (h < nh) *reinterpret_cast<uint32_t*>(srow[h] + base) = o[h];
    }
    __syncthreads();

    for (int i = tid; i < nh * kBins; i += kColThreads) {
        const int h = i / kBins, v = i % kBins;
        uint32_t t = 0;
#pragma unroll
        for (int w = 0; w < kColWaves; ++w) t += s_hist[w][h][v];
        const int hq = kvh * a.g + 4 * quad + h;
        const int64_t row = (int64_t)seq * a.hq + hq;
        a.chunk_hist[(row * a.n_chunks + chunk) * kBins + v] = t;
    }
}

// ---------------------------------------------------------------- threshold

constexpr int kThrThreads = 256;

__global__ __launch_bounds__(kThrThreads) void threshold_kernel(RetrieveArgs a) {
    __shared__ uint32_t s_hist[kBins];
    __shared__ int s_theta;
    __shared__ uint32_t s_wsum[kThrThreads / 64][2];
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int64_t row = blockIdx.x;
    const uint32_t* ch = a.chunk_hist + row * a.n_chunks * kBins;

    if (tid < kBins) {
        uint32_t t = 0;
        for (int64_t c = 0; c < a.n_chunks; ++c) t += ch[c * kBins + tid];
        s_hist[tid] = t;
    }
    __syncthreads();
    if (tid == 0) {
        const uint32_t C = (uint32_t)a.c_eff;
        uint32_t acc = 0;
        int theta = 0;
        for (int v = kMaxScore; v >= 0; --v) {
            acc += s_hist[v];
            if (acc >= C) { theta = v; break; }
        }
        const uint32_t gt = acc - s_hist[theta];
        s_theta = theta;
        int32_t* th = a.thresh + row * 4;
        th[0] = theta;
        th[1] = (int32_t)gt;
        th[2] = (int32_t)(C - gt);
        th[3] = (int32_t)C;
    }
    __syncthreads();
    const int theta = s_theta;

    // Exclusive prefix over chunks of (#S > theta, #S == theta).
    uint32_t carry_g = 0, carry_e = 0;
    for (int64_t c0 = 0; c0 < a.n_chunks; c0 += kThrThreads) {
        const int64_t c = c0 + tid;
        uint32_t g = 0, e = 0;
        if (c < a.n_chunks) {
            for (int v = theta + 1; v <= kMaxScore; ++v) g += ch[c * kBins + v];
            e = ch[c * kBins + theta];
        }
        const uint32_t ig = wave_incl_scan_u32(g, lane);
        const uint32_t ie = wave_incl_scan_u32(e, lane);
        if (lane == 63) { s_wsum[wave][0] = ig; s_wsum[wave][1] = ie; }
        __syncthreads();
        uint32_t pg = carry_g, pe = carry_e;
        for (int w = 0; w < wave; ++w) { pg += s_wsum[w][0]; pe += s_wsum[w][1]; }
        if (c < a.n_chunks) {
            int32_t* cb = a.chunk_base + (row * a.n_chunks + c) * 2;
            cb[0] = (int32_t)(pg + ig - g);
            cb[1] = (int32_t)(pe + ie - e);
        }
        for (int w = 0; w < kThrThreads / 64; ++w) { carry_g += s_wsum[w][0]; carry_e += s_wsum[w][1]; }
        __syncthreads();
    }
}

// ---------------------------------------------------------------- compaction

constexpr int kCmpThreads = 256;  // 16 keys per thread, one chunk per block

__global__ __launch_bounds__(kCmpThreads) void compact_kernel(RetrieveArgs a) {
    __shared__ uint32_t s_wsum[kCmpThreads / 64];
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int64_t chunk = blockIdx.x;
    const int64_t row = blockIdx.y;
    const int32_t* th = a.thresh + row * 4;
    const uint32_t theta = (uint32_t)th[0];
    const uint32_t quota = (uint32_t)th[2];
    const int32_t* cb = a.chunk_base + (row * a.n_chunks + chunk) * 2;
    const uint32_t base_g = (uint32_t)cb[0], base_e = (uint32_t)cb[1];

    const int64_t i0 = chunk * kChunk + 16 * tid;
    uint32_t gmask = 0, emask = 0;
    uint8_t sv[16];
    if (i0 < a.n) {
        const uint4 w = *reinterpret_cast<const uint4*>(a.score8 + row * a.n_pad + i0);
        const uint32_t ww[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
        for (int j = 0; j < 16; ++j) {
            sv[j] = (uint8_t)((ww[j >> 2] >> (8 * (j & 3))) & 0xffu);
            const bool in = i0 + j < a.n;
            gmask |= (in && sv[j] > theta ? 1u : 0u) << j;
            emask |= (in && sv[j] == theta ? 1u : 0u) << j;
        }
    }
    // Packed (gt, eq) counts: each at most 4096 per chunk, 16 bits each.
    const uint32_t mine = (uint32_t)__popc(gmask) | ((uint32_t)__popc(emask) << 16);
    const uint32_t incl = wave_incl_scan_u32(mine, lane);
    if (lane == 63) s_wsum[wave] = incl;
    __syncthreads();
    uint32_t pre = incl - mine;
    for (int w = 0; w < wave; ++w) pre += s_wsum[w];
    uint32_t gb = base_g + (pre & 0xffffu);
    uint32_t eb = base_e + (pre >> 16);
    int32_t* cand = a.cand + row * a.n_cand;
#pragma unroll
    for (int j = 0; j < 16; ++j) {
        if ((gmask >> j) & 1u) {
            const uint32_t p = gb + min(eb, quota);
            if (p < (uint32_t)a.c_eff) cand[p] = (int32_t)(i0 + j);
            ++gb;
        } else if ((emask >> j) & 1u) {
            if (eb < quota && gb + eb < (uint32_t)a.c_eff) cand[gb + eb] = (int32_t)(i0 + j);
            ++eb;
        }
    }
}

}  // namespace

hipError_t launch_query_lut(const RetrieveArgs& a, hipStream_t s) {
    const int64_t blocks = (int64_t)a.batch * a.hkv * a.quads * 4;
    prof_begin("query_lut", s);
    hipLaunchKernelGGL(query_lut_kernel, dim3((unsigned)blocks), dim3(kLutThreads), 0, s, a);
    prof_end(s);
    return hipGetLastError();
}

hipError_t launch_collide(const RetrieveArgs& a, hipStream_t s) {
    prof_begin("collide", s);
    hipLaunchKernelGGL(collide_kernel, dim3((unsigned)a.n_chunks, (unsigned)(a.batch * a.hkv * a.quads)),
                       dim3(kColThreads), 0, s, a);
    prof_end(s);
    return hipGetLastError();
}

hipError_t launch_threshold(const RetrieveArgs& a, hipStream_t s) {
    prof_begin("threshold", s);
    hipLaunchKernelGGL(threshold_kernel, dim3((unsigned)(a.batch * a.hq)), dim3(kThrThreads), 0, s, a);
    prof_end(s);
    return hipGetLastError();
}

hipError_t launch_compact(const RetrieveArgs& a, hipStream_t s) {
    prof_begin("compact", s);
    hipLaunchKernelGGL(compact_kernel, dim3((unsigned)a.n_chunks, (unsigned)(a.batch * a.hq)),
                       dim3(kCmpThreads), 0, s, a);
    prof_end(s);
    return hipGetLastError();
}

}  // namespace pariskv
