// Stage I of the decode-time retrieval: query transform, per-subspace
// cluster ranking -> tier-bonus table, collision scan over every key, and the
// bucket top-beta selection (Sec. "Retrieval" (1); Appendix "Coarse Candidate
// Generation (Collision Ratio and Multi-Tier Weights)", Eq. collision_score,
// "Top-beta selection with small-range integer scores"; Alg. 1 Stage I).
//
// Kernels, in launch order:
//   query_lut_kernel   one block per (sequence, KV head, quad, 4 subspaces), one
//                      wave per (head slot, subspace): z = H(s q) in exact
//                      float64 (written as z/D float for the rerank), the 256
//                      centroids ranked by the exact proxy sum_j +-z_j (ties:
//                      lower id), cluster counts prefix-summed in that order, and
//                      the tier bonus of each cluster placed in byte `slot` of a
//                      packed word (4 query heads of a KV head share one uint32),
//                      assembled in LDS and stored whole.
//   collide_kernel     streams the 16 id bytes of every key once per quad of
//                      query heads, sums 16 packed LDS lookups (4 head scores in
//                      the 4 bytes of one uint32; each is at most 96, so no
//                      carries), writes S as bytes per head and a suffix
//                      histogram #{S >= v} per head and 4096-key chunk (frequent
//                      low scores counted by wave ballots, the rest by LDS atomics).
//   threshold_kernel   one wave per query head: theta = largest v with
//                      #{S >= v} >= C_eff, the quota of S == theta keys, and per
//                      chunk the number of S > theta / S == theta keys in
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

constexpr int kLutThreads = 1024;  // 16 waves: 4 head slots x 4 subspaces

__global__ __launch_bounds__(kLutThreads) void query_lut_kernel(RetrieveArgs a) {
    __shared__ double s_z[4][kD];
    __shared__ uint32_t s_cnt[4][kCentroids];
    __shared__ uint32_t s_lut[4][kCentroids];  // packed bonus words of the 4 subspaces
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int slot = wave >> 2;          // head of the quad
    const int sub = wave & 3;

    // blockIdx.x = ((seq * hkv + kvh) * quads + quad) * 4 + subspace group
    const int sg = blockIdx.x & 3;
    const int64_t gq = blockIdx.x >> 2;  // (seq * hkv + kvh) * quads + quad
    const int quad = (int)(gq % a.quads);
    const int64_t grp = gq / a.quads;    // seq * hkv + kvh
    const int seq = (int)(grp / a.hkv);
    const int kvh = (int)(grp % a.hkv);
    const int b = 4 * sg + sub;          // this wave's subspace
    const int hg = quad * 4 + slot;      // head within the KV group
    const bool live = hg < a.g;
    const int64_t row = (int64_t)seq * a.hq + kvh * a.g + hg;

    // Cluster counts of the 4 subspaces; z = H (s (.) q) of the 4 heads, exactly in float64.
    const uint32_t* cnt = a.counts + grp * (kB * kCentroids) + (4 * sg) * kCentroids;
    (&s_cnt[0][0])[tid] = cnt[tid];
    (&s_lut[0][0])[tid] = 0u;
    const int zh = tid >> 7, zi = tid & (kD - 1);  // threads < 512: 4 heads x 128 coordinates
    const bool zlive = zh < 4 && quad * 4 + zh < a.g;
    if (zlive) {
        const __half* qp = static_cast<const __half*>(a.q) + (row + (zh - slot)) * kD;
        double v = (double)__half2float(qp[zi]);
        if ((a.sb.w[zi >> 5] >> (zi & 31)) & 1u) v = -v;
        s_z[zh][zi] = v;
    }
    __syncthreads();
    for (int h = 1; h < kD; h <<= 1) {
        if (zi < kD / 2 && zlive) {
            const int i = ((zi / h) * 2 * h) + (zi % h);
            const double x0 = s_z[zh][i], x1 = s_z[zh][i + h];
            s_z[zh][i] = __dadd_rn(x0, x1);
            s_z[zh][i + h] = __dsub_rn(x0, x1);
        }
        __syncthreads();
    }
    if (sg == 0 && zlive)
        a.zq[(row + (zh - slot)) * kD + zi] = (float)(s_z[zh][zi] * (1.0 / kD));

    if (live) {
        double zb[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) zb[j] = s_z[slot][8 * b + j];
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
            cc[r] = s_cnt[sub][cid[r]];
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
            if (bonus) atomicOr(&s_lut[sub][cid[r]], bonus << (8 * slot));
            start += cc[r];
        }
    }
    __syncthreads();
    // Unused slots of the last quad keep bonus 0.
    a.lut[gq * (kB * kCentroids) + (4 * sg) * kCentroids + tid] = (&s_lut[0][0])[tid];
}

// ---------------------------------------------------------------- collision scan

constexpr int kColThreads = 256;
constexpr int kColWaves = kColThreads / 64;
constexpr int kColKeysPerIter = 4 * kColThreads;  // 4 keys per thread per iteration
constexpr int kLowCut = 4;  // scores below this are counted by ballot, not by LDS atomics

// Suffix sums of a 97-bin histogram held as (lo = bins 0..63 by lane, hi = bins
// 64..96 by lane < 33): returns (sfx_lo, sfx_hi) with sfx[v] = sum_{u >= v} h[u].
__device__ __forceinline__ void wave_suffix97(uint32_t lo, uint32_t hi, int lane, uint32_t* s_lo,
                                              uint32_t* s_hi) {
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const uint32_t o = __shfl_down(hi, d, 64);
        if (lane + d < 64) hi += o;
    }
    const uint32_t tot_hi = __shfl(hi, 0, 64);
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
        const uint32_t o = __shfl_down(lo, d, 64);
        if (lane + d < 64) lo += o;
    }
    *s_lo = lo + tot_hi;
    *s_hi = hi;
}

__global__ __launch_bounds__(kColThreads) void collide_kernel(RetrieveArgs a) {
    __shared__ uint32_t s_lut[kB * kCentroids];
    __shared__ uint32_t s_hist[kColWaves][4][kBins + 3];
    __shared__ uint32_t s_pack[kColKeysPerIter];
    __shared__ uint32_t s_low[kColWaves][kLowCut - 1][4];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int64_t chunk = blockIdx.x;
    const int64_t gq = blockIdx.y;             // (seq * hkv + kvh) * quads + quad
    const int quad = (int)(gq % a.quads);
    const int64_t grp = gq / a.quads;          // seq * hkv + kvh
    const int seq = (int)(grp / a.hkv);
    const int kvh = (int)(grp % a.hkv);
    const int nh = min(4, a.g - 4 * quad);     // heads in this quad
    const int64_t row0 = (int64_t)seq * a.hq + kvh * a.g + 4 * quad;  // row of head 0 of the quad

    const uint4* lsrc = reinterpret_cast<const uint4*>(a.lut + gq * (kB * kCentroids));
    for (int i = tid; i < kB * kCentroids / 4; i += kColThreads)
        reinterpret_cast<uint4*>(s_lut)[i] = lsrc[i];
    for (int i = tid; i < kColWaves * 4 * (kBins + 3); i += kColThreads) (&s_hist[0][0][0])[i] = 0;
    __syncthreads();

    const uint8_t* ids = a.ids + grp * a.capacity * kB;
    const int64_t c0 = chunk * kChunk;
    const int64_t c1 = min(c0 + (int64_t)kChunk, a.n);
    uint32_t low[kLowCut - 1][4];  // wave-uniform: #{S >= v} for v = 1 .. kLowCut-1, per head
#pragma unroll
    for (int v = 0; v < kLowCut - 1; ++v)
#pragma unroll
        for (int h = 0; h < 4; ++h) low[v][h] = 0;

    for (int64_t base = c0; base < c1; base += kColKeysPerIter) {
        // Key base + tid + 256 j: one 16-byte id row per lane, a wave reads 1 KiB contiguous.
        uint4 w[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int64_t i = base + tid + kColThreads * j;
            w[j] = i < c1 ? *reinterpret_cast<const uint4*>(ids + i * kB) : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int64_t i = base + tid + kColThreads * j;
            const uint32_t ww[4] = {w[j].x, w[j].y, w[j].z, w[j].w};
            uint32_t acc = 0;
#pragma unroll
            for (int b = 0; b < kB; ++b)
                acc += s_lut[b * kCentroids + ((ww[b >> 2] >> (8 * (b & 3))) & 0xffu)];
            const bool live = i < c1;
            acc = live ? acc : 0u;
            // Low scores are frequent: #{S >= v} for v < kLowCut is counted for all 4
            // heads at once with a byte-wise compare ((x | 0x80) - v has its top bit set
            // iff x >= v, for bytes below 128) and one wave ballot per head.
#pragma unroll
            for (int v = 1; v < kLowCut; ++v) {
                const uint32_t ge = ((acc | 0x80808080u) - (uint32_t)v * 0x01010101u) & 0x80808080u;
#pragma unroll
                for (int h = 0; h < 4; ++h)
                    low[v - 1][h] += (uint32_t)__popcll(__ballot(live && ((ge >> (8 * h + 7)) & 1u)));
            }
            // Higher scores are rare and spread out: exact per-value LDS histogram.
#pragma unroll
            for (int h = 0; h < 4; ++h) {
                const uint32_t sh = (acc >> (8 * h)) & 0xffu;
                if (h < nh && live && sh >= (uint32_t)kLowCut) atomicAdd(&s_hist[wave][h][sh], 1u);
            }
            s_pack[tid + kColThreads * j] = acc;
        }
        __syncthreads();
        // Thread t now writes keys base + 4t .. 4t+3 for every head: transpose 4 keys x 4
        // heads of bytes into one word per head.
        const int64_t k4 = base + 4 * tid;
        if (k4 < c1) {
            const uint4 sp = reinterpret_cast<const uint4*>(s_pack)[tid];
            const uint32_t lo01 = __builtin_amdgcn_perm(sp.y, sp.x, 0x05010400u);
            const uint32_t hi01 = __builtin_amdgcn_perm(sp.y, sp.x, 0x07030602u);
            const uint32_t lo23 = __builtin_amdgcn_perm(sp.w, sp.z, 0x05010400u);
            const uint32_t hi23 = __builtin_amdgcn_perm(sp.w, sp.z, 0x07030602u);
            uint32_t o[4];
            o[0] = __builtin_amdgcn_perm(lo23, lo01, 0x05040100u);
            o[1] = __builtin_amdgcn_perm(lo23, lo01, 0x07060302u);
            o[2] = __builtin_amdgcn_perm(hi23, hi01, 0x05040100u);
            o[3] = __builtin_amdgcn_perm(hi23, hi01, 0x07060302u);
#pragma unroll
            for (int h = 0; h < 4; ++h)
                if (h < nh) *reinterpret_cast<uint32_t*>(a.score8 + (row0 + h) * a.n_pad + k4) = o[h];
        }
        __syncthreads();
    }

    if (lane == 0) {
#pragma unroll
        for (int v = 0; v < kLowCut - 1; ++v)
#pragma unroll
            for (int h = 0; h < 4; ++h) s_low[wave][v][h] = low[v][h];
    }
    __syncthreads();

    // Per-chunk suffix histogram of every head: sfx[v] = #{keys in chunk : S >= v}, v = 0..97.
    if (wave < nh) {
        const int h = wave;
        uint32_t lo = 0, hi = 0;
#pragma unroll
        for (int w2 = 0; w2 < kColWaves; ++w2) {
            lo += s_hist[w2][h][lane];
            hi += lane < kBins - 64 ? s_hist[w2][h][64 + lane] : 0u;
        }
        uint32_t sl, sh;
        wave_suffix97(lo, hi, lane, &sl, &sh);  // exact for v >= kLowCut
        if (lane == 0) sl = (uint32_t)(c1 - c0);
        if (lane >= 1 && lane < kLowCut) {
            uint32_t t = 0;
#pragma unroll
            for (int w2 = 0; w2 < kColWaves; ++w2) t += s_low[w2][lane - 1][h];
            sl = t;
        }
        uint32_t* dst = a.chunk_sfx + ((row0 + h) * a.n_chunks + chunk) * kSfx;
        dst[lane] = sl;
        if (lane < kSfx - 64) dst[64 + lane] = lane < kBins - 64 ? sh : 0u;
    }

}

// ---------------------------------------------------------------- threshold

constexpr int kThrThreads = 256;  // one wave per query head

__global__ __launch_bounds__(kThrThreads) void threshold_kernel(RetrieveArgs a) {
    const int lane = threadIdx.x & 63;
    const int64_t row = (int64_t)blockIdx.x * (kThrThreads / 64) + (threadIdx.x >> 6);
    if (row >= (int64_t)a.batch * a.hq) return;
    const uint32_t* sfx = a.chunk_sfx + row * a.n_chunks * kSfx;
    // Whole-row suffix histogram; lane holds v = lane and v = 64 + lane.
    uint32_t tl = 0, th = 0;
    for (int64_t c = 0; c < a.n_chunks; ++c) {
        tl += sfx[c * kSfx + lane];
        if (lane < kSfx - 64) th += sfx[c * kSfx + 64 + lane];
    }
    const uint32_t C = (uint32_t)a.c_eff;
    // theta = largest v with #{S >= v} >= C (suffix counts fall with v; #{S >= 0} = n >= C).
    const uint64_t ok_lo = __ballot(tl >= C);
    const uint64_t ok_hi = __ballot(lane < kBins - 64 && th >= C);
    const int theta = ok_hi ? 64 + (63 - __clzll(ok_hi)) : (63 - __clzll(ok_lo));
    const uint32_t gt = theta + 1 < 64 ? __shfl(tl, theta + 1, 64) : __shfl(th, theta + 1 - 64, 64);
    if (lane == 0) {
        int32_t* t = a.thresh + row * 4;
        t[0] = theta;
        t[1] = (int32_t)gt;
        t[2] = (int32_t)(C - gt);
        t[3] = (int32_t)C;
    }
    // Keys with S > theta and S == theta in the chunks before each chunk.
    uint32_t carry_g = 0, carry_e = 0;
    for (int64_t cb = 0; cb < a.n_chunks; cb += 64) {
        const int64_t c = cb + lane;
        uint32_t g = 0, e = 0;
        if (c < a.n_chunks) {
            g = sfx[c * kSfx + theta + 1];
            e = sfx[c * kSfx + theta] - g;
        }
        const uint32_t ig = wave_incl_scan_u32(g, lane);
        const uint32_t ie = wave_incl_scan_u32(e, lane);
        if (c < a.n_chunks) {
            int32_t* cbp = a.chunk_base + (row * a.n_chunks + c) * 2;
            cbp[0] = (int32_t)(carry_g + ig - g);
            cbp[1] = (int32_t)(carry_e + ie - e);
        }
        carry_g += __shfl(ig, 63, 64);
        carry_e += __shfl(ie, 63, 64);
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
    const int64_t rows = (int64_t)a.batch * a.hq;
    prof_begin("threshold", s);
    hipLaunchKernelGGL(threshold_kernel, dim3((unsigned)((rows + 3) / 4)), dim3(kThrThreads), 0, s, a);
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
