// Stage I of the decode-time retrieval: query transform, per-subspace
// cluster ranking -> tier-bonus table, collision scan over every key, and the
// bucket top-beta selection (Sec. "Retrieval" (1); Appendix "Coarse Candidate
// Generation (Collision Ratio and Multi-Tier Weights)", Eq. collision_score,
// "Top-beta selection with small-range integer scores"; Alg. 1 Stage I).
//
// Kernels, in launch order:
//   query_lut_kernel   one block per (sequence, KV head, quad, 4 subspaces), one
//                      wave per (head slot, subspace): z = H(s q) in exact
//                      float64 by a register FWHT in one wave per head
//                      (written as z/D float for the rerank), the 256
//                      centroids ranked by the exact proxy sum_j +-z_j (ties:
//                      lower id) by a 64-bit bitonic sort, in registers, of the
//                      128 pair representatives (of c and c ^ 255 the one with
//                      the larger proxy), cluster counts prefix-summed in that
//                      order, and the tier
//                      bonus of each cluster placed in byte `slot` of a packed
//                      word (4 query heads of a KV head share one uint32) at the
//                      entry of the stored id form slot(c), assembled in LDS and
//                      stored whole.
//   collide_kernel     streams the 16 id bytes of every key once per quad of
//                      query heads, sums 16 packed LDS lookups (4 head scores in
//                      the 4 bytes of one uint32; each is at most 96, so no
//                      carries), writes S as bytes per head (64 consecutive
//                      bytes per wave store) and a suffix histogram
//                      #{S >= v} per head and 4096-key chunk (nonzero scores
//                      by LDS atomics into two lane-partitioned copies).  Loads and stores go
//                      through range-checked buffer descriptors, so the ragged
//                      last chunk needs no branches, and each XCD scans whole
//                      score rows.
//   threshold_kernel   one block of 16 waves per query head: theta = largest v
//                      with #{S >= v} >= C_eff, the quota of S == theta keys,
//                      and per chunk the number of S > theta / S == theta keys
//                      in earlier chunks.
// The compaction of the candidates lives with the rerank (stage2.hip).

#include <hip/hip_fp16.h>

#include "internal.hpp"

#pragma clang fp contract(off)

namespace pariskv {

namespace {

// ---------------------------------------------------------------- helpers

// Ranking the 256 centroids of a subspace.  Flipping every sign of a centroid
// negates its proxy, so the pairs {c, c ^ 255} hold proxies p and -p: sorting the
// member with the larger proxy of each pair (128 keys, 2 per lane) ranks the upper
// half, and the other members take the lower half in the reverse order.  One
// 128-key sort replaces a 256-key sort (28 stages of compare-exchanges on 2 keys
// per lane instead of 36 on 4).
//
// Each compare-exchange is one 64-bit compare into a lane mask, a scalar XOR with
// the stage's direction pattern, and two v_cndmask; partners 1 or 2 lanes away come
// through DPP, 4..16 lanes away through ds_swizzle, 32 away through ds_bpermute.

// Lanes whose bit t is set (t = 0 .. 5); 0 past bit 5.
__device__ constexpr uint64_t lane_bit(int t) {
    return t == 0 ? 0xAAAAAAAAAAAAAAAAull : t == 1 ? 0xCCCCCCCCCCCCCCCCull
         : t == 2 ? 0xF0F0F0F0F0F0F0F0ull : t == 3 ? 0xFF00FF00FF00FF00ull
         : t == 4 ? 0xFFFF0000FFFF0000ull : t == 5 ? 0xFFFFFFFF00000000ull : 0ull;
}

__device__ constexpr int log2i(int x) { return x <= 1 ? 0 : 1 + log2i(x >> 1); }

// Key a takes its partner's key b iff (b > a) == keep_max, lane by lane.
__device__ __forceinline__ int64_t exchange(int64_t a, uint32_t blo, uint32_t bhi, uint64_t keep_max) {
    const int64_t b = (int64_t)(((uint64_t)bhi << 32) | blo);
    const uint64_t take = ~(__ballot(b > a) ^ keep_max);  // keys are distinct
    const uint32_t alo = (uint32_t)a, ahi = (uint32_t)((uint64_t)a >> 32);
    return (int64_t)(((uint64_t)select_mask(take, bhi, ahi) << 32) | select_mask(take, blo, alo));
}

// In-lane pair (x, y): afterwards x >= y on lanes in desc, x <= y elsewhere.
__device__ __forceinline__ void order_pair(int64_t& x, int64_t& y, uint64_t desc) {
    const uint64_t swap = ~(__ballot(x < y) ^ desc);
    const uint32_t xl = (uint32_t)x, xh = (uint32_t)((uint64_t)x >> 32);
    const uint32_t yl = (uint32_t)y, yh = (uint32_t)((uint64_t)y >> 32);
    x = (int64_t)(((uint64_t)select_mask(swap, yh, xh) << 32) | select_mask(swap, yl, xl));
    y = (int64_t)(((uint64_t)select_mask(swap, xh, yh) << 32) | select_mask(swap, xl, yl));
}

// Bitonic sort of the 128 keys key[0..1] of every lane (element e = 2 lane + r),
// descending.  Bit b >= 1 of e is bit b - 1 of the lane.
__device__ __forceinline__ void sort128_desc(int64_t (&key)[2], int lane) {
#pragma unroll
    for (int k = 2; k <= 128; k <<= 1) {
#pragma unroll
        for (int j = k >> 1; j > 0; j >>= 1) {
            if (j >= 2) {
                // Element e keeps the larger key iff bits log2 j and log2 k of e agree.
                const uint64_t keep_max = ~(lane_bit(log2i(j) - 1) ^ lane_bit(log2i(k) - 1));
#pragma unroll
                for (int r = 0; r < 2; ++r) {
                    const uint32_t lo = (uint32_t)key[r], hi = (uint32_t)((uint64_t)key[r] >> 32);
                    key[r] = exchange(key[r], lane_xor(lo, j >> 1, lane), lane_xor(hi, j >> 1, lane), keep_max);
                }
            } else {
                // Descending where bit log2 k of e is clear.
                order_pair(key[0], key[1], ~lane_bit(log2i(k) - 1));
            }
        }
    }
}

// The histogram floor v_lo of a query head: the collision scan histograms only scores
// S >= v_lo.  It is the integer part of a normal-law estimate of the selection threshold with the
// subspaces' bonus weights taken as independent: mean sum_b E[bonus_b], variance
// sum_b Var[bonus_b] from the moments stats[b] = (sum_c count_c bonus_c, sum_c count_c
// bonus_c^2), and the upper-tail quantile z of the selected fraction p = C_eff / n by the
// rational approximation of Abramowitz & Stegun 26.2.23 (|error| < 4.5e-4).  Keys that
// resemble the query tend to be admitted in many subspaces at once, which fattens the
// upper tail, so the estimate usually lies below the true threshold; when it does not,
// the threshold kernel recounts (the floor never changes a result).  Floor 1 counts every
// nonzero score (for p >= 1/2, where little would be saved).  The scan and the threshold
// kernel evaluate this same function on the same inputs.
__device__ __forceinline__ uint32_t hist_floor(const float* st, int64_t n, int64_t c_eff, uint32_t flags) {
    if (flags & kFlagRecount) return kBins;  // above every score: nothing is histogrammed
    const float inv_n = 1.0f / (float)n;
    const float p = (float)c_eff * inv_n;
    if (!(p < 0.5f)) return 1u;
    float mu = 0.0f, var = 0.0f;
#pragma unroll
    for (int b = 0; b < kB; ++b) {
        const float m1 = st[2 * b] * inv_n, m2 = st[2 * b + 1] * inv_n;
        mu += m1;
        var += fmaxf(m2 - m1 * m1, 0.0f);
    }
    const float t = sqrtf(-2.0f * logf(p));
    const float z = t - (2.515517f + t * (0.802853f + t * 0.010328f)) /
                            (1.0f + t * (1.432788f + t * (0.189269f + t * 0.001308f)));
    const float est = mu + z * sqrtf(var);
    if (!(est >= 1.0f)) return 1u;
    return est >= (float)kMaxScore ? (uint32_t)kMaxScore : (uint32_t)est;
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

    // Cluster counts of the 4 subspaces, requested first and put in LDS after the
    // transform; the sign word of this lane's coordinates picked without indexing.
    const uint32_t* cnt = a.counts + grp * (kB * kCentroids) + (4 * sg) * kCentroids;
    const uint32_t cval = cnt[tid];
    const uint32_t sword = select_mask(0xFFFFFFFF00000000ull,
                                       select_mask(0xFFFF0000FFFF0000ull, a.sb.w[3], a.sb.w[2]),
                                       select_mask(0xFFFF0000FFFF0000ull, a.sb.w[1], a.sb.w[0]));
    (&s_lut[0][0])[tid] = 0u;
    // z = H (s (.) q) of the 4 heads exactly in float64: the wave of head `slot` and
    // subspace `slot` takes it in registers (coordinates 2 lane + r; stride-1 butterflies
    // inside a lane, the others across lanes) and leaves it in LDS for the other three
    // waves.  Waves w = 4 slot + sub go to SIMD w mod 4, so the 4 transforms run on 4
    // different SIMDs.
    const bool rotate = !(a.flags & kFlagNoRotation);
    if (sub == slot && live) {
        const uint32_t qw = reinterpret_cast<const uint32_t*>(static_cast<const __half*>(a.q) + row * kD)[lane];
        double z[2];
#pragma unroll
        for (int r = 0; r < 2; ++r) {
            const int zi = 2 * lane + r;
            double v = (double)__half2float(__ushort_as_half((unsigned short)(r ? qw >> 16 : qw & 0xffffu)));
            if (!rotate) v *= (double)kD;  // z = D q without the rotation (exact: D = 2^7)
            else if ((sword >> (zi & 31)) & 1u) v = -v;  // word zi / 32 = lane / 16
            z[r] = v;
        }
        if (rotate) {
            {
                const double x0 = z[0], x1 = z[1];
                z[0] = __dadd_rn(x0, x1);
                z[1] = __dsub_rn(x0, x1);
            }
#pragma unroll
            for (int h = 2; h < kD; h <<= 1) {
                // Partner index e ^ h is lane ^ (h / 2); the element with bit log2 h of
                // its index clear takes the sum, the other the difference.
                const bool upper = (lane & (h >> 1)) != 0;
#pragma unroll
                for (int r = 0; r < 2; ++r) {
                    const uint64_t u = (uint64_t)__double_as_longlong(z[r]);
                    const uint32_t lo = lane_xor((uint32_t)u, h >> 1, lane), hi = lane_xor((uint32_t)(u >> 32), h >> 1, lane);
                    const double o = __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
                    z[r] = upper ? __dsub_rn(o, z[r]) : __dadd_rn(z[r], o);
                }
            }
        }
#pragma unroll
        for (int r = 0; r < 2; ++r) {
            s_z[slot][2 * lane + r] = z[r];
            if (sg == 0) a.zq[row * kD + 2 * lane + r] = (float)(z[r] * (1.0 / kD));
        }
    }
    (&s_cnt[0][0])[tid] = cval;
    __syncthreads();

    if (live) {
        double zb[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) zb[j] = s_z[slot][8 * b + j];
        // Each pair {c, c ^ 255} (c with bit 7 clear) has proxies p and -p.  Its
        // representative is the member with the larger proxy (c when p = 0, the lower
        // id); sorting the 128 representatives by (|p| desc, id asc) ranks them 0..127,
        // and the other members follow in the reverse order: the one of the
        // representative at position i has rank 255 - i (proxy -|p| desc, and for
        // equal |p| the representatives' id order reverses under c ^ 255).
        int64_t key[2];
#pragma unroll
        for (int r = 0; r < 2; ++r) {
            const int c = 2 * lane + r;
            double p = 0.0;
#pragma unroll
            for (int j = 0; j < 8; ++j) p = ((c >> j) & 1) ? __dsub_rn(p, zb[j]) : __dadd_rn(p, zb[j]);
            // p is an exact multiple of 2^-24 with |p| < 2^26: exact as an integer.
            const int64_t pi = (int64_t)(p * 16777216.0);
            const bool neg = pi < 0;
            const int rep = neg ? c ^ 255 : c;
            key[r] = (neg ? -pi : pi) * 256 + (255 - rep);  // descending key: |proxy| desc, then id asc
        }
        sort128_desc(key, lane);
        // Representatives at positions 2 lane + r (r = 0, 1), ranks 2 lane + r; the
        // other members at ranks 255 - (2 lane + r).  Exclusive prefix of cluster
        // counts in rank order -> start rank P(c): the representatives' by a wave scan,
        // the other members' as everything before rank 128 plus the members of the
        // positions after theirs (the total less an inclusive scan).
        uint32_t cc[4];
        int cid[4];
#pragma unroll
        for (int r = 0; r < 2; ++r) {
            cid[r] = 255 - (int)(key[r] & 255);
            cid[2 + r] = cid[r] ^ 255;
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) cc[r] = s_cnt[sub][cid[r]];
        const uint32_t t0 = cc[0] + cc[1], t1 = cc[2] + cc[3];
        const uint32_t incl0 = wave_incl_sum(t0);
        const uint32_t incl1 = wave_incl_sum(t1);
        const uint32_t half = (uint32_t)__builtin_amdgcn_readlane((int)incl0, 63);  // counts of ranks 0..127
        const uint32_t tot1 = (uint32_t)__builtin_amdgcn_readlane((int)incl1, 63);
        uint32_t starts[4];
        starts[0] = incl0 - t0;
        starts[1] = starts[0] + cc[0];
        starts[2] = half + tot1 - (incl1 - t1 + cc[2]);
        starts[3] = half + tot1 - incl1;
        float m1 = 0.0f, m2 = 0.0f;  // sum of count * bonus and count * bonus^2 (an estimate's input)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const uint32_t start = starts[r];
            uint32_t bonus = 0;
#pragma unroll
            for (int l = kTierCount - 1; l >= 0; --l)
                if (start < a.cuts[l]) bonus = (uint32_t)(kTierCount - l);
            // Binary collisions: every admitted cluster (start below C_rho) scores 1.
            if (a.flags & kFlagBinary) bonus = bonus ? 1u : 0u;
            // The table is indexed like the stored ids, by slot.
            if (bonus) atomicOr(&s_lut[sub][id_slot((uint32_t)cid[r])], bonus << (8 * slot));
            m1 += (float)cc[r] * (float)bonus;
            m2 += (float)cc[r] * (float)(bonus * bonus);
        }
        m1 = wave_sum_f32(m1);
        m2 = wave_sum_f32(m2);
        if (lane == 0) {
            float* st = a.stats + (row * kB + b) * 2;
            st[0] = m1;
            st[1] = m2;
        }
    }
    __syncthreads();
    // Unused slots of the last quad keep bonus 0.
    a.lut[gq * (kB * kCentroids) + (4 * sg) * kCentroids + tid] = (&s_lut[0][0])[tid];
}

// ---------------------------------------------------------------- collision scan

constexpr int kColThreads = 256;
constexpr int kColKeysPerIter = 4 * kColThreads;  // 4 keys per thread per iteration
// Scores >= 1 go to one of two histogram copies picked by lane & 1 (fewer
// same-address atomics per instruction), one 32-bit counter per (copy, head, value);
// #{S >= 0} is the chunk's key count.
constexpr int kHistCopies = 2;
constexpr int kHistStride = 100;  // counters per (copy, head): values 0 .. kMaxScore
static_assert(kMaxScore < kHistStride, "histogram row");
// Word 3 of a gfx9 buffer descriptor for raw (untyped, unswizzled) access.
constexpr int kRawBufferWord3 = 0x00020000;
// A buffer offset past every range: the access is dropped (stores) or reads 0 (loads).
constexpr uint32_t kOffsetOutOfRange = 0x80000000u;

// Suffix sums of a 97-bin histogram held as (lo = bins 0..63 by lane, hi = bins
// 64..96 by lane < 33, 0 above): sfx[v] = sum_{u >= v} h[u], the total less the
// exclusive prefix, from two DPP scans.  Returns (sfx_lo, sfx_hi).
__device__ __forceinline__ void wave_suffix97(uint32_t lo, uint32_t hi, int lane, uint32_t* s_lo,
                                              uint32_t* s_hi) {
    const uint32_t ilo = wave_incl_sum(lo), ihi = wave_incl_sum(hi);
    const uint32_t tlo = (uint32_t)__builtin_amdgcn_readlane((int)ilo, 63);
    const uint32_t thi = (uint32_t)__builtin_amdgcn_readlane((int)ihi, 63);
    *s_lo = thi + tlo - (ilo - lo);
    *s_hi = thi - (ihi - hi);
}

__global__ __launch_bounds__(kColThreads) void collide_kernel(RetrieveArgs a) {
    __shared__ uint32_t s_lut[kB * kCentroids];
    __shared__ uint32_t s_hist[kHistCopies * 4 * kHistStride];
    __shared__ uint32_t s_floor[4];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    // Workgroups go to the 8 XCDs round-robin in dispatch order L.  With at least 4 rows
    // per XCD, XCD x scans every chunk of the rows gq = x (mod 8): a row's chunks and its
    // bonus table stay in one L2, and each XCD's id rows are still spread over the whole
    // array.  With fewer rows the plain order (XCD = chunk mod 8) keeps that spread; one
    // row per XCD, a contiguous stretch of ids, measured slower, as did giving each XCD a
    // contiguous eighth of a larger array.
    const uint32_t nx = gridDim.x;
    const uint32_t L = blockIdx.y * nx + blockIdx.x;
    int64_t chunk = blockIdx.x;
    int64_t gq = blockIdx.y;                   // (seq * hkv + kvh) * quads + quad
    if ((gridDim.y & 7u) == 0 && gridDim.y >= 32) {
        const uint32_t slot = L >> 3;
        chunk = slot % nx;
        gq = (L & 7u) + 8u * (slot / nx);
    }
    const int quad = (int)(gq % a.quads);
    const int64_t grp = gq / a.quads;          // seq * hkv + kvh
    const int seq = (int)(grp / a.hkv);
    const int kvh = (int)(grp % a.hkv);
    const int nh = min(4, a.g - 4 * quad);     // heads in this quad
    const int64_t row0 = (int64_t)seq * a.hq + kvh * a.g + 4 * quad;  // row of head 0 of the quad

    // The bonus table: every load in flight before the first LDS store.
    static_assert(kB * kCentroids / 4 == 4 * kColThreads, "four 16-byte table rows per thread");
    const uint4* lsrc = reinterpret_cast<const uint4*>(a.lut + gq * (kB * kCentroids)) + tid;
    const uint4 t0 = lsrc[0], t1 = lsrc[kColThreads], t2 = lsrc[2 * kColThreads], t3 = lsrc[3 * kColThreads];
    uint4* ldst = reinterpret_cast<uint4*>(s_lut) + tid;
    ldst[0] = t0;
    ldst[kColThreads] = t1;
    ldst[2 * kColThreads] = t2;
    ldst[3 * kColThreads] = t3;
    for (int i = tid; i < kHistCopies * 4 * kHistStride; i += kColThreads) s_hist[i] = 0;
    // Histogram floor of each head (a slot past the quad's last head scores 0: none).
    if (tid < 4) s_floor[tid] = tid < nh ? hist_floor(a.stats + (row0 + tid) * (kB * 2), a.n, a.c_eff, a.flags)
                                         : (uint32_t)kBins;
    __syncthreads();
    uint32_t floor_h[4];
#pragma unroll
    for (int h = 0; h < 4; ++h) floor_h[h] = s_floor[h];
    // The floors are the same in every chunk of a row; the first chunk records them
    // for the threshold kernel.
    if (chunk == 0 && tid < nh) a.thresh[(row0 + tid) * kThreshRow + 4] = (int32_t)s_floor[tid];

    const int64_t c0 = chunk * kChunk;
    const int64_t c1 = min(c0 + (int64_t)kChunk, a.n);
    const uint32_t nkeys = (uint32_t)(c1 - c0);

    // Buffer descriptors over the chunk: the id rows (nkeys x 16 bytes) and each head's
    // score bytes (nkeys, or none for a slot past the quad's last head).  The whole
    // offset goes in the VGPR operand, which the range check covers, so keys past the
    // chunk read 0 and store nothing without a branch.
    const __amdgpu_buffer_rsrc_t rid = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<uint8_t*>(a.ids + (grp * a.capacity + c0) * kB), 0, (int)(nkeys * kB), kRawBufferWord3);
    __amdgpu_buffer_rsrc_t rsc[4];
#pragma unroll
    for (int h = 0; h < 4; ++h)
        rsc[h] = __builtin_amdgcn_make_buffer_rsrc(a.score8 + (row0 + min(h, nh - 1)) * a.n_pad + c0, 0,
                                                   h < nh ? (int)nkeys : 0, kRawBufferWord3);
    uint32_t* hcopy = s_hist + (lane & (kHistCopies - 1)) * (4 * kHistStride);

    for (uint32_t base = 0; base < nkeys; base += kColKeysPerIter) {
        // Key base + tid + 256 j: one 16-byte id row per lane, a wave reads 1 KiB contiguous.
        uint4 w[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            typedef unsigned int v4u __attribute__((ext_vector_type(4)));
            const v4u t = __builtin_amdgcn_raw_buffer_load_b128(rid, (int)((base + tid + kColThreads * j) * kB), 0, 0);
            w[j] = make_uint4(t.x, t.y, t.z, t.w);
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const uint32_t i = base + tid + kColThreads * j;
            const uint32_t ww[4] = {w[j].x, w[j].y, w[j].z, w[j].w};
            uint32_t acc = 0;
#pragma unroll
            for (int b = 0; b < kB; ++b)
                acc += s_lut[b * kCentroids + ((ww[b >> 2] >> (8 * (b & 3))) & 0xffu)];
            const bool live = i < nkeys;
            acc = live ? acc : 0u;  // a key past the end scores 0 for every head
            // Exact per-value LDS histogram of the scores at or above the head's floor
            // (at least 1).  Slots of the last quad without a head have an all-zero
            // bonus table, so score 0, and floor 97.
#pragma unroll
            for (int h = 0; h < 4; ++h) {
                const uint32_t sh = (acc >> (8 * h)) & 0xffu;
                if (sh >= floor_h[h]) atomicAdd(hcopy + h * kHistStride + sh, 1u);
            }
            // A wave stores 64 consecutive score bytes of a head per instruction.
            const uint32_t off = live ? i : kOffsetOutOfRange;
#pragma unroll
            for (int h = 0; h < 4; ++h)
                __builtin_amdgcn_raw_buffer_store_b8((uint8_t)(acc >> (8 * h)), rsc[h], (int)off, 0, 0);
        }
    }

    __syncthreads();

    // Per-chunk suffix histogram of every head: sfx[v] = #{keys in chunk : S >= v} for
    // v = 0 and v >= floor; #{S >= floor} for 0 < v < floor.
    if (wave < nh) {
        const int h = wave;
        // Exact count of each value v >= 1: lane holds v = lane and v = 64 + lane.
        auto count_of = [&](int v) -> uint32_t {
            if (v < 1 || v > kMaxScore) return 0u;
            uint32_t t = 0;
#pragma unroll
            for (int c = 0; c < kHistCopies; ++c) t += s_hist[(c * 4 + h) * kHistStride + v];
            return t;
        };
        const uint32_t lo = count_of(lane);
        const uint32_t hi = count_of(64 + lane);
        uint32_t sl, sh;
        wave_suffix97(lo, hi, lane, &sl, &sh);  // exact for v >= floor
        if (lane == 0) sl = (uint32_t)(c1 - c0);
        uint32_t* dst = a.chunk_sfx + ((row0 + h) * a.n_chunks + chunk) * kSfx;
        dst[lane] = sl;
        if (lane < kSfx - 64) dst[64 + lane] = lane < kBins - 64 ? sh : 0u;
    }

}

// ---------------------------------------------------------------- threshold

constexpr int kThrThreads = 1024;  // one block per query head
constexpr int kThrWaves = kThrThreads / 64;

// theta = largest v with #{S >= v} >= C, from a whole-row suffix histogram held as
// (lo: v = lane, hi: v = 64 + lane), and gt = #{S > theta}.  Suffix counts fall with v
// and #{S >= 0} = n >= C.
__device__ __forceinline__ void theta_of(uint32_t ttl, uint32_t tth, uint32_t C, int lane, int* theta,
                                         uint32_t* gt) {
    const uint64_t ok_lo = __ballot(ttl >= C);
    const uint64_t ok_hi = __ballot(lane < kBins - 64 && tth >= C);
    const int th = ok_hi ? 64 + (63 - __clzll(ok_hi)) : (63 - __clzll(ok_lo));
    *gt = th + 1 < 64 ? __shfl(ttl, th + 1, 64) : __shfl(tth, th + 1 - 64, 64);
    *theta = th;
}

// kThrUnroll: chunks per wave and load round, the smallest power of two with
// 16 kThrUnroll >= n_chunks (at most 16: a 1M-key row in one round).
template <int kThrUnroll>
__global__ __launch_bounds__(kThrThreads) void threshold_kernel(RetrieveArgs a) {
    __shared__ uint32_t s_part[kThrWaves][2][64];
    __shared__ uint32_t s_wtot[2][kThrWaves];
    __shared__ uint32_t s_hist[kBins];
    __shared__ uint32_t s_cg[kThrWaves * kThrUnroll][2];  // per chunk: #{S > theta}, #{S == theta}
    __shared__ int s_theta;
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int64_t row = blockIdx.x;
    uint32_t* sfx = a.chunk_sfx + row * a.n_chunks * kSfx;
    int32_t* t = a.thresh + row * kThreshRow;
    const uint32_t fl = (uint32_t)t[4];  // the floor the scan used
    // Whole-row suffix histogram; lane holds v = lane and v = 64 + lane.  Wave w
    // sums chunks w, w + 16, ... with kThrUnroll chunks' loads in flight.  With at
    // most 16 kThrUnroll chunks that is one round, and each wave keeps its chunks'
    // histograms (chunk w + 16 u in tl[u], th[u]) for the chunk bases below.
    const bool one_round = a.n_chunks <= kThrWaves * kThrUnroll;
    uint32_t tl[kThrUnroll], th[kThrUnroll];
#pragma unroll
    for (int u = 0; u < kThrUnroll; ++u) tl[u] = th[u] = 0;
    for (int64_t c0 = wave; c0 < a.n_chunks; c0 += kThrWaves * kThrUnroll) {
        // Branch-free: every load is issued (clamped into the row) before the first
        // wait, and the entries past the row or past v = 97 are masked afterwards.
        uint32_t xl[kThrUnroll], xh[kThrUnroll];
#pragma unroll
        for (int u = 0; u < kThrUnroll; ++u) {
            const int64_t c = min(c0 + kThrWaves * u, a.n_chunks - 1);
            xl[u] = sfx[c * kSfx + lane];
            xh[u] = sfx[c * kSfx + 64 + min(lane, kSfx - 65)];
        }
#pragma unroll
        for (int u = 0; u < kThrUnroll; ++u) {
            const bool in = c0 + kThrWaves * u < a.n_chunks;
            tl[u] += in ? xl[u] : 0u;
            th[u] += in && lane < kSfx - 64 ? xh[u] : 0u;
        }
    }
    uint32_t sl = 0, sh = 0;
#pragma unroll
    for (int u = 0; u < kThrUnroll; ++u) { sl += tl[u]; sh += th[u]; }
    s_part[wave][0][lane] = sl;
    s_part[wave][1][lane] = sh;
    __syncthreads();
    const uint32_t C = (uint32_t)a.c_eff;
    // Every wave sums the wave totals and derives the same theta, so no second barrier
    // hands it out.
    uint32_t ttl = 0, tth = 0;
#pragma unroll
    for (int w = 0; w < kThrWaves; ++w) { ttl += s_part[w][0][lane]; tth += s_part[w][1][lane]; }
    // The counts are exact for v = 0 and v >= the floor the scan used (it left it in
    // t[4]).  With #{S >= floor} >= C (or floor 1) theta is found among them;
    // otherwise it lies below the floor and the row's scores are recounted.
    const uint32_t at_floor = fl < 64 ? __shfl(ttl, (int)fl, 64) : __shfl(tth, (int)fl - 64, 64);
    const int recount = fl > 1u && at_floor < C;
    int theta_w = 0;
    if (!recount) {
        uint32_t gt;
        theta_of(ttl, tth, C, lane, &theta_w, &gt);
        if (tid == 0) {
            t[0] = theta_w;
            t[1] = (int32_t)gt;
            t[2] = (int32_t)(C - gt);
            t[3] = (int32_t)C;
        }
    }
    if (tid == 0) {
        t[5] = recount;
        t[6] = t[7] = 0;
        s_theta = theta_w;
    }
    if (recount) {
        // Exact histogram of the row's stored scores, then theta from it.
        for (int i = tid; i < kBins; i += kThrThreads) s_hist[i] = 0;
        __syncthreads();
        const uint8_t* srow = a.score8 + row * a.n_pad;
        for (int64_t i = (int64_t)tid * 16; i < a.n; i += (int64_t)kThrThreads * 16) {
            const uint4 w = *reinterpret_cast<const uint4*>(srow + i);  // i + 16 <= n_pad
            const uint32_t ww[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
            for (int j = 0; j < 16; ++j)
                if (i + j < a.n) atomicAdd(&s_hist[(ww[j >> 2] >> (8 * (j & 3))) & 0xffu], 1u);
        }
        __syncthreads();
        if (wave == 0) {
            uint32_t sl, sh;
            wave_suffix97(s_hist[lane], lane < kBins - 64 ? s_hist[64 + lane] : 0u, lane, &sl, &sh);
            int theta;
            uint32_t gt;
            theta_of(sl, sh, C, lane, &theta, &gt);
            if (lane == 0) {
                t[0] = theta;
                t[1] = (int32_t)gt;
                t[2] = (int32_t)(C - gt);
                t[3] = (int32_t)C;
                s_theta = theta;
            }
        }
        __syncthreads();
        const int theta = s_theta;
        // Each chunk's exact #{S >= theta} and #{S > theta}, written over its suffix
        // entries theta and theta + 1 for the chunk bases below: wave w takes chunks
        // w, w + 16, ..., 16 bytes per lane and step.
        for (int64_t c = wave; c < a.n_chunks; c += kThrWaves) {
            uint32_t ge = 0, g = 0;
#pragma unroll
            for (int q = 0; q < kChunk / (64 * 16); ++q) {
                const int64_t i = c * kChunk + (int64_t)(q * 64 + lane) * 16;
                if (i < a.n) {
                    const uint4 w = *reinterpret_cast<const uint4*>(srow + i);
                    const uint32_t ww[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
                    for (int j = 0; j < 16; ++j) {
                        const int v = (int)((ww[j >> 2] >> (8 * (j & 3))) & 0xffu);
                        const bool in = i + j < a.n;
                        ge += (in && v >= theta) ? 1u : 0u;
                        g += (in && v > theta) ? 1u : 0u;
                    }
                }
            }
#pragma unroll
            for (int d = 1; d < 64; d <<= 1) {
                ge += __shfl_xor(ge, d, 64);
                g += __shfl_xor(g, d, 64);
            }
            if (lane == 0) {
                sfx[c * kSfx + theta] = ge;
                sfx[c * kSfx + theta + 1] = g;
            }
        }
        __syncthreads();
    }
    const int theta = recount ? s_theta : theta_w;  // the recount hands it out in s_theta
    // Each chunk's #{S > theta} and #{S == theta}: from the registers of the one-round
    // load (entries theta and theta + 1 of the chunk's suffix histogram), else (more
    // chunks, or the recount's entries) from memory below.
    const bool from_regs = one_round && !recount;
    if (from_regs) {
        const int th_s = __builtin_amdgcn_readfirstlane(theta);
#pragma unroll
        for (int u = 0; u < kThrUnroll; ++u) {
            const int64_t c = wave + kThrWaves * u;
            const uint32_t ge = th_s < 64 ? (uint32_t)__builtin_amdgcn_readlane((int)tl[u], th_s)
                                          : (uint32_t)__builtin_amdgcn_readlane((int)th[u], th_s - 64);
            const uint32_t g = th_s + 1 < 64 ? (uint32_t)__builtin_amdgcn_readlane((int)tl[u], th_s + 1)
                                              : (uint32_t)__builtin_amdgcn_readlane((int)th[u], th_s + 1 - 64);
            if (lane == 0 && c < a.n_chunks) {
                s_cg[c][0] = g;
                s_cg[c][1] = ge - g;
            }
        }
        __syncthreads();
    }
    // Keys with S > theta and S == theta in the chunks before each chunk.  Up to 64
    // chunks from the registers: one scan in wave 0.
    if (from_regs && a.n_chunks <= 64) {
        if (wave == 0) {
            const bool in = lane < a.n_chunks;
            const uint32_t g = in ? s_cg[lane][0] : 0u, e = in ? s_cg[lane][1] : 0u;
            const uint32_t ig = wave_incl_sum(g), ie = wave_incl_sum(e);
            if (in) {
                int32_t* cbp = a.chunk_base + (row * a.n_chunks + lane) * 2;
                cbp[0] = (int32_t)(ig - g);
                cbp[1] = (int32_t)(ie - e);
            }
        }
        return;
    }
    // Otherwise thread t takes chunk cb + t; wave scans, then a scan of the wave totals.
    uint32_t carry_g = 0, carry_e = 0;
    for (int64_t cb = 0; cb < a.n_chunks; cb += kThrThreads) {
        const int64_t c = cb + tid;
        uint32_t g = 0, e = 0;
        if (c < a.n_chunks) {
            if (from_regs) {
                g = s_cg[c][0];
                e = s_cg[c][1];
            } else {
                g = sfx[c * kSfx + theta + 1];
                e = sfx[c * kSfx + theta] - g;
            }
        }
        const uint32_t ig = wave_incl_sum(g);
        const uint32_t ie = wave_incl_sum(e);
        if (lane == 63) { s_wtot[0][wave] = ig; s_wtot[1][wave] = ie; }
        __syncthreads();
        uint32_t pg = 0, pe = 0, tg = 0, te = 0;
#pragma unroll
        for (int w = 0; w < kThrWaves; ++w) {
            const uint32_t xg = s_wtot[0][w], xe = s_wtot[1][w];
            if (w < wave) { pg += xg; pe += xe; }
            tg += xg;
            te += xe;
        }
        if (c < a.n_chunks) {
            int32_t* cbp = a.chunk_base + (row * a.n_chunks + c) * 2;
            cbp[0] = (int32_t)(carry_g + pg + ig - g);
            cbp[1] = (int32_t)(carry_e + pe + ie - e);
        }
        carry_g += tg;
        carry_e += te;
        __syncthreads();  // s_wtot is rewritten by the next round
    }
}

}  // namespace

hipError_t launch_query_lut(const RetrieveArgs& a, hipStream_t s) {
    const int64_t blocks = (int64_t)a.batch * a.hkv * a.quads * 4;
    const ProfEvents pe = prof_begin("query_lut");
    hipExtLaunchKernelGGL(query_lut_kernel, dim3((unsigned)blocks), dim3(kLutThreads), 0, s, pe.start, pe.stop, 0, a);
    return hipGetLastError();
}

hipError_t launch_collide(const RetrieveArgs& a, hipStream_t s) {
    const ProfEvents pe = prof_begin("collide");
    hipExtLaunchKernelGGL(collide_kernel, dim3((unsigned)a.n_chunks, (unsigned)(a.batch * a.hkv * a.quads)),
                       dim3(kColThreads), 0, s, pe.start, pe.stop, 0, a);
    return hipGetLastError();
}

hipError_t launch_threshold(const RetrieveArgs& a, hipStream_t s) {
    const int64_t rows = (int64_t)a.batch * a.hq;
    const ProfEvents pe = prof_begin("threshold");
    const dim3 grid((unsigned)rows), block(kThrThreads);
    if (a.n_chunks <= kThrWaves * 2)
        hipExtLaunchKernelGGL(threshold_kernel<2>, grid, block, 0, s, pe.start, pe.stop, 0, a);
    else if (a.n_chunks <= kThrWaves * 4)
        hipExtLaunchKernelGGL(threshold_kernel<4>, grid, block, 0, s, pe.start, pe.stop, 0, a);
    else if (a.n_chunks <= kThrWaves * 8)
        hipExtLaunchKernelGGL(threshold_kernel<8>, grid, block, 0, s, pe.start, pe.stop, 0, a);
    else
        hipExtLaunchKernelGGL(threshold_kernel<16>, grid, block, 0, s, pe.start, pe.stop, 0, a);
    return hipGetLastError();
}


}  // namespace pariskv
