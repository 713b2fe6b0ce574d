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
// compact_rerank_kernel: one block per (query head, 4096-key chunk).  Large
// grids take blocks of 128 threads (32 keys per thread), so that 16 blocks
// share a CU and their selection phases hide under each other's gathers; a
// grid that fits the chip in one round of 256-thread blocks takes those (16
// keys per thread), which halves each block's serial work.  It selects the chunk's candidates
// (all S > theta, then S == theta in ascending key order while the row's quota
// lasts), which occupy consecutive positions of the row's candidate list,
// writes them (and keeps them in LDS as 16-bit offsets in the chunk), and
// scores them at once: 8 lanes
// per candidate, lane l reads the 16-byte chunk l of the 128-byte record
// (codes of subspaces 2l, 2l+1 and their W), so one candidate is one fully
// used 128-byte line and a wave reads 8 lines per load instruction.  Lane l
// keeps the 16 query coordinates of its two subspaces in registers; the
// signed level table (16 floats) lives in LDS.
//
// topk_reg_kernel (at most 8 candidates per thread) and topk_lds_kernel (more):
// one block per list; the k-th largest estimate is found exactly on
// order-preserving uint32 keys, ties at it taken in candidate order, then an
// ordered compaction lists the winners in ascending key index (candidate order)
// without a sort.  The keys are held in registers (staged in LDS by the second
// kernel), binned linearly in value over [min, max] (the float bit patterns
// crowd into a few exponent prefixes), and the boundary bin is ranked by brute force when it holds
// at most 64 keys, else by 11/11/10-bit radix passes restricted to it.  A list
// is one query head's candidates (C <= 32768), or, in two passes, first every
// 4096-candidate slice of a head and then the concatenated winners of its slices
// (more than 32768 candidates, or more than 8192 for few heads).  With the
// attention fused (topk_reg_kernel), keys in bins above the boundary bin win
// whatever the rest of the selection finds, so once that bin is known each wave
// requests the K/V rows of up to 12 of them; those gathers run while the
// selection finishes, the rows wait in LDS, and the attention reads them there.

#include "attend_row.hpp"
#include "internal.hpp"

namespace pariskv {

namespace {

// One 4096-key chunk per block: 128 threads for large grids, 256 for grids of at
// most kRrWideGrid blocks (8 such blocks per CU on 256 CUs: one round).
constexpr int kRrWideGrid = 2048;
static_assert(kTopkPart >= PARISKV_MAX_TOPK, "a top-k slice holds at least k candidates");
static_assert(PARISKV_MAX_CAND / kTopkPart * PARISKV_MAX_TOPK <= 1024 * 32, "the slices' winners fit one block");
constexpr int kRrUnroll = 4;  // records in flight per lane

// Order-preserving uint32 key of a float (larger float, larger key; finite floats
// map above 0) and back.
__device__ __forceinline__ uint32_t order_key(float f) {
    const uint32_t u = __float_as_uint(f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float key_float(uint32_t k) {
    const uint32_t u = (k & 0x80000000u) ? (k & 0x7fffffffu) : ~k;
    return __uint_as_float(u);
}

// Compaction of one chunk's candidates (Stage I selection) fused with their
// RSQ-IP rerank (Stage II).  The selected keys of a chunk hold consecutive
// positions [P0, P0 + m) of the row's ascending candidate list, so the block
// writes them to `cand`, keeps them in LDS and scores them right away.
template <int kRrThreads>
__global__ __launch_bounds__(kRrThreads) void compact_rerank_kernel(RetrieveArgs a) {
    constexpr int kKpt = kChunk / kRrThreads;   // keys per thread
    constexpr int kRrSlots = kRrThreads / 8;    // candidates reranked per block iteration
    static_assert(kKpt % 16 == 0 && kKpt <= 32, "whole 16-byte score loads, one 32-bit mask");
    __shared__ float s_tab[16];
    __shared__ uint32_t s_wsum[kRrThreads / 64];
    // The selected keys as offsets in the chunk (2 bytes each, so 16 blocks fit a CU).
    __shared__ uint16_t s_list[kChunk];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int64_t chunk = blockIdx.x;
    const int64_t row = blockIdx.y;  // seq * hq + head
    const int seq = (int)(row / a.hq);
    const int hq = (int)(row % a.hq);
    const int64_t grp = (int64_t)seq * a.hkv + hq / a.g;

    // Everything this block reads up front.
    const int32_t* th = a.thresh + row * kThreshRow;
    const uint32_t theta = (uint32_t)th[0];
    const uint32_t quota = (uint32_t)th[2];
    const int32_t* cb = a.chunk_base + (row * a.n_chunks + chunk) * 2;
    const uint32_t base_g = (uint32_t)cb[0], base_e = (uint32_t)cb[1];
    // This thread's kKpt keys; score rows are padded to a multiple of 64 bytes, so a
    // load that starts before n stays inside the row.
    const int64_t i0 = chunk * kChunk + kKpt * tid;
    uint4 sw[kKpt / 16];
#pragma unroll
    for (int u = 0; u < kKpt / 16; ++u) {
        sw[u] = make_uint4(0, 0, 0, 0);
        if (i0 + 16 * u < a.n) sw[u] = *reinterpret_cast<const uint4*>(a.score8 + row * a.n_pad + i0 + 16 * u);
    }
    const int l = tid & 7;
    float z[16];
    {
        const float4* zp = reinterpret_cast<const float4*>(a.zq + row * kD + 16 * l);
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const float4 t = zp[v];
            z[4 * v] = t.x; z[4 * v + 1] = t.y; z[4 * v + 2] = t.z; z[4 * v + 3] = t.w;
        }
    }
    if (tid < 16) s_tab[tid] = (tid & 8) ? -a.qc.a32[tid & 7] : a.qc.a32[tid & 7];

    // ---- compaction: all S > theta, and S == theta while the row's quota lasts.
    uint32_t gmask = 0, emask = 0;
    {
        uint32_t ww[kKpt / 4];
#pragma unroll
        for (int u = 0; u < kKpt / 16; ++u) {
            ww[4 * u] = sw[u].x;
            ww[4 * u + 1] = sw[u].y;
            ww[4 * u + 2] = sw[u].z;
            ww[4 * u + 3] = sw[u].w;
        }
#pragma unroll
        for (int j = 0; j < kKpt; ++j) {
            const uint32_t sv = (ww[j >> 2] >> (8 * (j & 3))) & 0xffu;
            const bool in = i0 + j < a.n;
            gmask |= (in && sv > theta ? 1u : 0u) << j;
            emask |= (in && sv == theta ? 1u : 0u) << j;
        }
    }
    // Packed (gt, eq) counts: each at most 4096 per chunk, 16 bits each.
    const uint32_t mine = (uint32_t)__popc(gmask) | ((uint32_t)__popc(emask) << 16);
    const uint32_t incl = wave_incl_sum(mine);
    if (lane == 63) s_wsum[wave] = incl;
    __syncthreads();
    uint32_t pre = incl - mine, tot = 0;
#pragma unroll
    for (int w = 0; w < kRrThreads / 64; ++w) {
        const uint32_t x = s_wsum[w];
        if (w < wave) pre += x;
        tot += x;
    }
    const uint32_t P0 = base_g + min(base_e, quota);
    const uint32_t m = (tot & 0xffffu) + (min(base_e + (tot >> 16), quota) - min(base_e, quota));
    const uint32_t gb = base_g + (pre & 0xffffu);  // S > theta keys before this thread's keys
    const uint32_t eb = base_e + (pre >> 16);      // S == theta keys before them
    int32_t* cand = a.cand + row * a.n_cand;
    const uint32_t c_eff = (uint32_t)a.c_eff;
    // Visit only the selected keys (about 1 in 16); a key's place in the row's
    // ascending list is the number of taken keys before it.
    for (uint32_t sel = gmask | emask; sel; sel &= sel - 1u) {
        const int j = __builtin_ctz(sel);
        const uint32_t below = (1u << j) - 1u;
        const uint32_t g = gb + (uint32_t)__popc(gmask & below);
        const uint32_t e = eb + (uint32_t)__popc(emask & below);
        uint32_t p = 0xffffffffu;
        if ((gmask >> j) & 1u)
            p = g + min(e, quota);
        else if (e < quota)
            p = g + e;
        if (p < c_eff) {
            const int32_t key = (int32_t)i0 + j;
            cand[p] = key;
            s_list[p - P0] = (uint16_t)(kKpt * tid + j);
        }
    }
    __syncthreads();

    // ---- RSQ-IP: 8 lanes per candidate, lane l reads record chunk l (subspaces 2l, 2l+1).
    const int slot = tid >> 3;
    float* out = a.cand_score + row * a.n_cand + P0;
    const uint4* rec = reinterpret_cast<const uint4*>(a.rec + grp * a.capacity * kRec);
    const uint32_t two = 2u;
    const char* tab = reinterpret_cast<const char*>(s_tab);
    auto entry = [&](uint32_t byte_off) { return *reinterpret_cast<const float*>(tab + byte_off); };
#pragma unroll 1
    for (uint32_t it = 0; it < m; it += kRrSlots * kRrUnroll) {
        uint4 rc[kRrUnroll];
#pragma unroll
        for (int u = 0; u < kRrUnroll; ++u) {
            // Past the end, re-read the last candidate; its result is not stored.
            const uint32_t ci = min(it + u * kRrSlots + slot, m - 1u);
            rc[u] = rec[((uint64_t)chunk * kChunk + s_list[ci]) * (kRec / 16) + l];
        }
#pragma unroll
        for (int u = 0; u < kRrUnroll; ++u) {
            // Code of coordinate 2k in the low nibble of byte k, of 2k+1 in the high
            // nibble: one mask per word, then one byte-select shift per lookup.
            const uint32_t e0 = rc[u].x & 0x0f0f0f0fu, o0 = rc[u].x & 0xf0f0f0f0u;
            const uint32_t e1 = rc[u].y & 0x0f0f0f0fu, o1 = rc[u].y & 0xf0f0f0f0u;
            float d0 = 0.f, d1 = 0.f;
            d0 += entry(byte_shl2<0>(e0, two)) * z[0];
            d0 += entry(byte_shr2<0>(o0, two)) * z[1];
            d0 += entry(byte_shl2<1>(e0, two)) * z[2];
            d0 += entry(byte_shr2<1>(o0, two)) * z[3];
            d0 += entry(byte_shl2<2>(e0, two)) * z[4];
            d0 += entry(byte_shr2<2>(o0, two)) * z[5];
            d0 += entry(byte_shl2<3>(e0, two)) * z[6];
            d0 += entry(byte_shr2<3>(o0, two)) * z[7];
            d1 += entry(byte_shl2<0>(e1, two)) * z[8];
            d1 += entry(byte_shr2<0>(o1, two)) * z[9];
            d1 += entry(byte_shl2<1>(e1, two)) * z[10];
            d1 += entry(byte_shr2<1>(o1, two)) * z[11];
            d1 += entry(byte_shl2<2>(e1, two)) * z[12];
            d1 += entry(byte_shr2<2>(o1, two)) * z[13];
            d1 += entry(byte_shl2<3>(e1, two)) * z[14];
            d1 += entry(byte_shr2<3>(o1, two)) * z[15];
            float part = __uint_as_float(rc[u].z) * d0 + __uint_as_float(rc[u].w) * d1;
            part += __uint_as_float(lane_xor(__float_as_uint(part), 1, lane));
            part += __uint_as_float(lane_xor(__float_as_uint(part), 2, lane));
            part += __uint_as_float(lane_xor(__float_as_uint(part), 4, lane));
            // + 0.0f turns -0 into +0, so equal estimates compare equal in the top-k keys.
            const uint32_t ci = it + u * kRrSlots + slot;
            if (l == 0 && ci < m) out[ci] = part + 0.0f;
        }
    }
}

// ---------------------------------------------------------------- top-k


// Shared by both top-k kernels, run by one whole wave: the digit holding the
// need-th largest element of a histogram of NB bins.  Lane L owns bins
// NB-1-L*PER .. NB-PER-L*PER (descending); a scan of the lane totals finds the
// lane whose bins hold the crossing, then PER lanes take its bins from the
// largest down and a second scan finds the bin.  Writes s_digit and s_need (the
// rank inside that bin).  Needs 1 <= need <= the histogram's total.
template <int NB>
__device__ __forceinline__ void find_digit(const uint32_t* hist, uint32_t need, int lane, uint32_t* s_digit,
                                           uint32_t* s_need) {
    constexpr int PER = NB / 64;
    static_assert(PER >= 1 && PER <= 64, "bins per lane");
    const uint32_t* h = hist + NB - PER * (lane + 1);  // this lane's bins, ascending
    uint32_t tot = 0;
#pragma unroll 8
    for (int r = 0; r < PER; ++r) tot += h[r];
    const uint32_t above = wave_incl_sum(tot) - tot;  // elements with a larger digit
    const int L = (int)__builtin_ctzll(__ballot(above < need && above + tot >= need));
    const uint32_t above_L = __shfl(above, L, 64);
    const int bin = NB - PER * (L + 1) + (PER - 1 - lane);  // lane r < PER: L's bins, largest first
    const uint32_t c = lane < PER ? hist[bin] : 0u;
    const uint32_t ci = wave_incl_sum(c);
    if (lane == (int)__builtin_ctzll(__ballot(lane < PER && above_L + ci >= need))) {
        *s_digit = (uint32_t)bin;
        *s_need = need - (above_L + ci - c);
    }
}

// Top-k for C <= TH * EPT held in LDS (more than 8 candidates per thread).  Scores and candidate indices are staged
// with coalesced 16-byte loads; each thread then owns EPT consecutive candidates.
// Exact radix select with 11-bit digits taken from the top of the occupied
// [min, max] key range, then an ordered compaction (ascending key index).
template <int TH, int EPT, bool kAttend>
__global__ __launch_bounds__(TH) void topk_lds_kernel(RetrieveArgs a) {
    constexpr int kWaves = TH / 64;
    constexpr int kCap = TH * EPT;
    constexpr int kNB = 2048;
    // Up to 16 keys per thread the candidate indices are staged in LDS too (the
    // winners then read them without a global round trip); beyond that they are
    // read back from global memory for the k winners only.
    constexpr bool kStageIdx = EPT <= 16;
    // One LDS area: region A = staged keys (+ indices), region B = two histograms.
    // With kAttend the winners list reuses B once the histograms are done, and
    // the attention's per-slot state reuses A once the winners are out.
    constexpr size_t kA0 = (size_t)kCap * 4 * (kStageIdx ? 2 : 1);
    constexpr size_t kA = kAttend && kA0 < sizeof(AttendScratch) ? sizeof(AttendScratch) : kA0;
    constexpr size_t kBytes = kA + 2 * kNB * 4;
    static_assert(!kAttend || 2 * kNB * 4 >= kMaxAttendRows * 4, "the attention list fits in region B");
    __shared__ __align__(16) unsigned char s_raw[kBytes];
    uint32_t* s_key = reinterpret_cast<uint32_t*>(s_raw);
    int32_t* s_idx = reinterpret_cast<int32_t*>(s_raw + (size_t)kCap * 4);
    uint32_t (*s_hist)[kNB] = reinterpret_cast<uint32_t (*)[kNB]>(s_raw + kA);
    int32_t* s_win = reinterpret_cast<int32_t*>(s_raw + kA);
    __shared__ uint32_t s_w[kWaves];
    __shared__ uint32_t s_mm[2][kWaves];
    __shared__ uint32_t s_digit, s_need, s_nsmall;
    __shared__ uint32_t s_small[64];
    // With kAttend the winners' estimates wait here until the attention is done.
    __shared__ float s_wsc[kAttend ? PARISKV_MAX_TOPK : 1];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    // This block's list: part blk % tk_parts of row blk / tk_parts (see RetrieveArgs).
    const int64_t blk = blockIdx.x;
    const int64_t row = blk / a.tk_parts;
    const int64_t off = (blk % a.tk_parts) * (int64_t)a.tk_part_len;
    const int C = (int)min((int64_t)a.tk_part_len, a.tk_c - off);
    const int kk = min(a.top_k, C);
    const float* sc = a.tk_score + row * a.tk_stride + off;
    const int32_t* cand = a.tk_idx + row * a.tk_stride + off;
    if (tid == 0) s_nsmall = 0;

    // With kAttend, this thread's part of the query, requested first.
    const uint4 qv = kAttend ? attend_query_part(static_cast<const __half*>(a.q) + row * kD)
                             : make_uint4(0, 0, 0, 0);

    // Staging of the estimates as order-preserving keys (and of the candidate
    // indices): every load of the thread is issued before the first LDS store, and
    // the smallest and largest valid keys are reduced on the way.  The arrays start
    // 256-byte aligned, so 16-byte loads are taken when the row stride and the part's
    // offset are multiples of 4 (the list then starts 16-byte aligned); slots past
    // the list re-read the row's last 16 bytes and are masked.
    uint32_t kmin = 0xffffffffu, kmax = 0u;
    if (((a.tk_stride | off) & 3) == 0) {
        constexpr int kIt = kCap / 4 / TH;
        const int nq = (int)((a.tk_stride - off) >> 2);
        float4 f[kIt];
        int4 ix[kIt];
#pragma unroll
        for (int it = 0; it < kIt; ++it) {
            const int p4 = min(tid + it * TH, nq - 1);
            f[it] = reinterpret_cast<const float4*>(sc)[p4];
            if (kStageIdx) ix[it] = reinterpret_cast<const int4*>(cand)[p4];
        }
#pragma unroll
        for (int it = 0; it < kIt; ++it) {
            const int p = 4 * (tid + it * TH);
            const float fq[4] = {f[it].x, f[it].y, f[it].z, f[it].w};
            uint32_t k4[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                k4[q] = p + q < C ? order_key(fq[q]) : 0u;  // valid keys are all > 0
                if (k4[q] != 0u) { kmin = min(kmin, k4[q]); kmax = max(kmax, k4[q]); }
            }
            reinterpret_cast<uint4*>(s_key)[tid + it * TH] = make_uint4(k4[0], k4[1], k4[2], k4[3]);
            if (kStageIdx)
                reinterpret_cast<int4*>(s_idx)[tid + it * TH] =
                    make_int4(p < C ? ix[it].x : -1, p + 1 < C ? ix[it].y : -1, p + 2 < C ? ix[it].z : -1,
                              p + 3 < C ? ix[it].w : -1);
        }
    } else {
        for (int p = tid; p < kCap; p += TH) {
            const uint32_t k1 = p < C ? order_key(sc[p]) : 0u;
            if (k1 != 0u) { kmin = min(kmin, k1); kmax = max(kmax, k1); }
            s_key[p] = k1;
            if (kStageIdx) s_idx[p] = p < C ? cand[p] : -1;
        }
    }
    kmin = wave_min_u32(kmin);
    kmax = wave_max_u32(kmax);
    if (lane == 0) { s_mm[0][wave] = kmin; s_mm[1][wave] = kmax; }
    for (int i = tid; i < 2 * kNB; i += TH) (&s_hist[0][0])[i] = 0;
    __syncthreads();

    // Each thread then owns EPT consecutive candidates.
    uint32_t key[EPT];
#pragma unroll
    for (int e4 = 0; e4 < EPT / 4; ++e4) {
        const uint4 kv = reinterpret_cast<const uint4*>(s_key)[tid * (EPT / 4) + e4];
        key[4 * e4] = kv.x; key[4 * e4 + 1] = kv.y; key[4 * e4 + 2] = kv.z; key[4 * e4 + 3] = kv.w;
    }
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
        kmin = min(kmin, s_mm[0][w]);
        kmax = max(kmax, s_mm[1][w]);
    }

    // Pass 0: 2048 bins linear in the score over [min, max].  The float bit
    // patterns of the scores are concentrated in few sign/exponent prefixes, so
    // value-linear bins spread the counts (and the atomics) far better.  The bin
    // index is a non-decreasing function of the score, so the keys of a higher
    // bin are all larger.
    const float fmin = key_float(kmin), fmax = key_float(kmax);
    const float frange = fmax - fmin;
    float inv = frange > 0.0f ? (float)kNB / frange : 0.0f;
    if (!(inv < 1e30f)) inv = 0.0f;  // a range that under- or overflows: one bin
    auto bin_of = [&](uint32_t k) -> uint32_t {
        return (uint32_t)fminf((float)(kNB - 1), (key_float(k) - fmin) * inv);
    };
#pragma unroll
    for (int e = 0; e < EPT; ++e)
        if (key[e] != 0u) atomicAdd(&s_hist[0][bin_of(key[e])], 1u);
    __syncthreads();
    if (wave == 0) find_digit<kNB>(s_hist[0], (uint32_t)kk, lane, &s_digit, &s_need);
    __syncthreads();
    const uint32_t bsel = s_digit;       // bin holding the kk-th largest key
    uint32_t need = s_need;              // its rank (from the top) inside that bin
    const uint32_t in_bin = s_hist[0][bsel];
    uint32_t T, quota;
    if (in_bin <= 64) {
        // Few keys in the bin: gather them and rank them by brute force in one wave.
#pragma unroll
        for (int e = 0; e < EPT; ++e)
            if (key[e] != 0u && bin_of(key[e]) == bsel) s_small[atomicAdd(&s_nsmall, 1u)] = key[e];
        __syncthreads();
        if (wave == 0) {
            const uint32_t kl = lane < (int)in_bin ? s_small[lane] : 0u;
            uint32_t gt = 0, eq = 0;
            for (uint32_t j = 0; j < in_bin; ++j) {
                const uint32_t kj = s_small[j];
                gt += kj > kl ? 1u : 0u;
                eq += kj == kl ? 1u : 0u;
            }
            const bool hit = lane < (int)in_bin && gt < need && need <= gt + eq;
            const uint64_t hits = __ballot(hit);
            if (hit && lane == __builtin_ctzll(hits)) {
                s_digit = kl;
                s_need = need - gt;
            }
        }
        __syncthreads();
        T = s_digit;
        quota = s_need;
    } else {
        // Exact radix select on the full key restricted to the bin: 11, 11, 10 bits.
        uint32_t prefix = 0, mask = 0;
        int shift = 21;
#pragma unroll 1
        for (int pass = 1; pass <= 3; ++pass) {
            uint32_t* hist = s_hist[pass & 1];
#pragma unroll
            for (int e = 0; e < EPT; ++e)
                if (key[e] != 0u && (key[e] & mask) == prefix && bin_of(key[e]) == bsel)
                    atomicAdd(&hist[(key[e] >> shift) & (kNB - 1)], 1u);
            __syncthreads();
            if (wave == 0) find_digit<kNB>(hist, need, lane, &s_digit, &s_need);
            // The other buffer was read in the previous pass; clear it for the next one.
            for (int i = tid; i < kNB; i += TH) s_hist[(pass + 1) & 1][i] = 0;
            __syncthreads();
            prefix |= s_digit << shift;
            mask |= (uint32_t)(kNB - 1) << shift;
            need = s_need;
            shift = shift >= 11 ? shift - 11 : 0;
        }
        T = prefix;     // the kk-th largest key value
        quota = need;   // how many keys equal to T are taken (lowest indices)
    }

    // Ordered compaction: an element's output slot is (#keys > T before it) +
    // min(#keys == T before it, quota), which lists the winners by ascending index.
    uint32_t ng = 0, ne = 0;
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
        ng += (key[e] > T) ? 1u : 0u;
        ne += (key[e] == T && key[e] != 0u) ? 1u : 0u;
    }
    const uint32_t mine = ng | (ne << 16);
    // This thread's candidate indices, read before they are needed.
    int32_t widx[EPT];
    if (kStageIdx) {
#pragma unroll
        for (int e4 = 0; e4 < EPT / 4; ++e4) {
            const int4 v4 = reinterpret_cast<const int4*>(s_idx)[tid * (EPT / 4) + e4];
            widx[4 * e4] = v4.x; widx[4 * e4 + 1] = v4.y; widx[4 * e4 + 2] = v4.z; widx[4 * e4 + 3] = v4.w;
        }
    }
    const uint32_t incl = wave_incl_sum(mine);
    if (lane == 63) s_w[wave] = incl;
    __syncthreads();
    uint32_t pre = incl - mine;
#pragma unroll
    for (int w = 0; w < kWaves; ++w)
        if (w < wave) pre += s_w[w];
    uint32_t gb = pre & 0xffffu, eb = pre >> 16;
    int32_t* oi = a.tk_out_idx + blk * a.top_k;
    float* os = a.tk_out_score ? a.tk_out_score + blk * a.top_k : nullptr;
    // With kAttend the attention list in region B is Sink rows, then Local +
    // Update Buffer rows (nd in all), then the winners at their cache rows
    // (retr_begin + key; the host checked they stay below dense_begin), and the
    // outputs are written after the attention, so that its first loads do not
    // wait behind these stores.
    const int nd = kAttend ? (int)a.win.dense_rows() : 0;
#pragma unroll
    for (int e = 0; e < EPT; ++e) {
        uint32_t p = 0xffffffffu;
        if (key[e] > T) {
            p = gb + min(eb, quota);
            ++gb;
        } else if (key[e] == T && key[e] != 0u) {
            if (eb < quota) p = gb + eb;
            ++eb;
        }
        if (p < (uint32_t)kk) {
            const int32_t win = kStageIdx ? widx[e] : cand[tid * EPT + e];
            if (kAttend) {
                s_win[nd + p] = (int32_t)(a.win.retr_begin + win);
                s_wsc[p] = key_float(key[e]);
            } else {
                oi[p] = win;
                if (os) os[p] = key_float(key[e]);
            }
        }
    }
    if (!kAttend) {
        for (int r = kk + tid; r < a.top_k; r += TH) {
            oi[r] = -1;
            if (os) os[r] = -__builtin_huge_valf();
        }
    }
    if (kAttend) {
        // Attention over the dense rows and the kk winners (Eqs. approx_weight,
        // approx_output), from LDS.  Region B is free once the compaction runs.
        for (int r = tid; r < nd; r += TH) s_win[r] = a.win.dense_entry(r);
        __syncthreads();
        const int seq = (int)(row / a.hq);
        const int h = (int)(row % a.hq);
        const int64_t kvrow0 = ((int64_t)seq * a.hkv + h / a.g) * a.kv_capacity;
        const bool wc = a.win.win_capacity > 0;
        const int64_t wrow0 = wc ? ((int64_t)seq * a.hkv + h / a.g) * a.win.win_capacity : kvrow0;
        attend_row(qv, static_cast<const __half*>(a.K) + kvrow0 * kD,
                   static_cast<const __half*>(a.V) + kvrow0 * kD, a.kv_capacity,
                   static_cast<const __half*>(wc ? a.Kw : a.K) + wrow0 * kD,
                   static_cast<const __half*>(wc ? a.Vw : a.V) + wrow0 * kD, a.win.win_capacity,
                   s_win, nd + kk, a.scale,
                   a.attn_out + row * kD, *reinterpret_cast<AttendScratch*>(s_raw));
        // The winners in ascending key index, then the padding.
        for (int r = tid; r < a.top_k; r += TH) {
            const bool w = r < kk;
            oi[r] = w ? (int32_t)((int64_t)s_win[nd + r] - a.win.retr_begin) : -1;
            if (os) os[r] = w ? s_wsc[r] : -__builtin_huge_valf();
        }
    }
}

// Top-k for C <= TH * EPT <= 8192 candidates, held in registers: thread t owns the 4-candidate
// groups at positions 4 (t + j TH) .. 4 (t + j TH) + 3 for j < EPT / 4, read with
// coalesced 16-byte loads.  Exact selection on order-preserving uint32 keys: one
// histogram pass with 2048 bins linear in the estimate over [min, max], then the
// boundary bin ranked by brute force (at most 64 keys) or by 11/11/10-bit radix
// passes restricted to it; ties at the k-th key taken in candidate order.  An ordered
// compaction (a block scan per group of positions) then lists the winners in
// ascending key index without a sort.
template <int TH, int EPT, bool kAttend>
__global__ __launch_bounds__(TH) void topk_reg_kernel(RetrieveArgs a) {
    constexpr int kWaves = TH / 64;
    constexpr int kIt = EPT / 4;   // 4-candidate groups per thread
    constexpr int kNB = 2048;
    // LDS: region A = the attention's per-slot state (kAttend), region B = two
    // histograms, whose place the attention list takes once they are done.
    constexpr size_t kA = kAttend ? sizeof(AttendScratch) : 0;
    constexpr size_t kBytes = kA + 2 * kNB * 4;
    static_assert(!kAttend || 2 * kNB * 4 >= kMaxAttendRows * 4, "the attention list fits in region B");
    static_assert(EPT % 4 == 0 && EPT <= 8, "whole 4-candidate groups, few enough to stay in registers");
    __shared__ __align__(16) unsigned char s_raw[kBytes];
    uint32_t (*s_hist)[kNB] = reinterpret_cast<uint32_t (*)[kNB]>(s_raw + kA);
    int32_t* s_win = reinterpret_cast<int32_t*>(s_raw + kA);
    __shared__ uint32_t s_w[kIt][kWaves];
    __shared__ uint32_t s_mm[2][kWaves];
    __shared__ uint32_t s_digit, s_need, s_nsmall;
    __shared__ uint32_t s_small[64];
    // With kAttend the winners' estimates wait here until the attention is done.
    __shared__ float s_wsc[kAttend ? PARISKV_MAX_TOPK : 1];
    __shared__ int32_t s_dump[kAttend ? TH : 1];  // a word per thread for non-winners' stores
    // With kAttend: K/V rows of up to kPf sure winners per wave, requested as soon as
    // the boundary bin is known (see below), and their cache rows.
    constexpr int kPf = 12;
    __shared__ uint4 s_prow[kAttend ? kWaves * kPf * 32 : 1];
    __shared__ __align__(16) int32_t s_pfrow[kAttend ? kWaves : 1][kPf];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    // This block's list: part blk % tk_parts of row blk / tk_parts (see RetrieveArgs).
    const int64_t blk = blockIdx.x;
    const int64_t row = blk / a.tk_parts;
    const int64_t off = (blk % a.tk_parts) * (int64_t)a.tk_part_len;
    const int C = (int)min((int64_t)a.tk_part_len, a.tk_c - off);
    const int kk = min(a.top_k, C);
    const float* sc = a.tk_score + row * a.tk_stride + off;
    const int32_t* cand = a.tk_idx + row * a.tk_stride + off;
    if (tid == 0) s_nsmall = 0;

    uint32_t kmin = 0xffffffffu, kmax = 0u;

    // The estimates as keys (0 past the list; valid keys are all > 0) and the
    // candidate indices.  The arrays start 256-byte aligned, so 16-byte loads are
    // taken when the row stride and the part's offset are multiples of 4 (the list
    // then starts 16-byte aligned); groups past the list re-read the row's last 16
    // bytes and are masked.  Otherwise every candidate is read on its own.
    uint32_t key[EPT];
    int32_t widx[EPT];
    if (((a.tk_stride | off) & 3) == 0) {
        const int nq = (int)((a.tk_stride - off) >> 2);
        float4 f[kIt];
        int4 ix[kIt];
#pragma unroll
        for (int it = 0; it < kIt; ++it)
            f[it] = reinterpret_cast<const float4*>(sc)[min(tid + it * TH, nq - 1)];
#pragma unroll
        for (int it = 0; it < kIt; ++it)
            ix[it] = reinterpret_cast<const int4*>(cand)[min(tid + it * TH, nq - 1)];
        // The estimates are needed first (the indices only after the digit search):
        // an empty asm that reads them keeps each 16-byte load whole and makes the
        // one wait here cover just them.
#pragma unroll
        for (int it = 0; it < kIt; ++it) asm volatile("" ::"v"(f[it].x), "v"(f[it].y), "v"(f[it].z), "v"(f[it].w));
#pragma unroll
        for (int it = 0; it < kIt; ++it) {
            const int p = 4 * (tid + it * TH);
            key[4 * it] = p < C ? order_key(f[it].x) : 0u;
            key[4 * it + 1] = p + 1 < C ? order_key(f[it].y) : 0u;
            key[4 * it + 2] = p + 2 < C ? order_key(f[it].z) : 0u;
            key[4 * it + 3] = p + 3 < C ? order_key(f[it].w) : 0u;
            widx[4 * it] = ix[it].x;
            widx[4 * it + 1] = ix[it].y;
            widx[4 * it + 2] = ix[it].z;
            widx[4 * it + 3] = ix[it].w;
        }
    } else {
#pragma unroll
        for (int e = 0; e < EPT; ++e) {
            const int p = 4 * (tid + (e >> 2) * TH) + (e & 3);
            key[e] = p < C ? order_key(sc[p]) : 0u;
            widx[e] = p < C ? cand[p] : -1;
        }
    }
    // With kAttend, this thread's part of the query (needed only by the attention).
    const uint4 qv = kAttend ? attend_query_part(static_cast<const __half*>(a.q) + row * kD)
                             : make_uint4(0, 0, 0, 0);
    for (int i = tid; i < 2 * kNB; i += TH) (&s_hist[0][0])[i] = 0;
#pragma unroll
    for (int e = 0; e < EPT; ++e)
        if (key[e] != 0u) { kmin = min(kmin, key[e]); kmax = max(kmax, key[e]); }
    kmin = wave_min_u32(kmin);
    kmax = wave_max_u32(kmax);
    if (lane == 0) { s_mm[0][wave] = kmin; s_mm[1][wave] = kmax; }
    __syncthreads();
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
        kmin = min(kmin, s_mm[0][w]);
        kmax = max(kmax, s_mm[1][w]);
    }

    // Pass 0: 2048 bins linear in the score over [min, max].  The float bit
    // patterns of the scores are concentrated in few sign/exponent prefixes, so
    // value-linear bins spread the counts (and the atomics) far better.  The bin
    // index is a non-decreasing function of the score, so the keys of a higher
    // bin are all larger.
    const float fmin = key_float(kmin), fmax = key_float(kmax);
    const float frange = fmax - fmin;
    float inv = frange > 0.0f ? (float)kNB / frange : 0.0f;
    if (!(inv < 1e30f)) inv = 0.0f;  // a range that under- or overflows: one bin
    auto bin_of = [&](uint32_t k) -> uint32_t {
        return (uint32_t)fminf((float)(kNB - 1), (key_float(k) - fmin) * inv);
    };
#pragma unroll
    for (int e = 0; e < EPT; ++e)
        if (key[e] != 0u) atomicAdd(&s_hist[0][bin_of(key[e])], 1u);
    __syncthreads();
    if (wave == 0) find_digit<kNB>(s_hist[0], (uint32_t)kk, lane, &s_digit, &s_need);
    __syncthreads();
    const uint32_t bsel = s_digit;       // bin holding the kk-th largest key
    uint32_t need = s_need;              // its rank (from the top) inside that bin
    const uint32_t in_bin = s_hist[0][bsel];
    const int32_t retr0 = (int32_t)a.win.retr_begin;  // below kv_capacity <= 2^30 - 1 (host-checked)
    // KV group of the row: row = seq hq + h with hq = hkv g, so seq hkv + h / g = row / g.
    const int64_t kvrow0 = kAttend ? (int64_t)((int)row / a.g) * a.kv_capacity : 0;

    // With kAttend: a key in a bin above bsel wins whatever the rest of the selection
    // finds.  Each lane offers the first such key among its first kPfKeys, and each
    // wave requests the K/V rows of the first kPf lanes that offer one into registers
    // now, so that these gathers overlap the rest of the selection (a barrier does not
    // wait for them); they go to LDS just before the attention, which reads them from
    // there (listed as -2 - LDS row).  The bin test is the bin's own arithmetic: the
    // bin is the truncated (f - fmin) inv, so bin > bsel iff that product >= bsel + 1.
    constexpr int kPfKeys = EPT < 4 ? EPT : 4;
    static_assert(kPf == 12, "six row loads per lane, in named registers");
    uint4 pf0 = make_uint4(0, 0, 0, 0), pf1 = pf0, pf2 = pf0, pf3 = pf0, pf4 = pf0, pf5 = pf0;
    int npf = 0, pf_e = -1, pf_slot = 0;  // this lane's held key (index e, or -1) and its LDS row
    if (kAttend) {
        const float edge = (float)(bsel + 1);
        const uint32_t cap = (uint32_t)a.kv_capacity;
        int e1 = -1;
        int32_t r1 = 0;
#pragma unroll
        for (int e = kPfKeys - 1; e >= 0; --e) {
            const int32_t rowi = retr0 + widx[e];
            const bool sure = key[e] != 0u && (key_float(key[e]) - fmin) * inv >= edge && (uint32_t)rowi < cap;
            e1 = sure ? e : e1;
            r1 = sure ? rowi : r1;
        }
        const uint64_t m = __ballot(e1 >= 0);
        const int pos = (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
        npf = min(kPf, (int)__popcll(m));
        if (e1 >= 0 && pos < kPf) {
            s_pfrow[wave][kPf / 2 * (pos & 1) + (pos >> 1)] = r1;
            pf_e = e1;
            pf_slot = wave * kPf + pos;
        }
        // The wave reads back its own LDS words (in order, no barrier needed).  Load u:
        // lanes 0-31 take row 2u (K in lanes 0-15, V in 16-31), lanes 32-63 row 2u + 1;
        // row w sits at word kPf/2 (w % 2) + w / 2, so a lane's ids are consecutive.
        // Loads 0 and 1 go out now, 2 and 3 before the compaction scan, 4 and 5 before
        // the winner list is built (more at once stalled the waves at issue).  The
        // loads are unconditional: a missing row reads the group's row 0 (there is
        // one, kv_capacity >= 1 is checked on the host) and is not used; branches
        // around them made the compiler wait for their data early.
        const uint4* kv = reinterpret_cast<const uint4*>(static_cast<const __half*>((lane & 16) ? a.V : a.K) +
                                                         kvrow0 * kD) + (lane & 15);
        const int hi = lane >> 5;
        const int32_t* idp = &s_pfrow[wave][kPf / 2 * hi];
        pf0 = kv[(int64_t)(hi < npf ? idp[0] : 0) * (kD / 8)];
        pf1 = kv[(int64_t)(2 + hi < npf ? idp[1] : 0) * (kD / 8)];
    }
    uint32_t T, quota;
    if (in_bin <= 64) {
        // Few keys in the bin: gather them, then every wave ranks them by brute force
        // (the same result in each, so no second barrier hands it out).
#pragma unroll
        for (int e = 0; e < EPT; ++e)
            if (key[e] != 0u && bin_of(key[e]) == bsel) s_small[atomicAdd(&s_nsmall, 1u)] = key[e];
        __syncthreads();
        const uint32_t kl = lane < (int)in_bin ? s_small[lane] : 0u;
        uint32_t gt = 0, eq = 0;
        for (uint32_t j = 0; j < in_bin; ++j) {
            const uint32_t kj = s_small[j];
            gt += kj > kl ? 1u : 0u;
            eq += kj == kl ? 1u : 0u;
        }
        const bool hit = lane < (int)in_bin && gt < need && need <= gt + eq;
        const int first = (int)__builtin_ctzll(__ballot(hit));  // some key of the bin has rank need
        T = (uint32_t)__builtin_amdgcn_readlane((int)kl, first);
        quota = need - (uint32_t)__builtin_amdgcn_readlane((int)gt, first);
    } else {
        // Exact radix select on the full key restricted to the bin: 11, 11, 10 bits.
        uint32_t prefix = 0, mask = 0;
        int shift = 21;
#pragma unroll 1
        for (int pass = 1; pass <= 3; ++pass) {
            uint32_t* hist = s_hist[pass & 1];
#pragma unroll
            for (int e = 0; e < EPT; ++e)
                if (key[e] != 0u && (key[e] & mask) == prefix && bin_of(key[e]) == bsel)
                    atomicAdd(&hist[(key[e] >> shift) & (kNB - 1)], 1u);
            __syncthreads();
            if (wave == 0) find_digit<kNB>(hist, need, lane, &s_digit, &s_need);
            // The other buffer was read in the previous pass; clear it for the next one.
            for (int i = tid; i < kNB; i += TH) s_hist[(pass + 1) & 1][i] = 0;
            __syncthreads();
            prefix |= s_digit << shift;
            mask |= (uint32_t)(kNB - 1) << shift;
            need = s_need;
            shift = shift >= 11 ? shift - 11 : 0;
        }
        T = prefix;     // the kk-th largest key value
        quota = need;   // how many keys equal to T are taken (lowest indices)
    }

    if constexpr (kAttend) {
        // Prefetch loads 2 and 3 (see above).
        const uint4* kv = reinterpret_cast<const uint4*>(static_cast<const __half*>((lane & 16) ? a.V : a.K) +
                                                         kvrow0 * kD) + (lane & 15);
        const int hi = lane >> 5;
        const int2 t = *reinterpret_cast<const int2*>(&s_pfrow[wave][kPf / 2 * hi + 2]);
        pf2 = kv[(int64_t)(4 + hi < npf ? t.x : 0) * (kD / 8)];
        pf3 = kv[(int64_t)(6 + hi < npf ? t.y : 0) * (kD / 8)];
    }
    // Ordered compaction: an element's output slot is (#keys > T before it) +
    // min(#keys == T before it, quota), which lists the winners by ascending index.
    // Positions run group by group (j), thread by thread inside a group, so the
    // counts before an element are the earlier groups' totals plus a block scan of
    // this group (counts > T in the low 16 bits, == T in the high 16).
    uint32_t pre[kIt];
#pragma unroll
    for (int it = 0; it < kIt; ++it) {
        uint32_t mine = 0;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const uint32_t k1 = key[4 * it + q];
            mine += (k1 > T) ? 1u : (k1 == T && k1 != 0u) ? 0x10000u : 0u;
        }
        const uint32_t incl = wave_incl_sum(mine);
        if (lane == 63) s_w[it][wave] = incl;
        pre[it] = incl - mine;
    }
    __syncthreads();
    // The waves' totals of each group: lane w < 16 takes wave w's, one wave scan, and
    // the prefix before this wave read from lane wave - 1 (the group total from 15).
    static_assert(kWaves == 16, "one lane per wave in the scan of the wave totals");
    uint32_t before_groups = 0;
#pragma unroll
    for (int it = 0; it < kIt; ++it) {
        const uint32_t x = lane < kWaves ? s_w[it][lane] : 0u;
        const uint32_t ix = wave_incl_sum(x);
        const int wv = __builtin_amdgcn_readfirstlane(wave);
        const uint32_t earlier = wv > 0 ? (uint32_t)__builtin_amdgcn_readlane((int)ix, wv - 1) : 0u;
        const uint32_t tot = (uint32_t)__builtin_amdgcn_readlane((int)ix, kWaves - 1);
        pre[it] += before_groups + earlier;
        before_groups += tot;
    }
    int32_t* oi = a.tk_out_idx + blk * a.top_k;
    float* os = a.tk_out_score ? a.tk_out_score + blk * a.top_k : nullptr;
    // With kAttend the attention list in region B is Sink rows, then Local +
    // Update Buffer rows (nd in all), then the winners at their cache rows
    // (retr_begin + key; the host checked they stay below dense_begin), and the
    // outputs are written after the attention, so that its first loads do not
    // wait behind these stores.
    const int nd = kAttend ? (int)a.win.dense_rows() : 0;
    if constexpr (kAttend) {
        // Prefetch loads 4 and 5 (see above).
        const uint4* kv = reinterpret_cast<const uint4*>(static_cast<const __half*>((lane & 16) ? a.V : a.K) +
                                                         kvrow0 * kD) + (lane & 15);
        const int hi = lane >> 5;
        const int2 t = *reinterpret_cast<const int2*>(&s_pfrow[wave][kPf / 2 * hi + 4]);
        pf4 = kv[(int64_t)(8 + hi < npf ? t.x : 0) * (kD / 8)];
        pf5 = kv[(int64_t)(10 + hi < npf ? t.y : 0) * (kD / 8)];
    }
#pragma unroll
    for (int it = 0; it < kIt; ++it) {
        uint32_t gb = pre[it] & 0xffffu, eb = pre[it] >> 16;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int e = 4 * it + q;
            const bool gt = key[e] > T;
            const bool eq = key[e] == T && key[e] != 0u;
            const uint32_t p = gt ? gb + min(eb, quota) : (eq && eb < quota) ? gb + eb : 0xffffffffu;
            gb += gt ? 1u : 0u;
            eb += eq ? 1u : 0u;
            if (kAttend) {
                // Branch-free: a key that does not win writes this thread's own dump word.
                const bool w = p < (uint32_t)kk;
                int32_t* dw = w ? &s_win[nd + p] : &s_dump[tid];
                float* ds = w ? &s_wsc[p] : reinterpret_cast<float*>(&s_dump[tid]);
                *dw = e == pf_e ? -2 - pf_slot : retr0 + widx[e];
                *ds = key_float(key[e]);
            } else if (p < (uint32_t)kk) {
                oi[p] = widx[e];
                if (os) os[p] = key_float(key[e]);
            }
        }
    }
    if (!kAttend) {
        for (int r = kk + tid; r < a.top_k; r += TH) {
            oi[r] = -1;
            if (os) os[r] = -__builtin_huge_valf();
        }
    }
    if (kAttend) {
        // Attention over the dense rows and the kk winners (Eqs. approx_weight,
        // approx_output), from LDS.  Region B is free once the compaction runs.
        for (int r = tid; r < nd; r += TH) s_win[r] = a.win.dense_entry(r);
        {
            uint4* dst = s_prow + 32 * (wave * kPf + (lane >> 5)) + (lane & 31);
            const int hi = lane >> 5;
            // Unconditional: rows past npf are never listed, and a store on every
            // path keeps the compiler's view of the loads settled from here on.
            dst[0] = pf0;
            dst[2 * 32] = pf1;
            dst[4 * 32] = pf2;
            dst[6 * 32] = pf3;
            dst[8 * 32] = pf4;
            dst[10 * 32] = pf5;
        }
        __syncthreads();
        const bool wc = a.win.win_capacity > 0;
        const int64_t wrow0 = wc ? (int64_t)((int)row / a.g) * a.win.win_capacity : kvrow0;
        attend_row(qv, static_cast<const __half*>(a.K) + kvrow0 * kD,
                   static_cast<const __half*>(a.V) + kvrow0 * kD, a.kv_capacity,
                   static_cast<const __half*>(wc ? a.Kw : a.K) + wrow0 * kD,
                   static_cast<const __half*>(wc ? a.Vw : a.V) + wrow0 * kD, a.win.win_capacity,
                   s_win, nd + kk, a.scale,
                   a.attn_out + row * kD, *reinterpret_cast<AttendScratch*>(s_raw), s_prow);
        // The winners in ascending key index (a held row's from its prefetch record),
        // then the padding.
        for (int r = tid; r < a.top_k; r += TH) {
            const bool w = r < kk;
            int32_t v = w ? s_win[nd + r] : 0;
            if (v <= -2) {
                const int slot = -2 - v, pos = slot % kPf;
                v = s_pfrow[slot / kPf][kPf / 2 * (pos & 1) + (pos >> 1)];
            }
            oi[r] = w ? (int32_t)((int64_t)v - a.win.retr_begin) : -1;
            if (os) os[r] = w ? s_wsc[r] : -__builtin_huge_valf();
        }
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

hipError_t launch_compact_rerank(const RetrieveArgs& a, hipStream_t s) {
    const ProfEvents pe = prof_begin("compact_rerank");
    const dim3 grid((unsigned)a.n_chunks, (unsigned)(a.batch * a.hq));
    if ((int64_t)a.n_chunks * a.batch * a.hq <= kRrWideGrid)
        hipExtLaunchKernelGGL(compact_rerank_kernel<256>, grid, dim3(256), 0, s, pe.start, pe.stop, 0, a);
    else
        hipExtLaunchKernelGGL(compact_rerank_kernel<128>, grid, dim3(128), 0, s, pe.start, pe.stop, 0, a);
    return hipGetLastError();
}

hipError_t launch_topk(const RetrieveArgs& a0, hipStream_t s, bool attend, bool* fused) {
    RetrieveArgs a = a0;
    a.tk_score = a.cand_score;
    a.tk_idx = a.cand;
    a.tk_stride = a.n_cand;
    a.tk_c = a.c_eff;
    a.tk_parts = 1;
    a.tk_part_len = (int32_t)a.c_eff;
    a.tk_out_idx = a.out_idx;
    a.tk_out_score = a.out_score;
    const int64_t rows = (int64_t)a.batch * a.hq;
    if (a.topk_parts > 1) {
        // First pass: the k best of every 4096-candidate slice, in ascending key
        // index.  Every winner of the row is among its slice's k best (fewer than k
        // keys of its slice precede it), so the final pass over the slices' winners,
        // concatenated in slice order, selects the same keys in the same order.
        RetrieveArgs p = a;
        p.tk_parts = a.topk_parts;
        p.tk_part_len = kTopkPart;
        p.tk_out_idx = a.surv_idx;
        p.tk_out_score = a.surv_score;
        const ProfEvents pp = prof_begin("topk_part");
        hipExtLaunchKernelGGL((topk_reg_kernel<1024, 4, false>), dim3((unsigned)(rows * a.topk_parts)), dim3(1024),
                              0, s, pp.start, pp.stop, 0, p);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return e;
        a.tk_score = a.surv_score;
        a.tk_idx = a.surv_idx;
        a.tk_stride = (int64_t)a.topk_parts * a.top_k;
        // only the last slice can hold fewer than k candidates (kTopkPart >= k)
        const int64_t last = a.c_eff - (int64_t)(a.topk_parts - 1) * kTopkPart;
        a.tk_c = (int64_t)(a.topk_parts - 1) * a.top_k + (last < a.top_k ? last : a.top_k);
        a.tk_part_len = (int32_t)a.tk_c;
    }
    const dim3 grid((unsigned)rows);
    const int64_t C = a.tk_c;
    if (fused) *fused = attend;
    const ProfEvents pe = prof_begin(attend ? "topk_attend" : "topk");
#define PARISKV_TOPK_REG(EPT)                                                                        \
    (attend ? hipExtLaunchKernelGGL((topk_reg_kernel<1024, EPT, true>), grid, dim3(1024), 0, s,       \
                                    pe.start, pe.stop, 0, a)                                          \
            : hipExtLaunchKernelGGL((topk_reg_kernel<1024, EPT, false>), grid, dim3(1024), 0, s,      \
                                    pe.start, pe.stop, 0, a))
#define PARISKV_TOPK_LDS(EPT)                                                                        \
    (attend ? hipExtLaunchKernelGGL((topk_lds_kernel<1024, EPT, true>), grid, dim3(1024), 0, s,       \
                                    pe.start, pe.stop, 0, a)                                          \
            : hipExtLaunchKernelGGL((topk_lds_kernel<1024, EPT, false>), grid, dim3(1024), 0, s,      \
                                    pe.start, pe.stop, 0, a))
    if (C <= 1024 * 4)
        PARISKV_TOPK_REG(4);
    else if (C <= 1024 * 8)
        PARISKV_TOPK_REG(8);
    else if (C <= 1024 * 16)
        PARISKV_TOPK_LDS(16);
    else
        PARISKV_TOPK_LDS(32);  // C <= 32768: at most 16 slices x 2048 winners after a first pass
#undef PARISKV_TOPK_LDS
#undef PARISKV_TOPK_REG
    return hipGetLastError();
}

hipError_t launch_pad_outputs(const RetrieveArgs& a, hipStream_t s) {
    const int64_t count = (int64_t)a.batch * a.hq * a.top_k;
    const ProfEvents pe = prof_begin("pad_outputs");
    hipExtLaunchKernelGGL(pad_outputs_kernel, dim3((unsigned)((count + 255) / 256)), dim3(256), 0, s, pe.start, pe.stop, 0,
                       a.out_idx, a.out_score, count);
    return hipGetLastError();
}

}  // namespace pariskv
